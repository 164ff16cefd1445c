// Internal launch interface between the host C-ABI layer and the HIP kernels.
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace dc {

// Everything one decode-step launch needs (device pointers and host-derived scalars).
struct DecodeArgs {
  const void* q;        // [units][G][D]
  const void* k_new;    // [units][D] or null
  const void* v_new;
  void* out;            // [units][G][D]
  void* k;              // [units][cap][D]
  void* v;
  float* alpha;         // feature state, [units][cap]; null for the plain (teacher) step
  double* num;
  double* den;
  int32_t* pos;
  float* vnorm;
  void* qring;          // [units][w][G][D]
  float* qstat;         // [units][w][G][3]
  float* sigma;         // [units][cap] head variance of this step's weights, or null
  int32_t* unit_len;    // [units] rows of each unit before this step (ragged caches), or null:
                        // then every unit has len_old rows; L, len_old are upper bounds
  int64_t cap;
  int units;
  int len_old;          // valid rows before the append
  int L;                // valid rows after the append
  int append;
  float scale;
  int T;                // tokens seen after the append
  int window;           // w (0 = unbounded)
  int slot;             // ring slot written by this step
  int retire;           // the step leaving the window has a ring record
  int arec;             // alpha = this step's mass only (not accumulated)
  int pmax_ret;         // largest position present at that step
  // chunked (split) path scratch
  float* ws_s;          // [units][lmax][G] logits
  float* ws_r;          // [units][lmax][2] retired contributions
  float* ws_v;          // [units][lmax] value norms
  float* ws_part;       // [units][nchunks][3G + G*D] per-chunk softmax partials
  int y0;               // first unit of a launch whose grid rows are units (see for_grid_y)
  int lmax;             // row stride of the scratch per unit: L + 8 rounded up to 32 (rows
                        // past L are padding that absorbs the stores of lanes without a row)
  int chunk;
  int nchunks;
  int fused_rows;       // ragged caches: units of at most this many rows after the append were
                        // served by the single-launch kernel; the chunked kernels skip them (0: none)
};

struct EvictArgs {
  void* k;
  void* v;
  float* alpha;
  double* num;
  double* den;
  int32_t* pos;
  float* vnorm;
  float* sigma;         // [units][cap] or null (moved with the rows; read by 5-input policies)
  const int32_t* unit_len;  // [units] rows of each unit (ragged caches) or null (L rows each)
  const int32_t* budgets;   // [units] budget of each unit, or null (budget for all)
  int ld_kept;          // row stride of kept_out (the budget, or its bound for per-unit budgets)
  const float* params;
  float* scores_out;
  int32_t* kept_out;
  int64_t cap;
  int units;
  int L;
  int budget;           // kept rows after the call (min(budget, L))
  int T;
  int nh;               // hidden layers (1 or 2)
  int h1, h2;
  int n_in;             // 4 or 5 policy inputs
  int ln;               // 1: LayerNorm in every hidden layer
  int ext;              // 1: policy outside the fixed fast paths (n_in 5 or LayerNorm)
  int evict;            // 1 if rows are removed
  uint64_t* ws_keys;    // [units][kstride] row keys (long caches only)
  int mv_ints;          // ints of the compaction move list at the start of the dynamic LDS
  int y0;               // first unit of a launch whose grid rows are units (see for_grid_y)
                        // (the two-hidden-layer policy's weights follow it); set by the launchers
  int sample;           // 1: rank by the Gumbel-perturbed score s / tau + g (training mode)
  float tau;            // sampling temperature
  uint32_t seed0, seed1, draw;  // Philox key and draw number of the Gumbel noise
  int fused_rows;       // ragged caches: units of at most this many rows were scored, selected
                        // and compacted by the single-launch step; these kernels skip them (0: none)
};

// Log-partition / log-probability of size-B subsets (one call covers every unit).
struct LogzArgs {
  const float* scores;      // [units][L] policy scores s_i (row stride L)
  const int32_t* kept;      // [units][nk] kept rows (indices into the scores) or null (row stride nk)
  int nk;                   // min(B, L)
  const int32_t* unit_len;  // [units] rows of each unit (ragged) or null: L for all
  const int32_t* budgets;   // [units] budget of each unit or null: B for all
  double* logz;             // [units] or null
  double* logp;             // [units] or null (needs kept)
  float* col_m;             // [units][L] band column (K > logz_band_entries()) or null
  int* col_k;
  int units, L, B;
  int K;                    // min(B, L - B); 0 when B >= L
  int neg;                  // 1: the programme runs over exp(-r) (K = L - B < B)
  float tau;
};

// REINFORCE rollout terms over [steps][rollouts] arrays.
struct ReinforceArgs {
  const float* rewards;
  const double* logp;
  double* ema;              // [1] in/out
  double* returns;          // required (also read back by the baseline pass)
  double* baseline;         // optional outputs
  double* adv;
  double* weight;
  double* stats;            // [3] loss, mean entropy surrogate, mean return (optional)
  int steps, rollouts;
  double gamma, beta, ema_decay;
};

struct KLArgs {
  const void* h_full;
  const void* h_comp;
  const void* w;
  float* out;
  float* part;          // [rows][ntiles][4]
  int rows, hidden, vocab, ntiles;
  // lm-head addressing: vocabulary row v, hidden elements 64 k .. 64 k + 63 sit at
  // byte (v / 64) 128 hidden + (v mod 64) w_row + k w_stage.  Row-major
  // [vocab][hidden]: w_row = 2 hidden, w_stage = 128; the packed tile layout of
  // dc_kl_pack_lm_head: w_row = 128, w_stage = 8192.
  int w_row, w_stage;
};

// The cross-unit alpha average of one decode step (dc_alpha.hip).
struct GlobalAlphaArgs {
  float* alpha;             // [units][cap]
  const int32_t* pos;       // [units][cap]
  const int32_t* unit_len;  // [units] (ragged caches) or null
  uint64_t* acc;            // [sequences][T] fixed-point sums, then the groups' partial sums
  int64_t cap;
  int units;
  int len;                  // rows per unit (bound with unit_len)
  int per_seq;              // units per sequence (n_layers x n_kv_heads)
  int T;                    // positions 0..T-1
  int y0;                   // first grid row of the launch (see for_grid_y)
};

// Grids whose rows are units (or unit groups) are launched in slices of at
// most MAX_GRID_Y rows (the hardware limit of a grid's y dimension): f(y0, ny)
// launches rows y0 .. y0 + ny - 1, the kernel adding y0 to blockIdx.y.
constexpr int MAX_GRID_Y = 65535;
template <typename F>
inline void for_grid_y(int n, F&& f) {
  for (int y0 = 0; y0 < n; y0 += MAX_GRID_Y) f(y0, n - y0 < MAX_GRID_Y ? n - y0 : MAX_GRID_Y);
}

// Launchers return a hipError_t value (0 on success).
int launch_decode(const DecodeArgs& a, int dtype, int D, int G, bool feat, bool split,
                  void* stream);
int launch_feat_init(const DecodeArgs& a, int dtype, int D, int first_pos, void* stream);
size_t decode_lds_bytes(int L, int G, int D, bool feat);
bool decode_fits_lds(int L, int G, int D);
int decode_chunk_rows();
int launch_evict(const EvictArgs& a, int dtype, int D, void* stream);
int launch_logz(const LogzArgs& a, void* stream);
// Ragged caches: len[u] += add, or len[u] = min(len[u], budgets ? budgets[u] : b).
int launch_unit_len_add(int32_t* len, int units, int add, void* stream);
int launch_unit_len_min(int32_t* len, const int32_t* budgets, int b, int units, void* stream);
int launch_reinforce(const ReinforceArgs& a, void* stream);
size_t logz_ws_bytes(int units, int L, int B);
int logz_band_entries();
int evict_max_len();
size_t evict_ws_bytes(int units, int L);
size_t evict_ext_ws_bytes(int units, int L);
int launch_kl(const KLArgs& a, void* stream);
int launch_kl_pack(const void* w, void* packed, int hidden, int vocab, void* stream);
// Device address of the allocation-free KL entry point's scratch on the current
// device (looked up once per device); 0 on success.
int kl_static_scratch(float** out);
int launch_global_alpha(const GlobalAlphaArgs& a, void* stream);
int global_alpha_groups(int per_seq);    // unit groups of one sequence (workspace sizing)
// bf16 matrix-core step (dc_step.hip); e != nullptr fuses scoring and eviction.
int launch_step(const DecodeArgs& a, const EvictArgs* e, int D, int G, bool feat, bool chunked,
                void* stream);
bool step_fits(int L, int G, int D, bool feat, int nmoves);
// Ragged caches: the most rows per unit (after the append) the single-launch
// step serves at two workgroups per CU, or 0 when it serves no unit of this shape.
int step_ragged_rows(int G, int D);
int step_chunk_rows();
int kl_tile_cols();

}  // namespace dc
