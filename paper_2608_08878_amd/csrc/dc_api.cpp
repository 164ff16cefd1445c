// Host side of the C ABI: argument validation (no HIP call before it passes),
// workspace sizing, path selection and host bookkeeping.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include "../../include/distillcache.h"
#include "dc_kernels.hpp"

namespace {

constexpr int EVICT_REG_ROWS = 8192;
constexpr int MAX_MOVES = 16384;   // rows one compaction may move (its move list is in LDS)

int64_t units_of(const dc_dims* d) { return (int64_t)d->batch * d->n_layers * d->n_kv_heads; }
int group_of(const dc_dims* d) { return d->n_q_heads / d->n_kv_heads; }

dc_status check_dims(const dc_dims* d) {
  if (!d) return DC_ERR_NULL;
  if (d->batch < 1 || d->n_layers < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1 || d->capacity < 1 ||
      d->head_dim < 1)
    return DC_ERR_SHAPE;
  if (d->n_q_heads % d->n_kv_heads) return DC_ERR_SHAPE;
  const int G = group_of(d);
  if (G != 1 && G != 2 && G != 4 && G != 8) return DC_ERR_UNSUPPORTED;
  if (d->head_dim != 64 && d->head_dim != 128) return DC_ERR_UNSUPPORTED;
  if (d->dtype != DC_F32 && d->dtype != DC_BF16) return DC_ERR_UNSUPPORTED;
  if (d->ent_window < 0 || d->ent_window > DC_MAX_WINDOW) return DC_ERR_SHAPE;
  if (!(d->scale >= 0.0f) || isinf(d->scale)) return DC_ERR_SHAPE;
  if (units_of(d) > (1 << 24) || d->capacity > (1 << 26)) return DC_ERR_UNSUPPORTED;
  return DC_OK;
}

float scale_of(const dc_dims* d) { return d->scale > 0.0f ? d->scale : 1.0f / sqrtf((float)d->head_dim); }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Units below which one workgroup per unit leaves most of the chip idle.
constexpr int FEW_UNITS = 128;
// bf16 caches of more than one chunk of rows on this many units or fewer take
// the chunked decode as well.  Measured per step (decode, scoring, selection
// and compaction), single launch -> chunked: 8 units 43.5 -> 39.0 us at 2049
// rows and 59.6 -> 42.3 us at 3073 rows, 48 units 45.9 -> 42.1 and
// 61.5 -> 55.6 us; at 64 units 2049 rows favour the single launch (45.7
// against 51.9 us), and 1025 rows always do (28 us against 33-36 us).
constexpr int VERY_FEW_UNITS = 48;
constexpr int MIN_CHUNK = 512;   // rows per workgroup on the chunked path, at least

// Rows per workgroup on the chunked path.  Many units (or fp32): full chunks.
// Few bf16 units: at most 16 chunks per unit (every workgroup of the combining
// kernels walks all of its unit's partials) and about 512 workgroups in all,
// rounded up to 128 rows and kept within [512, full chunk].  Measured for 1-64
// units at 4097-32769 rows: 1-8 units of 4097 rows take 46-47 us per step
// against 61-63 us with full chunks; the rule never measured slower.
int chunk_rows(const dc_dims* d, int L) {
  const int c = dc::decode_chunk_rows();
  const long U = (long)units_of(d);
  if (d->dtype != DC_BF16 || U >= FEW_UNITS) return c;
  const long by_chunks = (L + 15) / 16, by_groups = ((long)L * U + 511) / 512;
  const long want = by_chunks > by_groups ? by_chunks : by_groups;
  const long r = (want + 127) / 128 * 128;
  return r < MIN_CHUNK ? MIN_CHUNK : r > c ? c : (int)r;
}

int nchunks_of(const dc_dims* d, int L) {
  const int c = chunk_rows(d, L);
  return (L + c - 1) / c;
}

// Chunks of any length up to L: the workspace bound (the chunk grows with L,
// so the count is not monotone in L).
int nchunks_bound(const dc_dims* d, int L) {
  const bool few = d->dtype == DC_BF16 && units_of(d) < FEW_UNITS;
  return few ? (L + MIN_CHUNK - 1) / MIN_CHUNK : nchunks_of(d, L);
}

// Per-unit row stride of the decode scratch: L rows plus padding that takes the
// stores of lanes past the last row (so those stores need no branch), rounded
// to 32 rows so that every unit's rows start on a 256-byte boundary (a 16-row
// tile of retired pairs is then exactly one 128-byte line).
int scratch_rows(int L) { return (L + 8 + 31) / 32 * 32; }

// Scratch of the chunked decode path for caches of L rows.
size_t split_bytes(const dc_dims* d, int L) {
  const size_t U = (size_t)units_of(d), G = group_of(d), D = d->head_dim;
  const size_t rows = U * (size_t)scratch_rows(L) * (G + 3) * sizeof(float);
  const size_t parts = U * (size_t)nchunks_bound(d, L) * (3 * G + G * D) * sizeof(float);
  return align256(rows) + align256(parts);
}

bool use_split(const dc_dims* d, int L, bool feat) {
  const int G = group_of(d);
  if (feat && !dc::decode_fits_lds(L, G, d->head_dim)) return true;
  // few units: spread one unit's rows over several workgroups
  return units_of(d) < FEW_UNITS && L > 2 * dc::decode_chunk_rows();
}

size_t evict_bytes(const dc_dims* d, int L) { return align256(dc::evict_ws_bytes((int)units_of(d), L)); }

size_t kl_bytes(int rows, int vocab) {
  return align256((size_t)rows * (size_t)(vocab / dc::kl_tile_cols()) * 4 * sizeof(float));
}

}  // namespace

extern "C" {

const char* dc_status_str(dc_status s) {
  switch (s) {
    case DC_OK: return "DC_OK";
    case DC_ERR_NULL: return "DC_ERR_NULL: a required pointer is NULL";
    case DC_ERR_SHAPE: return "DC_ERR_SHAPE: inconsistent sizes";
    case DC_ERR_UNSUPPORTED: return "DC_ERR_UNSUPPORTED: shape or option not implemented";
    case DC_ERR_CAPACITY: return "DC_ERR_CAPACITY: append exceeds the cache capacity";
    case DC_ERR_BUDGET: return "DC_ERR_BUDGET: budget must be >= 1";
    case DC_ERR_WORKSPACE: return "DC_ERR_WORKSPACE: workspace missing or too small";
    case DC_ERR_HIP: return "DC_ERR_HIP: a HIP launch failed";
    case DC_ERR_VALUE: return "DC_ERR_VALUE: scalar argument out of range";
    case DC_ERR_SCRATCH: return "DC_ERR_SCRATCH: larger than the fixed scratch of the allocation-free entry point";
  }
  return "unknown dc_status";
}

size_t dc_workspace_bytes(const dc_dims* dims, int32_t max_len, int32_t kl_rows, int32_t kl_vocab) {
  size_t need = 0;
  if (max_len > 0) {
    if (check_dims(dims) != DC_OK) return 0;
    const size_t a = split_bytes(dims, max_len), b = evict_bytes(dims, max_len);
    const size_t x = align256(dc::evict_ext_ws_bytes((int)units_of(dims), max_len));
    need = a > b ? a : b;
    need = x > need ? x : need;
  }
  if (kl_rows > 0 && kl_vocab > 0) {
    const size_t c = kl_bytes(kl_rows, kl_vocab);
    need = c > need ? c : need;
  }
  return need;
}

dc_status dc_feat_init(const dc_dims* dims, const dc_kv* kv, dc_feat* feat, int32_t first_pos,
                       void* hip_stream) {
  dc_status st = check_dims(dims);
  if (st != DC_OK) return st;
  if (!kv || !feat || !kv->v || !feat->alpha || !feat->ent_num || !feat->ent_den || !feat->pos ||
      !feat->vnorm)
    return DC_ERR_NULL;
  if (kv->len < 0 || kv->len > dims->capacity || first_pos < 0) return DC_ERR_SHAPE;
  if (kv->len > 0) {
    dc::DecodeArgs a;
    memset(&a, 0, sizeof(a));
    a.v = kv->v;
    a.alpha = feat->alpha;
    a.num = feat->ent_num;
    a.den = feat->ent_den;
    a.pos = feat->pos;
    a.vnorm = feat->vnorm;
    a.sigma = feat->sigma;
    a.cap = dims->capacity;
    a.units = (int)units_of(dims);
    a.L = kv->len;
    if (dc::launch_feat_init(a, dims->dtype, dims->head_dim, first_pos, hip_stream) != 0)
      return DC_ERR_HIP;
  }
  feat->step = 0;
  feat->next_pos = first_pos + kv->len;
  memset(feat->ring_pmax, 0, sizeof(feat->ring_pmax));
  return DC_OK;
}

int32_t dc_dynamic_budget(float ratio, int32_t seq_len, int32_t b_min) {
  if (!(ratio > 0.0f && ratio <= 1.0f) || seq_len < 0 || b_min < 1) return -1;
  const double b = floor((double)ratio * (double)seq_len);
  return b > (double)b_min ? (int32_t)b : b_min;
}

dc_status dc_reinforce_terms(int32_t steps, int32_t rollouts, const dc_reinforce_cfg* cfg,
                             const float* rewards, const double* logp, double* ema,
                             double* returns_out, double* baseline_out, double* adv_out,
                             double* weight_out, double* stats_out, void* hip_stream) {
  if (!cfg || !rewards || !logp || !ema || !returns_out) return DC_ERR_NULL;
  if (steps < 1 || rollouts < 1) return DC_ERR_SHAPE;
  if ((int64_t)steps * rollouts > (1 << 26)) return DC_ERR_UNSUPPORTED;
  if (!(cfg->gamma >= 0.0 && cfg->gamma <= 1.0) || !isfinite(cfg->beta) ||
      !(cfg->ema_decay >= 0.0 && cfg->ema_decay < 1.0))
    return DC_ERR_VALUE;
  dc::ReinforceArgs a;
  a.rewards = rewards;
  a.logp = logp;
  a.ema = ema;
  a.returns = returns_out;
  a.baseline = baseline_out;
  a.adv = adv_out;
  a.weight = weight_out;
  a.stats = stats_out;
  a.steps = steps;
  a.rollouts = rollouts;
  a.gamma = cfg->gamma;
  a.beta = cfg->beta;
  a.ema_decay = cfg->ema_decay;
  if (dc::launch_reinforce(a, hip_stream) != 0) return DC_ERR_HIP;
  return DC_OK;
}

}  // extern "C"

namespace {

// Validate a decode step and fill its launch arguments; no side effects.
dc_status prep_decode(const dc_dims* dims, const dc_kv* kv, const dc_feat* feat, const void* q,
                      const void* k_new, const void* v_new, void* out, void* ws, size_t ws_bytes,
                      dc::DecodeArgs& a, bool& split, size_t& need) {
  dc_status st = check_dims(dims);
  if (st != DC_OK) return st;
  if (!kv || !kv->k || !kv->v || !q || !out) return DC_ERR_NULL;
  if ((k_new == nullptr) != (v_new == nullptr)) return DC_ERR_NULL;
  const int W = dims->ent_window;
  if (feat) {
    if (!feat->alpha || !feat->ent_num || !feat->ent_den || !feat->pos || !feat->vnorm)
      return DC_ERR_NULL;
    if (W > 0 && (!feat->qring || !feat->qstat)) return DC_ERR_NULL;
    if (feat->step < 0 || feat->next_pos < 0) return DC_ERR_SHAPE;
    if (feat->alpha_recent != 0 && feat->alpha_recent != 1) return DC_ERR_VALUE;
  }
  const int len = kv->len;
  const int append = k_new != nullptr;
  if (len < 0 || len > dims->capacity) return DC_ERR_SHAPE;
  if (append && len + 1 > dims->capacity) return DC_ERR_CAPACITY;
  if (!append && len == 0) return DC_ERR_SHAPE;
  const int L = len + append;
  const int G = group_of(dims), D = dims->head_dim;
  const int U = (int)units_of(dims);
  const bool ragged = kv->unit_len != nullptr;
  if (ragged && dims->dtype != DC_BF16) return DC_ERR_UNSUPPORTED;
  if (dims->dtype == DC_BF16)
    split = ragged || !dc::step_fits(L, G, D, feat != nullptr, 0) ||
            (U < FEW_UNITS && L > 2 * dc::step_chunk_rows()) ||
            (U <= VERY_FEW_UNITS && L > dc::step_chunk_rows());
  else
    split = use_split(dims, L, feat != nullptr);
  // the matrix-core unit path parks each row's retired (cz, cn) in the workspace
  const bool unit_scratch = dims->dtype == DC_BF16 && feat && !split;
  need = split ? split_bytes(dims, L)
         : unit_scratch ? align256((size_t)U * scratch_rows(L) * 2 * sizeof(float)) : 0;
  if (need && (!ws || ws_bytes < need)) return DC_ERR_WORKSPACE;

  memset(&a, 0, sizeof(a));
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.out = out;
  a.k = kv->k;
  a.v = kv->v;
  a.cap = dims->capacity;
  a.units = U;
  a.len_old = len;
  a.L = L;
  a.append = append;
  a.unit_len = kv->unit_len;
  a.scale = scale_of(dims);
  if (feat) {
    a.alpha = feat->alpha;
    a.num = feat->ent_num;
    a.den = feat->ent_den;
    a.pos = feat->pos;
    a.vnorm = feat->vnorm;
    a.sigma = feat->sigma;
    a.qring = feat->qring;
    a.qstat = feat->qstat;
    a.T = feat->next_pos + append;
    a.arec = feat->alpha_recent;
    a.window = W;
    if (W > 0) {
      a.slot = feat->step % W;
      a.retire = feat->step >= W;
      a.pmax_ret = a.retire ? feat->ring_pmax[a.slot] : 0;
    }
  }
  if (unit_scratch) {
    a.ws_r = (float*)ws;
    a.lmax = scratch_rows(L);
  }
  if (split) {
    const size_t rows = (size_t)U * scratch_rows(L);
    float* base = (float*)ws;
    a.lmax = scratch_rows(L);
    a.chunk = chunk_rows(dims, L);
    a.nchunks = nchunks_of(dims, L);
    a.ws_s = base;
    a.ws_r = base + rows * G;
    a.ws_v = base + rows * (G + 2);
    a.ws_part = (float*)((char*)ws + align256(rows * (G + 3) * sizeof(float)));
  }
  return DC_OK;
}

dc_status launch_decode_any(const dc_dims* dims, const dc::DecodeArgs& a, bool feat, bool split,
                            void* stream) {
  const int G = group_of(dims), D = dims->head_dim;
  const int rc = dims->dtype == DC_BF16 ? dc::launch_step(a, nullptr, D, G, feat, split, stream)
                                        : dc::launch_decode(a, dims->dtype, D, G, feat, split, stream);
  return rc == 0 ? DC_OK : DC_ERR_HIP;
}

void commit_decode(dc_kv* kv, dc_feat* feat, const dc::DecodeArgs& a, int W) {
  kv->len = a.L;
  if (feat) {
    feat->next_pos += a.append;
    if (W > 0) feat->ring_pmax[a.slot] = feat->next_pos - 1;
    feat->step += 1;
  }
}

// Validate a score/evict call on a cache of L rows with T tokens seen.
dc_status prep_evict(const dc_dims* dims, const dc_kv* kv, const dc_feat* feat,
                     const dc_policy* policy, int32_t budget, float* scores_out, int32_t* kept_out,
                     void* ws, size_t ws_bytes, int L, int T, dc::EvictArgs& e, size_t& need) {
  dc_status st = check_dims(dims);
  if (st != DC_OK) return st;
  if (!kv || !kv->k || !kv->v || !feat || !policy || !policy->params) return DC_ERR_NULL;
  if (!feat->alpha || !feat->ent_num || !feat->ent_den || !feat->pos || !feat->vnorm)
    return DC_ERR_NULL;
  if ((policy->n_in != 4 && policy->n_in != 5) ||
      (policy->n_hidden_layers != 1 && policy->n_hidden_layers != 2) ||
      (policy->layer_norm != 0 && policy->layer_norm != 1))
    return DC_ERR_UNSUPPORTED;
  if (policy->hidden[0] < 1 || policy->hidden[0] > 128) return DC_ERR_UNSUPPORTED;
  if (policy->n_hidden_layers == 2 && (policy->hidden[1] < 1 || policy->hidden[1] > 128))
    return DC_ERR_UNSUPPORTED;
  // outside the fused one-hidden-layer path: a fifth input, LayerNorm, or a
  // second hidden layer (a dense contraction: the matrix-core scoring pass)
  const int ext = policy->n_in == 5 || policy->layer_norm || policy->n_hidden_layers == 2;
  if (policy->n_in == 5 && !feat->sigma) return DC_ERR_NULL;
  if (budget < 1) return DC_ERR_BUDGET;
  if (L < 1 || L > dims->capacity) return DC_ERR_SHAPE;
  if (L > dc::evict_max_len()) return DC_ERR_UNSUPPORTED;
  if (T < 1) return DC_ERR_SHAPE;
  const int evict = budget < L;
  const bool ragged = kv->unit_len != nullptr;
  if (ragged && dims->dtype != DC_BF16) return DC_ERR_UNSUPPORTED;
  // the compaction's move list (two ints per move) lives in LDS
  // (per unit min(L_u - B_u, B_u) <= L_u / 2)
  const int moves = ragged ? (L / 2 < budget ? L / 2 : budget) : evict ? (L - budget < budget ? L - budget : budget) : 0;
  if (moves > MAX_MOVES) return DC_ERR_UNSUPPORTED;
  need = (ext || ragged) ? align256(dc::evict_ext_ws_bytes((int)units_of(dims), L))
                         : (L > EVICT_REG_ROWS ? evict_bytes(dims, L) : 0);
  if (need && (!ws || ws_bytes < need)) return DC_ERR_WORKSPACE;
  memset(&e, 0, sizeof(e));
  e.k = kv->k;
  e.v = kv->v;
  e.alpha = feat->alpha;
  e.num = feat->ent_num;
  e.den = feat->ent_den;
  e.pos = feat->pos;
  e.vnorm = feat->vnorm;
  e.sigma = feat->sigma;
  e.params = policy->params;
  e.scores_out = scores_out;
  e.kept_out = kept_out;
  e.cap = dims->capacity;
  e.units = (int)units_of(dims);
  e.L = L;
  e.budget = evict ? budget : L;
  e.ld_kept = e.budget;
  e.unit_len = kv->unit_len;
  e.T = T;
  e.nh = policy->n_hidden_layers;
  e.h1 = policy->hidden[0];
  e.h2 = policy->n_hidden_layers == 2 ? policy->hidden[1] : 0;
  e.n_in = policy->n_in;
  e.ln = policy->layer_norm;
  e.ext = ext;
  e.evict = evict;
  e.ws_keys = (uint64_t*)ws;
  return DC_OK;
}

// Ragged caches: each unit's length follows its append / eviction on the stream.
dc_status ragged_after_decode(const dc_kv* kv, const dc::DecodeArgs& a, void* stream) {
  if (!kv->unit_len || !a.append) return DC_OK;
  return dc::launch_unit_len_add(kv->unit_len, a.units, 1, stream) ? DC_ERR_HIP : DC_OK;
}
dc_status ragged_after_evict(const dc_kv* kv, const dc::EvictArgs& e, const int32_t* budgets,
                             int bmax, void* stream) {
  if (!kv->unit_len || (!budgets && !e.evict)) return DC_OK;
  return dc::launch_unit_len_min(kv->unit_len, budgets, bmax, e.units, stream) ? DC_ERR_HIP : DC_OK;
}

// Validate a log-partition call and fill its arguments.
dc_status prep_logz(int32_t units, int32_t L, int32_t B, float tau, const float* scores,
                    const int32_t* kept, double* logz, double* logp, void* ws, size_t ws_bytes,
                    dc::LogzArgs& z) {
  if (!scores || (logp && !kept)) return DC_ERR_NULL;
  if (units < 1 || L < 1) return DC_ERR_SHAPE;
  if (B < 1) return DC_ERR_BUDGET;
  if (!(tau > 0.0f) || isinf(tau)) return DC_ERR_VALUE;
  if (L > dc::evict_max_len() || units > (1 << 24)) return DC_ERR_UNSUPPORTED;
  const size_t need = dc::logz_ws_bytes(units, L, B);
  if (need && (!ws || ws_bytes < need)) return DC_ERR_WORKSPACE;
  memset(&z, 0, sizeof(z));
  z.scores = scores;
  z.kept = logp ? kept : nullptr;
  z.nk = B < L ? B : L;
  z.logz = logz;
  z.logp = logp;
  if (need) {
    z.col_m = (float*)ws;
    z.col_k = (int*)((char*)ws + (size_t)units * L * sizeof(float));
  }
  z.units = units;
  z.L = L;
  z.B = B;
  z.K = B >= L ? 0 : (B <= L - B ? B : L - B);
  z.neg = B < L && L - B < B;
  z.tau = tau;
  return DC_OK;
}

dc_status kl_check(int32_t rows, int32_t hidden, int32_t vocab, const void* h_full,
                   const void* h_comp, const void* w_lm, const float* kl_out) {
  if (!h_full || !h_comp || !w_lm || !kl_out) return DC_ERR_NULL;
  if (rows < 1 || hidden < 1 || vocab < 1) return DC_ERR_SHAPE;
  if (rows > DC_KL_MAX_ROWS || hidden % 128 || vocab % dc::kl_tile_cols()) return DC_ERR_UNSUPPORTED;
  return DC_OK;
}

// part: rows * (vocab / 64) * 4 floats of per-(row, tile) statistics.
dc_status kl_launch(int32_t rows, int32_t hidden, int32_t vocab, const void* h_full,
                    const void* h_comp, const void* w_lm, float* kl_out, float* part,
                    void* hip_stream, bool packed = false) {
  dc::KLArgs a;
  a.h_full = h_full;
  a.h_comp = h_comp;
  a.w = w_lm;
  a.out = kl_out;
  a.part = part;
  a.rows = rows;
  a.hidden = hidden;
  a.vocab = vocab;
  a.ntiles = vocab / dc::kl_tile_cols();
  // where a vocabulary row and a 64-element stage of it sit in the lm head
  a.w_row = packed ? 128 : 2 * hidden;
  a.w_stage = packed ? 128 * dc::kl_tile_cols() : 128;
  return dc::launch_kl(a, hip_stream) == 0 ? DC_OK : DC_ERR_HIP;
}

}  // namespace

extern "C" {

dc_status dc_decode_step(const dc_dims* dims, dc_kv* kv, dc_feat* feat, const void* q,
                         const void* k_new, const void* v_new, void* out, void* ws,
                         size_t ws_bytes, void* hip_stream) {
  dc::DecodeArgs a;
  bool split = false;
  size_t need = 0;
  dc_status st = prep_decode(dims, kv, feat, q, k_new, v_new, out, ws, ws_bytes, a, split, need);
  if (st != DC_OK) return st;
  st = launch_decode_any(dims, a, feat != nullptr, split, hip_stream);
  if (st != DC_OK) return st;
  if (ragged_after_decode(kv, a, hip_stream) != DC_OK) return DC_ERR_HIP;
  commit_decode(kv, feat, a, dims->ent_window);
  return DC_OK;
}

dc_status dc_score_evict(const dc_dims* dims, dc_kv* kv, dc_feat* feat, const dc_policy* policy,
                         int32_t budget, float* scores_out, int32_t* kept_out, void* ws,
                         size_t ws_bytes, void* hip_stream) {
  if (!kv || !feat) return DC_ERR_NULL;
  dc::EvictArgs e;
  size_t need = 0;
  dc_status st = prep_evict(dims, kv, feat, policy, budget, scores_out, kept_out, ws, ws_bytes,
                            kv->len, feat->next_pos, e, need);
  if (st != DC_OK) return st;
  if (dc::launch_evict(e, dims->dtype, dims->head_dim, hip_stream) != 0) return DC_ERR_HIP;
  if (ragged_after_evict(kv, e, nullptr, e.budget, hip_stream) != DC_OK) return DC_ERR_HIP;
  kv->len = e.budget;
  return DC_OK;
}

dc_status dc_sample_evict(const dc_dims* dims, dc_kv* kv, dc_feat* feat, const dc_policy* policy,
                          int32_t budget, const dc_gumbel* gumbel, float* scores_out,
                          int32_t* kept_out, double* logp_out, void* ws, size_t ws_bytes,
                          void* hip_stream) {
  if (!kv || !feat || !gumbel) return DC_ERR_NULL;
  if (logp_out && (!scores_out || !kept_out)) return DC_ERR_NULL;
  dc::EvictArgs e;
  size_t need = 0;
  dc_status st = prep_evict(dims, kv, feat, policy, budget, scores_out, kept_out, ws, ws_bytes,
                            kv->len, feat->next_pos, e, need);
  if (st != DC_OK) return st;
  if (!(gumbel->tau > 0.0f) || isinf(gumbel->tau)) return DC_ERR_VALUE;
  e.sample = 1;
  e.tau = gumbel->tau;
  e.seed0 = gumbel->seed[0];
  e.seed1 = gumbel->seed[1];
  e.draw = gumbel->draw;
  dc::LogzArgs z;
  if (logp_out) {
    // the log-partition runs after the selection on the same stream and may
    // reuse the selection's workspace
    st = prep_logz(e.units, e.L, budget, gumbel->tau, scores_out, kept_out, nullptr, logp_out, ws,
                   ws_bytes, z);
    if (st != DC_OK) return st;
    z.unit_len = kv->unit_len;      // pre-eviction lengths: committed after the log-partition
  }
  if (dc::launch_evict(e, dims->dtype, dims->head_dim, hip_stream) != 0) return DC_ERR_HIP;
  if (logp_out && dc::launch_logz(z, hip_stream) != 0) return DC_ERR_HIP;
  if (ragged_after_evict(kv, e, nullptr, e.budget, hip_stream) != DC_OK) return DC_ERR_HIP;
  kv->len = e.budget;
  return DC_OK;
}

dc_status dc_decode_sample_evict(const dc_dims* dims, dc_kv* kv, dc_feat* feat,
                                 const dc_policy* policy, int32_t budget, const dc_gumbel* gumbel,
                                 const void* q, const void* k_new, const void* v_new, void* out,
                                 float* scores_out, int32_t* kept_out, double* logp_out, void* ws,
                                 size_t ws_bytes, void* hip_stream) {
  if (!feat || !gumbel) return DC_ERR_NULL;
  if (logp_out && (!scores_out || !kept_out)) return DC_ERR_NULL;
  dc::DecodeArgs a;
  bool split = false;
  size_t need_d = 0, need_e = 0;
  dc_status st = prep_decode(dims, kv, feat, q, k_new, v_new, out, ws, ws_bytes, a, split, need_d);
  if (st != DC_OK) return st;
  dc::EvictArgs e;
  st = prep_evict(dims, kv, feat, policy, budget, scores_out, kept_out, ws, ws_bytes, a.L, a.T, e,
                  need_e);
  if (st != DC_OK) return st;
  if (!(gumbel->tau > 0.0f) || isinf(gumbel->tau)) return DC_ERR_VALUE;
  e.sample = 1;
  e.tau = gumbel->tau;
  e.seed0 = gumbel->seed[0];
  e.seed1 = gumbel->seed[1];
  e.draw = gumbel->draw;
  dc::LogzArgs z;
  if (logp_out) {
    st = prep_logz(e.units, a.L, budget, gumbel->tau, scores_out, kept_out, nullptr, logp_out, ws,
                   ws_bytes, z);
    if (st != DC_OK) return st;
  }
  const int G = group_of(dims), D = dims->head_dim;
  const int nm = e.evict ? (a.L - e.budget < e.budget ? a.L - e.budget : e.budget) : 0;
  const bool fused = dims->dtype == DC_BF16 && !split && !e.ext && !feat->sigma && G >= 4 &&
                     !kv->unit_len && dc::step_fits(a.L, G, D, true, nm);
  if (fused) {
    if (dc::launch_step(a, &e, D, G, true, false, hip_stream) != 0) return DC_ERR_HIP;
  } else {
    st = launch_decode_any(dims, a, true, split, hip_stream);
    if (st != DC_OK) return st;
    if (ragged_after_decode(kv, a, hip_stream) != DC_OK) return DC_ERR_HIP;
    if (dc::launch_evict(e, dims->dtype, D, hip_stream) != 0) return DC_ERR_HIP;
  }
  if (logp_out) {
    z.unit_len = kv->unit_len;
    if (dc::launch_logz(z, hip_stream) != 0) return DC_ERR_HIP;
  }
  if (ragged_after_evict(kv, e, nullptr, e.budget, hip_stream) != DC_OK) return DC_ERR_HIP;
  commit_decode(kv, feat, a, dims->ent_window);
  kv->len = e.budget;
  return DC_OK;
}

dc_status dc_score_evict_units(const dc_dims* dims, dc_kv* kv, dc_feat* feat, const dc_policy* policy,
                               const int32_t* budgets, int32_t max_budget, const dc_gumbel* gumbel,
                               float* scores_out, int32_t* kept_out, double* logp_out, void* ws,
                               size_t ws_bytes, void* hip_stream) {
  if (!kv || !feat || !budgets || !kv->unit_len) return DC_ERR_NULL;
  if (logp_out && (!gumbel || !scores_out || !kept_out)) return DC_ERR_NULL;
  dc::EvictArgs e;
  size_t need = 0;
  dc_status st = prep_evict(dims, kv, feat, policy, max_budget, scores_out, kept_out, ws, ws_bytes,
                            kv->len, feat->next_pos, e, need);
  if (st != DC_OK) return st;
  e.budgets = budgets;              // per unit, clamped to [1, e.budget] by the kernels
  if (gumbel) {
    if (!(gumbel->tau > 0.0f) || isinf(gumbel->tau)) return DC_ERR_VALUE;
    e.sample = 1;
    e.tau = gumbel->tau;
    e.seed0 = gumbel->seed[0];
    e.seed1 = gumbel->seed[1];
    e.draw = gumbel->draw;
  }
  dc::LogzArgs z;
  if (logp_out) {
    // K of any unit is at most min(budget, rows / 2): the kernel is chosen for that bound
    st = prep_logz(e.units, e.L, e.budget, gumbel->tau, scores_out, kept_out, nullptr, logp_out, ws,
                   ws_bytes, z);
    if (st != DC_OK) return st;
    z.unit_len = kv->unit_len;
    z.budgets = budgets;
    z.nk = e.ld_kept;
    z.K = e.budget < e.L / 2 ? e.budget : e.L / 2;
    if (z.K > dc::logz_band_entries()) {
      // band history for that bound: 8 B per row, inside the row-key workspace
      // the selection used (it is finished with it when the log-partition runs)
      const size_t band = (size_t)e.units * e.L * (sizeof(float) + sizeof(int));
      if (!ws || ws_bytes < band) return DC_ERR_WORKSPACE;
      z.col_m = (float*)ws;
      z.col_k = (int*)((char*)ws + (size_t)e.units * e.L * sizeof(float));
    }
  }
  if (dc::launch_evict(e, dims->dtype, dims->head_dim, hip_stream) != 0) return DC_ERR_HIP;
  if (logp_out && dc::launch_logz(z, hip_stream) != 0) return DC_ERR_HIP;
  if (ragged_after_evict(kv, e, budgets, e.budget, hip_stream) != DC_OK) return DC_ERR_HIP;
  kv->len = e.budget;
  return DC_OK;
}

dc_status dc_decode_evict_units(const dc_dims* dims, dc_kv* kv, dc_feat* feat,
                                const dc_policy* policy, const int32_t* budgets, int32_t max_budget,
                                const void* q, const void* k_new, const void* v_new, void* out,
                                float* scores_out, int32_t* kept_out, void* ws, size_t ws_bytes,
                                void* hip_stream) {
  if (!kv || !feat || !budgets || !kv->unit_len || !k_new || !v_new) return DC_ERR_NULL;
  dc::DecodeArgs a;
  bool split = false;
  size_t need_d = 0, need_e = 0;
  dc_status st = prep_decode(dims, kv, feat, q, k_new, v_new, out, ws, ws_bytes, a, split, need_d);
  if (st != DC_OK) return st;
  dc::EvictArgs e;
  st = prep_evict(dims, kv, feat, policy, max_budget, scores_out, kept_out, ws, ws_bytes, a.L, a.T,
                  e, need_e);
  if (st != DC_OK) return st;
  e.budgets = budgets;              // per unit, clamped to [1, e.budget] by the kernels
  const int G = group_of(dims), D = dims->head_dim;
  // units of up to Lf rows after the append: the single-launch step (decode,
  // features, the fused one-hidden-layer policy, per-unit top-B, compaction).
  // Few units take the chunked decode whatever their rows: one workgroup per
  // unit leaves most of the chip idle (as for uniform caches)
  const int Lf = dc::step_ragged_rows(G, D);
  if (e.ext || feat->sigma || Lf < 1 || (int)units_of(dims) < FEW_UNITS) {
    // the two-call route: chunked decode, then the per-unit selection
    st = launch_decode_any(dims, a, true, split, hip_stream);
    if (st != DC_OK) return st;
    if (ragged_after_decode(kv, a, hip_stream) != DC_OK) return DC_ERR_HIP;
    if (dc::launch_evict(e, dims->dtype, D, hip_stream) != 0) return DC_ERR_HIP;
  } else {
    dc::DecodeArgs af = a;
    af.L = a.L < Lf ? a.L : Lf;     // the rows one workgroup serves (LDS); longer units leave
    dc::EvictArgs ef = e;
    ef.L = a.L;                     // row stride of scores_out
    if (dc::launch_step(af, &ef, D, G, true, false, hip_stream) != 0) return DC_ERR_HIP;
    if (a.L > af.L) {
      // the longer units: chunked decode, then their scoring and selection
      dc::DecodeArgs ac = a;
      ac.fused_rows = af.L;
      st = launch_decode_any(dims, ac, true, true, hip_stream);
      if (st != DC_OK) return st;
    }
    // every kernel of the decode has read the old lengths
    if (ragged_after_decode(kv, a, hip_stream) != DC_OK) return DC_ERR_HIP;
    if (a.L > af.L) {
      dc::EvictArgs el = e;
      el.fused_rows = af.L;
      if (dc::launch_evict(el, dims->dtype, D, hip_stream) != 0) return DC_ERR_HIP;
    }
  }
  if (ragged_after_evict(kv, e, budgets, e.budget, hip_stream) != DC_OK) return DC_ERR_HIP;
  commit_decode(kv, feat, a, dims->ent_window);
  kv->len = e.budget;
  return DC_OK;
}

dc_status dc_subset_log_prob(int32_t units, int32_t len, int32_t budget, float tau,
                             const float* scores, const int32_t* kept, double* logz_out,
                             double* logp_out, void* ws, size_t ws_bytes, void* hip_stream) {
  dc::LogzArgs z;
  const dc_status st =
      prep_logz(units, len, budget, tau, scores, kept, logz_out, logp_out, ws, ws_bytes, z);
  if (st != DC_OK) return st;
  if (!logz_out && !logp_out) return DC_OK;
  if (dc::launch_logz(z, hip_stream) != 0) return DC_ERR_HIP;
  return DC_OK;
}

size_t dc_subset_log_prob_workspace_bytes(int32_t units, int32_t len, int32_t budget) {
  if (units < 1 || len < 1 || budget < 1 || len > dc::evict_max_len() || units > (1 << 24)) return 0;
  return dc::logz_ws_bytes(units, len, budget);
}

dc_status dc_decode_evict(const dc_dims* dims, dc_kv* kv, dc_feat* feat, const dc_policy* policy,
                          int32_t budget, const void* q, const void* k_new, const void* v_new,
                          void* out, float* scores_out, int32_t* kept_out, void* ws,
                          size_t ws_bytes, void* hip_stream) {
  if (!feat) return DC_ERR_NULL;
  dc::DecodeArgs a;
  bool split = false;
  size_t need_d = 0, need_e = 0;
  dc_status st = prep_decode(dims, kv, feat, q, k_new, v_new, out, ws, ws_bytes, a, split, need_d);
  if (st != DC_OK) return st;
  dc::EvictArgs e;
  st = prep_evict(dims, kv, feat, policy, budget, scores_out, kept_out, ws, ws_bytes, a.L, a.T, e,
                  need_e);
  if (st != DC_OK) return st;
  const int G = group_of(dims), D = dims->head_dim;
  const int nm = e.evict ? (a.L - e.budget < e.budget ? a.L - e.budget : e.budget) : 0;
  // the single-launch step serves the four-input one-hidden-layer policy
  // without LayerNorm and does not produce sigma
  const bool fused = dims->dtype == DC_BF16 && !split && !e.ext && !feat->sigma &&
                     dc::step_fits(a.L, G, D, true, nm);
  if (fused) {
    if (dc::launch_step(a, &e, D, G, true, false, hip_stream) != 0) return DC_ERR_HIP;
  } else {
    st = launch_decode_any(dims, a, true, split, hip_stream);
    if (st != DC_OK) return st;
    if (ragged_after_decode(kv, a, hip_stream) != DC_OK) return DC_ERR_HIP;
    if (dc::launch_evict(e, dims->dtype, D, hip_stream) != 0) return DC_ERR_HIP;
  }
  if (ragged_after_evict(kv, e, nullptr, e.budget, hip_stream) != DC_OK) return DC_ERR_HIP;
  commit_decode(kv, feat, a, dims->ent_window);
  kv->len = e.budget;
  return DC_OK;
}

size_t dc_global_alpha_workspace_bytes(const dc_dims* dims, int32_t positions) {
  if (!dims || dims->batch < 1 || dims->n_layers < 1 || dims->n_kv_heads < 1 || positions < 1)
    return 0;
  // the sums, then every unit group's partial sums
  const size_t groups = (size_t)dc::global_alpha_groups(dims->n_layers * dims->n_kv_heads);
  return align256((size_t)dims->batch * (size_t)positions * (1 + groups) * sizeof(uint64_t));
}

dc_status dc_global_alpha(const dc_dims* dims, const dc_kv* kv, dc_feat* feat, void* ws,
                          size_t ws_bytes, void* hip_stream) {
  dc_status st = check_dims(dims);
  if (st != DC_OK) return st;
  if (!kv || !feat || !feat->alpha || !feat->pos) return DC_ERR_NULL;
  if (kv->len < 1 || kv->len > dims->capacity || feat->next_pos < 1) return DC_ERR_SHAPE;
  const int per_seq = dims->n_layers * dims->n_kv_heads;
  if (feat->alpha_recent != 1 || per_seq > 2048) return DC_ERR_UNSUPPORTED;
  const size_t need = dc_global_alpha_workspace_bytes(dims, feat->next_pos);
  if (!ws || ws_bytes < need) return DC_ERR_WORKSPACE;
  dc::GlobalAlphaArgs a;
  a.alpha = feat->alpha;
  a.pos = feat->pos;
  a.unit_len = kv->unit_len;
  a.acc = (uint64_t*)ws;
  a.cap = dims->capacity;
  a.units = (int)units_of(dims);
  a.len = kv->len;
  a.per_seq = per_seq;
  a.T = feat->next_pos;
  a.y0 = 0;
  return dc::launch_global_alpha(a, hip_stream) == 0 ? DC_OK : DC_ERR_HIP;
}

dc_status dc_kl_reward(int32_t rows, int32_t hidden, int32_t vocab, const void* h_full,
                       const void* h_comp, const void* w_lm, float* kl_out, void* ws,
                       size_t ws_bytes, void* hip_stream) {
  const dc_status st = kl_check(rows, hidden, vocab, h_full, h_comp, w_lm, kl_out);
  if (st != DC_OK) return st;
  if (!ws || ws_bytes < kl_bytes(rows, vocab)) return DC_ERR_WORKSPACE;
  return kl_launch(rows, hidden, vocab, h_full, h_comp, w_lm, kl_out, (float*)ws, hip_stream);
}

dc_status dc_kl_pack_lm_head(int32_t hidden, int32_t vocab, const void* w_lm, void* w_packed,
                             void* hip_stream) {
  if (!w_lm || !w_packed) return DC_ERR_NULL;
  if (hidden < 1 || vocab < 1) return DC_ERR_SHAPE;
  if (hidden % 128 || vocab % dc::kl_tile_cols()) return DC_ERR_UNSUPPORTED;
  const size_t bytes = (size_t)hidden * (size_t)vocab * 2;
  const uintptr_t s = (uintptr_t)w_lm, d = (uintptr_t)w_packed;
  if (s < d + bytes && d < s + bytes) return DC_ERR_UNSUPPORTED;    // in place / overlapping
  return dc::launch_kl_pack(w_lm, w_packed, hidden, vocab, hip_stream) == 0 ? DC_OK : DC_ERR_HIP;
}

dc_status dc_kl_reward_packed(int32_t rows, int32_t hidden, int32_t vocab, const void* h_full,
                              const void* h_comp, const void* w_packed, float* kl_out, void* ws,
                              size_t ws_bytes, void* hip_stream) {
  const dc_status st = kl_check(rows, hidden, vocab, h_full, h_comp, w_packed, kl_out);
  if (st != DC_OK) return st;
  if (!ws || ws_bytes < kl_bytes(rows, vocab)) return DC_ERR_WORKSPACE;
  return kl_launch(rows, hidden, vocab, h_full, h_comp, w_packed, kl_out, (float*)ws, hip_stream,
                   true);
}

dc_status dc_kl_reward_static(int32_t rows, int32_t hidden, int32_t vocab, const void* h_full,
                              const void* h_comp, const void* w_lm, float* kl_out,
                              void* hip_stream) {
  const dc_status st = kl_check(rows, hidden, vocab, h_full, h_comp, w_lm, kl_out);
  if (st != DC_OK) return st;
  if ((size_t)rows * (size_t)(vocab / dc::kl_tile_cols()) > (size_t)DC_KL_STATIC_MAX_PAIRS)
    return DC_ERR_SCRATCH;
  float* part = nullptr;
  if (dc::kl_static_scratch(&part) != 0 || !part) return DC_ERR_HIP;
  return kl_launch(rows, hidden, vocab, h_full, h_comp, w_lm, kl_out, part, hip_stream);
}

}  // extern "C"
