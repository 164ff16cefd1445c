/*
 * distillcache.h — C ABI of the DistillCache budgeted decode step for AMD
 * Instinct MI355X (gfx950).
 *
 * The method (DistillCache: KL-guided adaptive KV-cache eviction) keeps, at
 * every decode step, a subset C'_t of the cache C_t with |C'_t| <= B (problem
 * formulation, Sec. 3.1).  One step (Algorithm 1, "DistillCache Inference"):
 *   1. the forward pass appends the new key/value pair and attends over the
 *      cache that now contains it;
 *   2. per-token features x_i are built from that step's attention and the
 *      cache (state space, Sec. 3.1.1);
 *   3. a small MLP scores every cached token, s_i = f_phi(x_i) (Sec. 3.1.2);
 *   4. the top-B tokens are kept and the pruned cache serves the next step.
 * Training adds the per-step reward R_t = -KL(P_t || P^_t) between the
 * full-cache (teacher) and pruned-cache (student) next-token distributions
 * (reward, Sec. 3.1.4; teacher/student caches, Sec. 3.1.3).
 *
 * Terms used below
 *   unit   one (batch b, layer l, KV head g) cache; units are numbered
 *          u = (b * n_layers + l) * n_kv_heads + g and are fully independent.
 *   G      n_q_heads / n_kv_heads query heads per unit (grouped-query
 *          attention); query head h = g * G + j, j < G, reads KV head g.
 *   T      tokens seen so far; a token's position p is its 0-based index.
 *
 * Conventions for every entry point
 *   - Pointers are DEVICE memory owned by the caller unless marked "host".
 *     The library allocates and frees nothing; scratch comes from the
 *     caller's workspace (dc_workspace_bytes).
 *   - Arguments are validated on the host before any launch; an invalid call
 *     returns an error status and leaves every buffer and host field untouched.
 *   - Work is enqueued on the given HIP stream (NULL = default stream) and is
 *     asynchronous; outputs are valid once the stream reaches that point.  A
 *     failed launch returns DC_ERR_HIP.
 *   - Host bookkeeping fields (dc_kv.len, dc_feat.step/next_pos/ring_pmax) are
 *     updated at enqueue time; nothing is read back from the device.
 *   - Results are deterministic: the same inputs give the same bits (no
 *     floating-point atomics).
 *   - Calls on the same buffers must be ordered on one stream; calls on
 *     disjoint buffers and workspaces may run concurrently.
 */
#ifndef DISTILLCACHE_H
#define DISTILLCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DC_OK = 0,
  DC_ERR_NULL = 1,         /* a required pointer is NULL */
  DC_ERR_SHAPE = 2,        /* inconsistent sizes (e.g. len > capacity, empty cache) */
  DC_ERR_UNSUPPORTED = 3,  /* valid but not implemented (head_dim, G, len limits) */
  DC_ERR_CAPACITY = 4,     /* appending would exceed the capacity */
  DC_ERR_BUDGET = 5,       /* budget < 1 */
  DC_ERR_WORKSPACE = 6,    /* workspace missing or smaller than dc_workspace_bytes */
  DC_ERR_HIP = 7,          /* a HIP launch failed */
  DC_ERR_VALUE = 8,        /* a scalar argument out of range (temperature not finite and > 0) */
  DC_ERR_SCRATCH = 9       /* larger than the fixed scratch of an allocation-free entry point */
} dc_status;

typedef enum { DC_F32 = 0, DC_BF16 = 1 } dc_dtype;

#define DC_MAX_WINDOW 64

/* Shapes.  Supported: head_dim in {64, 128}; G = n_q_heads / n_kv_heads in
 * {1, 2, 4, 8}; dtype DC_F32 or DC_BF16. */
typedef struct {
  int32_t batch, n_layers, n_q_heads, n_kv_heads, head_dim;
  int32_t capacity;    /* rows allocated per unit in every per-row buffer */
  int32_t dtype;       /* dc_dtype of q, k, v, out and the query ring */
  int32_t ent_window;  /* entropy window w in decode steps, 1..64; 0 = unbounded */
  float scale;         /* logit scale; 0 selects 1/sqrt(head_dim) */
} dc_dims;

/* The student (or teacher) KV cache C_t.  Row i < len of unit u lives at
 * k[(u * capacity + i) * head_dim ...], likewise v.  Slot order is not token
 * order: eviction fills holes (see dc_score_evict). */
typedef struct {
  void *k, *v;         /* [units][capacity][head_dim], dtype */
  int32_t len;         /* host: valid rows per unit (identical for all units); with unit_len,
                          an upper bound of every unit's rows */
  int32_t *unit_len;   /* device [units] or NULL.  When present the cache is ragged: unit u
                          holds unit_len[u] rows (1 <= unit_len[u] <= len; kernels clamp
                          to that range).  Every entry point keeps it current (+1 per
                          append, min(rows, budget) per eviction) on the stream, and len
                          as the bound.  Ragged caches need bf16 and run the chunked
                          decode kernels and the row-key selection (no single-launch
                          step), with dc_workspace_bytes scratch. */
} dc_kv;

/* Per-token feature state of the student cache (Sec. 3.1.1, state space).
 * The feature vector is x_i = [alpha_i, ||v_i||_2, H_i, pos_i], or with a
 * five-input policy the paper's full [alpha_i, ||v_i||_2, sigma_i, H_i, pos_i]:
 *   alpha_i  attention mass token i received, averaged over the G query heads
 *            of its unit and accumulated over decode steps;
 *   H_i      = ent_num_i / ent_den_i (0 when ent_den_i = 0), where over the
 *            queries q of the last w steps (each (step, query head) pair)
 *            ent_den_i = sum_q a_q(i) and ent_num_i = sum_q a_q(i) H(a_q),
 *            H(a) = -sum a ln a the entropy of the query's attention;
 *   pos_i    = pos[i] / T;
 *   sigma_i  variance over the G query heads of the attention weight token i
 *            received at the last decode step, (1/G) sum_j (a_j(i) - mean_j a_j(i))^2
 *            (population variance; 0 when G = 1).
 * Row arrays are [units][capacity] and follow the K/V slots.  The query ring
 * keeps, for each of the last w steps (slot = step mod w), the G queries and
 * their softmax statistics so that the contribution of step t - w can be
 * recomputed and removed from ent_num/ent_den at step t. */
typedef struct {
  float   *alpha;      /* [units][capacity] */
  double  *ent_num;    /* [units][capacity] */
  double  *ent_den;    /* [units][capacity] */
  int32_t *pos;        /* [units][capacity] absolute position of the token in the slot */
  float   *vnorm;      /* [units][capacity] ||v_i||_2, set when the row is appended (or by
                          dc_feat_init) and carried with the row */
  void    *qring;      /* [units][w][G][head_dim], dtype: queries of the last w steps */
  float   *qstat;      /* [units][w][G][3]: (m, 1/l, H) of each query, where
                          m = max_i s_i, l = sum_i exp(s_i - m), s_i = scale * q.k_i */
  int32_t step;        /* host: decode steps done since the state was initialised */
  int32_t next_pos;    /* host: T, the position the next appended token receives */
  int32_t ring_pmax[DC_MAX_WINDOW]; /* host: per ring slot, largest position present (T - 1) */
  float   *sigma;      /* [units][capacity] sigma_i of the last step, or NULL; written by
                          every decode step and dc_feat_init (0) when present, moved by
                          eviction; required by five-input policies */
  int32_t alpha_recent; /* 0: alpha accumulates over steps (cumulative attention);
                          1: every decode step replaces alpha by that step's mass (the
                          paper's "most recent forward pass"; see dc_global_alpha) */
} dc_feat;

/* Policy MLP f_phi (Sec. 3.1.2; a small ReLU MLP per App. D).  params is a
 * packed float32 blob, row-major, per hidden layer l (width h_l, input width
 * h_{l-1}, h_0 = n_in):
 *   W_l[h_l][h_{l-1}], b_l[h_l], (gain_l[h_l], bias_l[h_l] if layer_norm)
 * followed by w_out[h_last], b_out.  Each hidden layer computes z = W h + b,
 * then, with layer_norm, z = gain (z - mean z) / sqrt(var z + 1e-5) + bias over
 * the layer's units (population variance), then h = relu(z); s = w_out . h + b_out.
 * Inputs: n_in = 4 takes [alpha, ||v||, H, pos/T]; n_in = 5 takes the paper's
 * [alpha, ||v||, sigma, H, pos/T] and needs dc_feat.sigma.
 * Supported: n_in in {4, 5}, n_hidden_layers in {1, 2}, hidden widths 1..128.
 * The four-input one-hidden-layer policy without layer_norm runs inside the
 * fused decode step; every other policy runs in a separate scoring pass (two
 * hidden layers on the matrix cores) that ranks through row keys in the
 * workspace, so it needs dc_workspace_bytes scratch at any length. */
typedef struct {
  int32_t n_in;
  int32_t n_hidden_layers;
  int32_t hidden[2];
  const float *params;  /* device */
  int32_t layer_norm;   /* 0 or 1 */
} dc_policy;

/* Bytes of caller workspace the entry points need for caches of up to max_len
 * rows per unit (dc_decode_step, dc_score_evict with any policy) and for a KL reward over
 * kl_rows rows of a kl_vocab-entry vocabulary (dc_kl_reward).  Pass 0 for the
 * parts not used.  Returns 0 for invalid dims. */
size_t dc_workspace_bytes(const dc_dims *dims, int32_t max_len, int32_t kl_rows, int32_t kl_vocab);

/* Initialise the feature state of a cache holding kv->len rows per unit whose
 * slot i holds the token at position first_pos + i (a freshly filled cache):
 * alpha = ent_num = ent_den = 0, pos, vnorm from the value rows; host fields
 * step = 0, next_pos = first_pos + kv->len. */
dc_status dc_feat_init(const dc_dims *dims, const dc_kv *kv, dc_feat *feat, int32_t first_pos,
                       void *hip_stream);

/* One decode-step forward over every unit (Algorithm 1, forward pass and
 * feature extraction; Sec. 3.1.1).
 *   q      [batch][n_layers][n_q_heads][head_dim], dtype
 *   k_new, v_new  [batch][n_layers][n_kv_heads][head_dim], dtype, or both NULL
 *          for no append.  The pair is written to slot len, its features are
 *          zeroed, pos = T, then len += 1 and T += 1 (host fields).
 *   out    [batch][n_layers][n_q_heads][head_dim], dtype: o_j = sum_i a_{j,i} v_i
 *          over the len rows (after the append), a_j = softmax_i(scale q_j.k_i).
 *   feat   NULL => plain attention (the never-pruned teacher cache of
 *          Sec. 3.1.3); otherwise alpha += (1/G) sum_j a_j(i), this step's
 *          queries enter the entropy window, step t - w leaves it, vnorm is
 *          rewritten, the ring slot (step mod w) is overwritten, step += 1.
 * Workspace: dc_workspace_bytes(dims, len + appended, 0, 0) bytes whenever feat is
 * not NULL (per-row scratch between the key and feature passes), and for
 * plain attention over caches longer than fit on chip.
 * Errors: DC_ERR_NULL, DC_ERR_SHAPE (len == 0 without append, len > capacity),
 * DC_ERR_CAPACITY (len + 1 > capacity), DC_ERR_UNSUPPORTED, DC_ERR_WORKSPACE. */
dc_status dc_decode_step(const dc_dims *dims, dc_kv *kv, dc_feat *feat, const void *q,
                         const void *k_new, const void *v_new, void *out, void *ws,
                         size_t ws_bytes, void *hip_stream);

/* Score every cached token with the policy and keep the top `budget` per unit
 * (Algorithm 1 scoring, argtop_B and prune; Sec. 3.1.2 deterministic top-B).
 * Order: higher score first; equal scores keep the earlier token (smaller
 * pos); -0 equals +0; NaN ranks below every number.  If budget >= len nothing
 * moves.  Otherwise the kept rows end in slots 0..budget-1: a kept row already
 * there stays in place, and the evicted slots below budget ("holes", in
 * ascending order) receive the kept rows from slots >= budget (ascending),
 * carrying k, v, alpha, ent_num, ent_den, pos and vnorm.  len = budget (host).
 *   scores_out  [units][len] float32 scores in pre-eviction slot order, or NULL.
 *   kept_out    [units][min(budget, len)] int32: pre-eviction slot of the row
 *               that ends in each slot, or NULL.
 * Errors: DC_ERR_NULL, DC_ERR_BUDGET (budget < 1), DC_ERR_UNSUPPORTED (policy
 * shape, len > 40960), DC_ERR_SHAPE, DC_ERR_WORKSPACE (dc_workspace_bytes
 * scratch is needed for len > 8192, ragged caches and every policy but the
 * four-input one-hidden-layer one without layer_norm). */
dc_status dc_score_evict(const dc_dims *dims, dc_kv *kv, dc_feat *feat, const dc_policy *policy,
                         int32_t budget, float *scores_out, int32_t *kept_out, void *ws,
                         size_t ws_bytes, void *hip_stream);

/* One whole decode step (Algorithm 1): dc_decode_step followed by
 * dc_score_evict with the same policy, budget and outputs.  Results and host
 * bookkeeping are bit-identical to the two calls in sequence; where the cache
 * fits on chip (bf16, up to about 5000 rows per unit) it runs as a single
 * launch that streams K/V once and compacts before it exits.
 *   scores_out  [units][len + appended] float32 or NULL (pre-eviction slot order)
 *   kept_out    [units][min(budget, len + appended)] int32 or NULL
 * Errors: those of dc_decode_step and dc_score_evict (feat must not be NULL);
 * nothing is enqueued unless both validate.  Workspace: dc_workspace_bytes for
 * the post-append length. */
dc_status dc_decode_evict(const dc_dims *dims, dc_kv *kv, dc_feat *feat, const dc_policy *policy,
                          int32_t budget, const void *q, const void *k_new, const void *v_new,
                          void *out, float *scores_out, int32_t *kept_out, void *ws,
                          size_t ws_bytes, void *hip_stream);

/* Gumbel noise of the training-mode selection (Sec. 3.1.2: during training the
 * ranking is sampled by perturbing every score with an independent standard
 * Gumbel draw; App. C adds the temperature tau).  The draw of the token at
 * position p in unit u is a pure function of (seed, draw, u, p):
 *   x = first output word of Philox4x32-10 (Salmon et al., SC'11) with
 *       counter (p, u, draw, 0) and key (seed[0], seed[1]),
 *   U = (2 (x >> 9) + 1) 2^-24   (exact in float32, 0 < U < 1),
 *   g = -ln(-ln U). */
typedef struct {
  float tau;           /* temperature, finite and > 0 */
  uint32_t seed[2];    /* Philox key: low and high word of a 64-bit seed */
  uint32_t draw;       /* draw number: use a new value for every sampling call on a cache */
} dc_gumbel;

/* Training-mode scoring and selection (Sec. 3.1.2 stochastic ranking, App. C).
 * As dc_score_evict, except that rows are ranked by the perturbed score
 *   s~_i = s_i / tau + g_i           (float32; same tie rule and compaction)
 * with g_i from `gumbel`; scores_out still receives the unperturbed s_i.  If
 * logp_out is not NULL it receives, per unit, the log-probability of the kept
 * set a under App. C's subset law,
 *   logp_out[u] = sum_{i in a} s_i / tau - log Z(s, budget, tau)
 * (see dc_subset_log_prob; 0 when budget >= len), which needs scores_out and
 * kept_out.  Workspace: as dc_score_evict (it also covers the log-partition).
 * Errors: those of dc_score_evict; DC_ERR_NULL (gumbel NULL, or logp_out
 * without scores_out and kept_out); DC_ERR_VALUE (tau). */
dc_status dc_sample_evict(const dc_dims *dims, dc_kv *kv, dc_feat *feat, const dc_policy *policy,
                          int32_t budget, const dc_gumbel *gumbel, float *scores_out,
                          int32_t *kept_out, double *logp_out, void *ws, size_t ws_bytes,
                          void *hip_stream);

/* Per-unit budgets (the appendix's head-level hybrid gives a subset of heads
 * their full cache and the policy's budget to the rest; Table "head-level
 * hybrid").  As dc_score_evict / dc_sample_evict with unit u
 * keeping the top budgets[u] of its rows:
 *   budgets     device [units]; each clamped to [1, max_budget]
 *   max_budget  host: the largest budget (>= 1)
 *   gumbel      NULL for the deterministic selection, else the training-mode
 *               ranking (and logp_out may be requested)
 *   scores_out  [units][kv->len] (rows past a unit's length untouched)
 *   kept_out    [units][min(max_budget, kv->len)]: pre-eviction slots of the
 *               rows that end in each slot, -1 past the unit's kept count
 *   logp_out    [units] log pi of each unit's kept set under its own budget
 * kv->unit_len is required (the units' lengths diverge); afterwards unit_len[u]
 * = min(rows, budget) and kv->len = min(kv->len, max_budget).  A unit whose
 * budget covers its rows keeps them all in place.
 * Errors: those of dc_score_evict; DC_ERR_NULL (budgets, kv->unit_len, logp_out
 * without gumbel, scores_out or kept_out), DC_ERR_BUDGET (max_budget < 1). */
dc_status dc_score_evict_units(const dc_dims *dims, dc_kv *kv, dc_feat *feat, const dc_policy *policy,
                               const int32_t *budgets, int32_t max_budget, const dc_gumbel *gumbel,
                               float *scores_out, int32_t *kept_out, double *logp_out, void *ws,
                               size_t ws_bytes, void *hip_stream);

/* One whole decode step of a ragged cache with per-unit budgets (the
 * appendix's head-level hybrid: a subset of KV heads keeps its full cache, the
 * others the policy's budget; Algorithm 1 per unit): dc_decode_step followed by
 * the deterministic dc_score_evict_units, with the same arguments and outputs
 * (scores_out [units][kv->len + 1], kept_out [units][min(max_budget,
 * kv->len + 1)], unit_len and host bookkeeping as after the two calls).  k_new
 * and v_new are required.  With the four-input one-hidden-layer policy
 * without LayerNorm, no sigma, bf16 and G >= 4, every unit whose rows after
 * the append fit on chip (at most a few thousand, two workgroups per CU) runs
 * the whole step in one launch (K/V read once, per-unit top-B and compaction
 * before the workgroup exits); longer units (the full-cache heads) take the
 * chunked decode and then their own scoring and selection.  Otherwise the call
 * is the two calls in sequence.  Results agree with the two calls to the
 * tolerances of the kernels (attention and features sum in a different order
 * on the two paths); the slot map follows the same rule.
 * Workspace: dc_workspace_bytes(dims, kv->len + 1, 0, 0).
 * Errors: those of dc_decode_step and dc_score_evict_units; DC_ERR_NULL also
 * for a missing append; nothing is enqueued unless both validate. */
dc_status dc_decode_evict_units(const dc_dims *dims, dc_kv *kv, dc_feat *feat,
                                const dc_policy *policy, const int32_t *budgets, int32_t max_budget,
                                const void *q, const void *k_new, const void *v_new, void *out,
                                float *scores_out, int32_t *kept_out, void *ws, size_t ws_bytes,
                                void *hip_stream);

/* One whole training-mode decode step: dc_decode_step followed by
 * dc_sample_evict with the same policy, budget, noise and outputs, with results
 * and host bookkeeping bit-identical to the two calls in sequence.  Where the
 * cache fits on chip (bf16, G >= 4, a four-input policy without LayerNorm) it
 * runs as one launch that streams K/V once, draws the noise, selects and
 * compacts, followed by the log-partition when logp_out is requested.
 * Errors: those of dc_decode_step and dc_sample_evict; nothing is enqueued
 * unless both validate. */
dc_status dc_decode_sample_evict(const dc_dims *dims, dc_kv *kv, dc_feat *feat,
                                 const dc_policy *policy, int32_t budget, const dc_gumbel *gumbel,
                                 const void *q, const void *k_new, const void *v_new, void *out,
                                 float *scores_out, int32_t *kept_out, double *logp_out, void *ws,
                                 size_t ws_bytes, void *hip_stream);

/* Exact log-partition function of the size-B subset law and the
 * log-probability of kept sets (App. C), for `units` independent score rows:
 *   logz_out[u] = log Z = log sum over size-budget subsets a of exp(sum_{i in a} s[u][i] / tau)
 *   logp_out[u] = sum_{i in kept[u]} s[u][i] / tau - logz_out[u]
 * When budget >= len the only subset is the whole row: log Z = sum_i s_i / tau
 * and logp = 0.
 *   scores    [units][len] float32
 *   kept      [units][min(budget, len)] int32 indices into the row (the
 *             kept_out layout of dc_score_evict); needed for logp_out only
 *   logz_out, logp_out  [units] float64; either may be NULL
 * Computed by an O(len K) recursion, K = min(budget, len - budget), exact up
 * to rounding: the relative error of Z stays below about (K + len) 2^-24.
 * Scores whose spread divided by tau exceeds about 11000 fall outside exact
 * coverage (the smallest weights are clamped); a non-finite score or a kept
 * index outside [0, len) gives NaN for that unit.
 * Workspace: dc_subset_log_prob_workspace_bytes(units, len, budget) bytes
 * (zero unless K > 4096).
 * Errors: DC_ERR_NULL (scores, or kept with logp_out), DC_ERR_SHAPE (units or
 * len < 1), DC_ERR_BUDGET, DC_ERR_VALUE (tau), DC_ERR_UNSUPPORTED (len > 40960,
 * units > 2^24), DC_ERR_WORKSPACE. */
dc_status dc_subset_log_prob(int32_t units, int32_t len, int32_t budget, float tau,
                             const float *scores, const int32_t *kept, double *logz_out,
                             double *logp_out, void *ws, size_t ws_bytes, void *hip_stream);

/* Workspace bytes of dc_subset_log_prob (0 for invalid sizes). */
size_t dc_subset_log_prob_workspace_bytes(int32_t units, int32_t len, int32_t budget);

/* The paper's alpha_i (Sec. 3.1.1, state space): the attention mass token i
 * received in the most recent forward pass, averaged over all heads and
 * layers.  With feat->alpha_recent = 1 every decode step leaves in alpha each
 * row's mass of that step averaged over the G query heads of its unit; this
 * call replaces it, for every row of every unit, by the mean over all units of
 * the same sequence (its n_layers x n_kv_heads KV units, which hold equally
 * many query heads) of those values at the row's position, a unit that no
 * longer holds the position counting 0.  Call it after dc_decode_step and
 * before dc_score_evict (dc_decode_evict scores inside the step, with each
 * unit's own recent mass).  The sums are 64-bit fixed point (2^-52 per unit
 * of alpha): integer sums do not depend on the order of their terms, so the
 * result is deterministic; alpha is clamped to [0, 1] first (recent masses lie
 * there).  Ragged caches are read through kv->unit_len.
 *   ws: dc_global_alpha_workspace_bytes(dims, feat->next_pos) bytes.
 * Errors: DC_ERR_NULL, DC_ERR_SHAPE (len outside 1..capacity, next_pos < 1),
 * DC_ERR_UNSUPPORTED (alpha_recent != 1, more than 2048 units per sequence),
 * DC_ERR_WORKSPACE. */
dc_status dc_global_alpha(const dc_dims *dims, const dc_kv *kv, dc_feat *feat, void *ws,
                          size_t ws_bytes, void *hip_stream);

/* Workspace bytes of dc_global_alpha for sequences of up to `positions` tokens
 * (0 for invalid sizes). */
size_t dc_global_alpha_workspace_bytes(const dc_dims *dims, int32_t positions);

/* Largest row count of one dc_kl_reward call. */
#define DC_KL_MAX_ROWS 16384

/* Per-step KL reward (Sec. 3.1.4): for each row r,
 *   kl_out[r] = KL(P || Q) = sum_v P_v (ln P_v - ln Q_v)   (nats),
 * P = softmax(h_full[r] W^T), Q = softmax(h_comp[r] W^T) over the whole vocab.
 *   h_full, h_comp  [rows][hidden] bfloat16
 *   w_lm            [vocab][hidden] bfloat16 (the lm-head weight)
 *   kl_out          [rows] float32; the reward is R = -kl_out.
 * Rows are independent, so a training loop may defer the rewards of a whole
 * rollout (steps x batch rows, the hidden states kept per step) to one call:
 * the lm head is then read once for all of them.
 * Supported: hidden % 128 == 0, vocab % 64 == 0, 1 <= rows <= DC_KL_MAX_ROWS.
 * Errors: DC_ERR_NULL, DC_ERR_SHAPE, DC_ERR_UNSUPPORTED, DC_ERR_WORKSPACE. */
dc_status dc_kl_reward(int32_t rows, int32_t hidden, int32_t vocab, const void *h_full,
                       const void *h_comp, const void *w_lm, float *kl_out, void *ws,
                       size_t ws_bytes, void *hip_stream);

/* Lays the lm-head weight out for dc_kl_reward_packed (the weight of the
 * Sec. 3.1.4 reward's output distribution; a once-per-model copy, not a
 * per-step operation):
 *   w_lm      [vocab][hidden] bfloat16, as for dc_kl_reward (read only)
 *   w_packed  vocab * hidden bfloat16 (caller-allocated, the same size as
 *             w_lm, not overlapping it), written as 64 x 64 blocks: block
 *             (t, k) holds vocabulary rows 64 t .. 64 t + 63, hidden elements
 *             64 k .. 64 k + 63, row-major (128 bytes per row), at element
 *             offset (t * (hidden / 64) + k) * 4096.
 * The packed weight is read as one contiguous run per vocabulary tile, which
 * the per-step (few-row) reward streams faster than 64 rows of the row-major
 * weight; the values and the results are the same.  Asynchronous on
 * hip_stream.
 * Supported: hidden % 128 == 0, vocab % 64 == 0.
 * Errors: DC_ERR_NULL, DC_ERR_SHAPE (hidden or vocab < 1), DC_ERR_UNSUPPORTED
 * (sizes, or w_packed overlapping w_lm), DC_ERR_HIP. */
dc_status dc_kl_pack_lm_head(int32_t hidden, int32_t vocab, const void *w_lm, void *w_packed,
                             void *hip_stream);

/* dc_kl_reward (Sec. 3.1.4) reading the lm head as dc_kl_pack_lm_head laid it
 * out.  Arguments, workspace (dc_workspace_bytes with kl_rows, kl_vocab),
 * limits and errors as dc_kl_reward; kl_out is bit-identical to
 * dc_kl_reward's on the row-major weight the packed one was made from. */
dc_status dc_kl_reward_packed(int32_t rows, int32_t hidden, int32_t vocab, const void *h_full,
                              const void *h_comp, const void *w_packed, float *kl_out, void *ws,
                              size_t ws_bytes, void *hip_stream);

/* Largest rows * (vocab / 64) of one dc_kl_reward_static call. */
#define DC_KL_STATIC_MAX_PAIRS 524288

/* dc_kl_reward without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, serving loops and harnesses that
 * forbid allocation).  Same arguments, kernels and result bits as
 * dc_kl_reward; the per-(row, 64-column tile) statistics go to a scratch array
 * of 16 * DC_KL_STATIC_MAX_PAIRS bytes (8 MiB) that the library holds on each
 * device it runs on until the process ends (e.g. 1024 rows of a
 * 32768-entry vocabulary).  The call allocates nothing.  Calls that overlap on
 * one device share that array and race: order them on one stream.  Every
 * entry a call reads is written earlier in the same call, so nothing left by
 * an earlier call is used.
 * Errors: those of dc_kl_reward except DC_ERR_WORKSPACE; DC_ERR_SCRATCH when
 * rows * (vocab / 64) > DC_KL_STATIC_MAX_PAIRS (checked before any device
 * work); DC_ERR_HIP when the scratch address cannot be obtained. */
dc_status dc_kl_reward_static(int32_t rows, int32_t hidden, int32_t vocab, const void *h_full,
                              const void *h_comp, const void *w_lm, float *kl_out,
                              void *hip_stream);

/* Dynamic budget (App. D, experimental protocol): the budget of a decode step
 * scales with the sequence, B_t = max(floor(ratio * seq_len), b_min).  The
 * paper writes the length as the cache size |C_t|, which would shrink the
 * budget geometrically once eviction starts; here seq_len is the number of
 * tokens seen (dc_feat.next_pos after the step's append).  The product is
 * formed in binary64 from the float32 ratio.  Host function: no device work.
 * Returns -1 unless 0 < ratio <= 1, seq_len >= 0 and b_min >= 1. */
int32_t dc_dynamic_budget(float ratio, int32_t seq_len, int32_t b_min);

/* Hyper-parameters of the REINFORCE update (Sec. 3.2; App. D gives gamma =
 * 0.99 and beta = 0.01). */
typedef struct {
  double gamma;       /* discount factor, 0 <= gamma <= 1 */
  double beta;        /* entropy regularisation coefficient, finite */
  double ema_decay;   /* decay d of the exponential-moving-average baseline, 0 <= d < 1 */
} dc_reinforce_cfg;

/* Rollout reward math of the REINFORCE update with entropy regularisation and
 * variance-reduction baselines (Sec. 3.2), for `steps` decode steps of
 * `rollouts` sampled rollouts.  All arrays are row-major [steps][rollouts]:
 *   rewards       float32 R[t][k] = -KL_t (dc_kl_reward)
 *   logp          float64 log pi(a_t | s_t) of the sampled kept sets
 *                 (dc_sample_evict, dc_subset_log_prob)
 *   returns_out   float64 G[t][k] = sum_{tau >= t} gamma^(tau - t) R[tau][k]   (required)
 *   baseline_out  float64 b[t][k]: the mean return of the other rollouts at step t
 *                 (leave-one-out, rollouts >= 2), else the EMA baseline      (or NULL)
 *   adv_out       float64 A = G - b                                          (or NULL)
 *   weight_out    float64 d loss / d log pi = -(A - beta) / (steps rollouts) (or NULL)
 *   stats_out     float64 [3]: loss = -mean(log pi A - beta log pi) (the
 *                 entropy term uses the single-sample surrogate -log pi), the
 *                 mean surrogate entropy, the mean return               (or NULL)
 *   ema           float64 [1], in/out: the EMA baseline e; after the call
 *                 e = d e + (1 - d) mean(G)
 * One small float64 kernel, deterministic.  Errors: DC_ERR_NULL, DC_ERR_SHAPE
 * (steps or rollouts < 1), DC_ERR_UNSUPPORTED (steps * rollouts > 2^26),
 * DC_ERR_VALUE (gamma, beta, ema_decay out of range). */
dc_status dc_reinforce_terms(int32_t steps, int32_t rollouts, const dc_reinforce_cfg *cfg,
                             const float *rewards, const double *logp, double *ema,
                             double *returns_out, double *baseline_out, double *adv_out,
                             double *weight_out, double *stats_out, void *hip_stream);

/* Static string naming a status. */
const char *dc_status_str(dc_status s);

#ifdef __cplusplus
}
#endif
#endif /* DISTILLCACHE_H */
