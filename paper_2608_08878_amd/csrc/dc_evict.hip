// Policy scoring, top-B selection and in-place compaction (gfx950).
//
// Per unit (Algorithm 1: scores, argtop_B, prune):
//   x_i = [alpha_i, ||v_i||_2, H_i = num_i / den_i (0 if den_i = 0), pos_i / T]
//   s_i = f_phi(x_i)                                   (ReLU MLP, float32)
//   keep the `budget` rows that rank highest under (s desc, pos asc)
// In training mode (Sec. 3.1.2, App. C) the ranking score is the
// Gumbel-perturbed s_i / tau + g_i instead; scores_out still receives s_i.
// Ranking uses one unsigned 64-bit key per row: the order-preserving image of
// the float32 score in the high word (-0 -> +0, NaN lowest) and ~pos in the low
// word, so keys are unique and "keep the top B" is "drop the E = L - B smallest
// keys".  E = 1 (the steady decode step) is a block-wide min; larger E uses an
// MSB-first radix select with 8-bit digits and an LDS histogram.
//
// Compaction moves the fewest rows: kept rows below `budget` stay, evicted slots
// below `budget` (holes, ascending) receive the kept rows from slots >= budget
// (ascending).  Sources and destinations are disjoint, so the copies need no
// ordering.
#include "dc_mlp.hpp"
#include "dc_select.hpp"

#pragma clang fp contract(off)

namespace dc {

// Caches up to NT * KPT rows: scores in registers, one workgroup of NT
// threads per unit.  Up to 4608 rows (the steady step of a 4096-row budget
// and more) 512 threads of 9 rows, two workgroups per CU, so one unit's
// scoring overlaps another's selection; up to 8192 rows 1024 threads of 8.
template <int DTYPE, int D, int NT, int KPT>
__global__ void __launch_bounds__(NT, 4) score_select_kernel(EvictArgs a) {
  extern __shared__ int dyn[];
  __shared__ SelShared sh;
  const int u = blockIdx.x, tid = threadIdx.x, wave = tid >> 6;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  const int L = a.L;
  const int kact = L > wave * 64 ? (L - wave * 64 + NT - 1) / NT : 0;
  float x[KPT][4];
  int32_t pk[KPT];
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    if (k < kact) {
      const int r = k * NT + tid;
      load_features(a, ub + (r < L ? r : L - 1), invT, x[k], pk[k]);
    }
  }
  float sc[KPT];
  policy_scores<KPT>(a, x, sc, kact);
  RegKeys<KPT> keys;
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const int r = k * NT + tid;
    keys.key[k] = ~0ull;
    if (k < kact && r < L) {
      if (a.scores_out) a.scores_out[(size_t)u * L + r] = sc[k];
      keys.key[k] = row_key(a.sample ? sampled_score(a, sc[k], pk[k], u) : sc[k], pk[k]);
    }
  }
  if (!a.evict) {
    if (a.kept_out)
      for (int r = tid; r < L; r += NT) a.kept_out[(size_t)u * L + r] = r;
    return;
  }
  select_compact<RegKeys<KPT>, DTYPE, D, NT, 2, true>(a, u, a.L, a.budget, keys, KPT, sh, dyn);
}

// Long caches: scores to keys in the workspace (grid over rows) ...
__global__ void __launch_bounds__(256) score_kernel(EvictArgs a, uint64_t* keys, int kstride) {
  const int u = a.y0 + blockIdx.y;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  const int L = unit_rows(a, u);
  if (L <= a.fused_rows) return;                         // served by the single-launch step
  if (!a.scores_out && unit_budget(a, u) >= L) return;   // a unit that keeps every row reads no key
  for (int base = blockIdx.x * 256; base < L; base += gridDim.x * 256) {
    const int r = base + threadIdx.x;
    float x[1][4];
    int32_t p;
    load_features(a, ub + (r < L ? r : L - 1), invT, x[0], p);
    float sc[1];
    policy_scores<1>(a, x, sc, 1);
    if (r < L) {
      if (a.scores_out) a.scores_out[(size_t)u * a.L + r] = sc[0];
      keys[(size_t)u * kstride + r] = row_key(a.sample ? sampled_score(a, sc[0], p, u) : sc[0], p);
    }
  }
}

// Extended one-hidden-layer policies: the same grid over rows, the out-of-line
// MLP per row.
__global__ void __launch_bounds__(256) score_ext_kernel(EvictArgs a, uint64_t* keys, int kstride) {
  const int u = a.y0 + blockIdx.y;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  const int L = unit_rows(a, u);
  if (L <= a.fused_rows) return;                         // served by the single-launch step
  if (!a.scores_out && unit_budget(a, u) >= L) return;   // a unit that keeps every row reads no key
  for (int base = blockIdx.x * 256; base < L; base += gridDim.x * 256) {
    const int r = base + threadIdx.x;
    if (r < L) {
      int32_t p;
      const float sc = ext_score(a, ub + r, invT, p);
      if (a.scores_out) a.scores_out[(size_t)u * a.L + r] = sc;
      keys[(size_t)u * kstride + r] = row_key(a.sample ? sampled_score(a, sc, p, u) : sc, p);
    }
  }
}

// ... then one workgroup per unit selects and compacts.  512 threads (several
// units per CU, so one unit's selection overlaps another's moves) unless a
// unit moves 4096 rows or more, where 1024 threads move them faster.
// Measured: workload 4's block eviction (1024 units, 64 moves) 67 -> 45 us and
// its compression (3277 moves) 1086 -> 1030 us with 512 threads; workload 3's
// compression (4096 units, 4096 moves) 3.13-3.16 ms with 1024 against 3.22 ms.
template <int DTYPE, int D, int NT>
__global__ void __launch_bounds__(NT, 4) select_kernel(EvictArgs a, const uint64_t* keys, int kstride) {
  extern __shared__ int dyn[];
  __shared__ SelShared sh;
  const int u = blockIdx.x;
  const int L = unit_rows(a, u);
  if (L <= a.fused_rows) return;        // served by the single-launch step
  const int Bu = unit_budget(a, u);
  if (Bu >= L) {                        // (per-unit budgets) this unit keeps every row
    if (a.kept_out)
      for (int r = threadIdx.x; r < a.ld_kept; r += NT) a.kept_out[(size_t)u * a.ld_kept + r] = r < L ? r : -1;
    return;
  }
  MemKeys mk{keys + (size_t)u * kstride};
  select_compact<MemKeys, DTYPE, D, NT, 2, true>(a, u, L, Bu, mk, (L + NT - 1) / NT, sh, dyn);
  if (a.kept_out && a.budgets)          // slots past this unit's budget
    for (int r = Bu + threadIdx.x; r < a.ld_kept; r += NT) a.kept_out[(size_t)u * a.ld_kept + r] = -1;
}

__global__ void identity_kept_kernel(int32_t* kept, int units, int L) {
  const size_t n = (size_t)units * L;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    kept[i] = (int32_t)(i % L);
}

int evict_max_len() { return MAX_LEN; }

template <int DTYPE, int D>
static int launch_evict_t(const EvictArgs& a, uint64_t* ws_keys, hipStream_t s) {
  const bool rg = a.unit_len || a.budgets;
  if (!a.evict && !rg && !a.scores_out && !a.kept_out) return 0;
  // moves: min(L - B, B); per-unit budgets: at most min(L / 2, the largest budget)
  const int E = a.L - a.budget;
  const int nmv = rg ? (a.L / 2 < a.budget ? a.L / 2 : a.budget) : a.evict ? (E < a.budget ? E : a.budget) : 0;
  EvictArgs b = a;
  b.mv_ints = (2 * (nmv > 0 ? nmv : 1) + 3) / 4 * 4;
  const size_t dyn = (size_t)b.mv_ints * sizeof(int);
  const int kstride = (a.L + ENT - 1) / ENT * ENT;
  const bool ragged = a.unit_len || a.budgets;
  if (!a.ext && !ragged && a.L <= ENT * REG_KPT) {
    // the one-hidden-layer policy on a short cache: scores in registers
    const bool half = a.L <= 512 * 9;
    auto k = half ? score_select_kernel<DTYPE, D, 512, 9> : score_select_kernel<DTYPE, D, ENT, REG_KPT>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    hipLaunchKernelGGL(k, dim3(a.units), dim3(half ? 512 : ENT), dyn, s, b);
    return (int)hipGetLastError();
  }
  // scores to row keys in the workspace (grid over rows), then one select per
  // unit (with per-unit lengths or budgets each unit decides whether it evicts)
  if (a.ext && a.nh == 2) {
    const int rc = launch_score_mlp2(b, ws_keys, kstride, s);
    if (rc) return rc;
  } else {
    for_grid_y(a.units, [&](int y0, int ny) {
      EvictArgs c = b;
      c.y0 = y0;
      // a quarter of the 256-row blocks, each workgroup striding over up to
      // four: ragged caches leave most workgroups of the longest unit's grid
      // idle otherwise, and uniform ones launch a quarter of the workgroups
      // (workload 3's compression step, 4096 units of 16385 rows: 784-832 ->
      // 746-750 us)
      const dim3 grid((a.L + 1023) / 1024, ny);
      if (a.ext) hipLaunchKernelGGL(score_ext_kernel, grid, dim3(256), 0, s, c, ws_keys, kstride);
      else hipLaunchKernelGGL(score_kernel, grid, dim3(256), 0, s, c, ws_keys, kstride);
    });
  }
  if (a.evict || ragged) {
    const bool wide = nmv >= 4096;
    auto k = wide ? select_kernel<DTYPE, D, ENT> : select_kernel<DTYPE, D, 512>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    hipLaunchKernelGGL(k, dim3(a.units), dim3(wide ? ENT : 512), dyn, s, b, (const uint64_t*)ws_keys,
                       kstride);
  } else if (a.kept_out) {
    hipLaunchKernelGGL(identity_kept_kernel, dim3(1024), dim3(256), 0, s, a.kept_out, a.units, a.L);
  }
  return (int)hipGetLastError();
}

int launch_evict(const EvictArgs& a, int dtype, int D, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (dtype == 1 && D == 128) return launch_evict_t<1, 128>(a, a.ws_keys, s);
  if (dtype == 1 && D == 64) return launch_evict_t<1, 64>(a, a.ws_keys, s);
  if (dtype == 0 && D == 128) return launch_evict_t<0, 128>(a, a.ws_keys, s);
  if (dtype == 0 && D == 64) return launch_evict_t<0, 64>(a, a.ws_keys, s);
  return (int)hipErrorInvalidValue;
}

size_t evict_ext_ws_bytes(int units, int L) {
  const size_t kstride = (size_t)(L + ENT - 1) / ENT * ENT;
  return (size_t)units * kstride * sizeof(uint64_t);
}

size_t evict_ws_bytes(int units, int L) {
  if (L <= ENT * REG_KPT) return 0;
  const size_t kstride = (size_t)(L + ENT - 1) / ENT * ENT;
  return (size_t)units * kstride * sizeof(uint64_t);
}

}  // namespace dc
