// Policy scoring, deterministic top-B selection and in-place compaction (gfx950).
//
// Per unit (Algorithm 1: scores, argtop_B, prune):
//   x_i = [alpha_i, ||v_i||_2, H_i = num_i / den_i (0 if den_i = 0), pos_i / T]
//   s_i = f_phi(x_i)                                   (ReLU MLP, float32)
//   keep the `budget` rows that rank highest under (s desc, pos asc)
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
#include "dc_device.hpp"
#include "dc_kernels.hpp"

#pragma clang fp contract(off)

namespace dc {

constexpr int ENT = 1024;            // threads of the per-unit select workgroup
constexpr int ENW = ENT / 64;
constexpr int REG_KPT = 8;           // rows per thread kept in registers (L <= 8192)
constexpr int MAX_LEN = 40960;
constexpr int MAX_H1_2L = 64;        // first hidden width supported with two hidden layers

__device__ __forceinline__ uint32_t score_key(float s) {
  uint32_t b = __float_as_uint(s);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return 0u;  // NaN ranks lowest
  if (b == 0x80000000u) b = 0u;                                           // -0 -> +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint64_t row_key(float s, int32_t pos) {
  return ((uint64_t)score_key(s) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)pos);
}

// Features of row gi.
__device__ __forceinline__ void load_features(const EvictArgs& a, size_t gi, float invT, float x[4],
                                              int32_t& p) {
  p = a.pos[gi];
  const double z = a.den[gi];
  x[0] = a.alpha[gi];
  x[1] = a.vnorm[gi];
  x[2] = z > 0.0 ? (float)(a.num[gi] / z) : 0.0f;
  x[3] = (float)p * invT;
}

// s = f_phi(x), float32, fixed evaluation order.
__device__ __forceinline__ float mlp1(const float* __restrict__ P, int h1, const float x[4]) {
  const float* W1 = P;
  const float* b1 = P + 4 * h1;
  const float* wo = b1 + h1;
  float out = wo[h1];
  for (int h = 0; h < h1; ++h) {
    float z = b1[h];
    z = __builtin_fmaf(W1[4 * h + 0], x[0], z);
    z = __builtin_fmaf(W1[4 * h + 1], x[1], z);
    z = __builtin_fmaf(W1[4 * h + 2], x[2], z);
    z = __builtin_fmaf(W1[4 * h + 3], x[3], z);
    out = __builtin_fmaf(wo[h], fmaxf(z, 0.0f), out);
  }
  return out;
}

__device__ __forceinline__ float mlp2(const float* __restrict__ P, int h1, int h2, const float x[4]) {
  const float* W1 = P;
  const float* b1 = P + 4 * h1;
  const float* W2 = b1 + h1;
  const float* b2 = W2 + h2 * h1;
  const float* wo = b2 + h2;
  float hv[MAX_H1_2L];
#pragma unroll
  for (int h = 0; h < MAX_H1_2L; ++h) {
    if (h < h1) {
      float z = b1[h];
      z = __builtin_fmaf(W1[4 * h + 0], x[0], z);
      z = __builtin_fmaf(W1[4 * h + 1], x[1], z);
      z = __builtin_fmaf(W1[4 * h + 2], x[2], z);
      z = __builtin_fmaf(W1[4 * h + 3], x[3], z);
      hv[h] = fmaxf(z, 0.0f);
    } else {
      hv[h] = 0.0f;
    }
  }
  float out = wo[h2];
  for (int o = 0; o < h2; ++o) {
    const float* w = W2 + o * h1;
    float z = b2[o];
#pragma unroll
    for (int h = 0; h < MAX_H1_2L; ++h)
      if (h < h1) z = __builtin_fmaf(w[h], hv[h], z);
    out = __builtin_fmaf(wo[o], fmaxf(z, 0.0f), out);
  }
  return out;
}

__device__ __forceinline__ float policy_score(const EvictArgs& a, const float x[4]) {
  return a.nh == 1 ? mlp1(a.params, a.h1, x) : mlp2(a.params, a.h1, a.h2, x);
}

// ---------------------------------------------------------------- key sources
// Keys of row r = k * ENT + tid live in registers (fused path) ...
template <int KPT>
struct RegKeys {
  static constexpr int KMAX = KPT;
  uint64_t key[KPT];
  __device__ uint64_t get(int k) const { return key[k]; }
};
// ... or in the workspace (long caches), written by score_kernel.
struct MemKeys {
  static constexpr int KMAX = MAX_LEN / ENT;
  const uint64_t* key;
  __device__ uint64_t get(int k) const { return key[k * ENT + threadIdx.x]; }
};

template <typename T>
__device__ __forceinline__ T wave_min(T x) {
  for (int off = 32; off > 0; off >>= 1) {
    T o = __shfl_xor(x, off);
    x = o < x ? o : x;
  }
  return x;
}

__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
  for (int off = 1; off < 64; off <<= 1) {
    int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

// Shared-memory layout of the select workgroup.
struct SelShared {
  uint64_t wmin[ENW];
  int hist[256];
  int sel[4];            // digit, count below, count in digit, done flag
  int wcnt[2][ENW];      // per-wave hole / mover counts
  int nmoves;
};

// Block exclusive scans of two flags over rows k*ENT + tid (one k at a time).
__device__ __forceinline__ void block_scan2(bool f0, bool f1, int& r0, int& r1, int& t0, int& t1,
                                            SelShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t b0 = __ballot(f0), b1 = __ballot(f1);
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int p0 = __popcll(b0 & below), p1 = __popcll(b1 & below);
  if (lane == 0) {
    sh.wcnt[0][wave] = __popcll(b0);
    sh.wcnt[1][wave] = __popcll(b1);
  }
  __syncthreads();
  int o0 = 0, o1 = 0;
  t0 = 0;
  t1 = 0;
  for (int w = 0; w < ENW; ++w) {
    if (w < wave) {
      o0 += sh.wcnt[0][w];
      o1 += sh.wcnt[1][w];
    }
    t0 += sh.wcnt[0][w];
    t1 += sh.wcnt[1][w];
  }
  __syncthreads();
  r0 = o0 + p0;
  r1 = o1 + p1;
}

// Select the E smallest keys and compact the unit.  `keys` holds the keys of
// rows k*ENT + tid for k < kpt (invalid rows beyond L are ignored).
template <typename Keys, int DTYPE, int D>
__device__ void select_compact(const EvictArgs& a, int u, const Keys& keys, int kpt, SelShared& sh,
                               int* mv) {
  constexpr int ELT = DTYPE == 0 ? 4 : 2;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = a.L, B = a.budget, E = L - B;
  const size_t ub = (size_t)u * a.cap;
  // threshold: evicted rows are those with key <= thr
  uint64_t thr;
  if (E == 1) {
    uint64_t m = ~0ull;
#pragma unroll
    for (int k = 0; k < Keys::KMAX; ++k) {
      if (k >= kpt) break;
      const int r = k * ENT + tid;
      if (r < L) {
        const uint64_t x = keys.get(k);
        m = x < m ? x : m;
      }
    }
    m = wave_min(m);
    if (lane == 0) sh.wmin[wave] = m;
    __syncthreads();
    thr = sh.wmin[0];
    for (int w = 1; w < ENW; ++w) thr = sh.wmin[w] < thr ? sh.wmin[w] : thr;
  } else {
    uint64_t prefix = 0;
    int need = E;
    int shift = 56;
    for (;; shift -= 8) {
      const uint64_t hmask = shift + 8 >= 64 ? 0ull : (~0ull << (shift + 8));
      for (int i = tid; i < 256; i += ENT) sh.hist[i] = 0;
      __syncthreads();
#pragma unroll
      for (int k = 0; k < Keys::KMAX; ++k) {
        if (k >= kpt) break;
        const int r = k * ENT + tid;
        if (r < L) {
          const uint64_t x = keys.get(k);
          if ((x & hmask) == prefix) atomicAdd(&sh.hist[(int)((x >> shift) & 255u)], 1);
        }
      }
      __syncthreads();
      if (wave == 0) {
        const int c0 = sh.hist[4 * lane], c1 = sh.hist[4 * lane + 1], c2 = sh.hist[4 * lane + 2],
                  c3 = sh.hist[4 * lane + 3];
        const int incl = wave_incl_scan(c0 + c1 + c2 + c3);
        int below = incl - (c0 + c1 + c2 + c3);
        const int cs[4] = {c0, c1, c2, c3};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (below < need && need <= below + cs[q]) {
            sh.sel[0] = 4 * lane + q;
            sh.sel[1] = below;
            sh.sel[2] = cs[q];
          }
          below += cs[q];
        }
      }
      __syncthreads();
      const int digit = sh.sel[0], cbelow = sh.sel[1], cin = sh.sel[2];
      __syncthreads();
      need -= cbelow;
      prefix |= (uint64_t)digit << shift;
      if (cin == need || shift == 0) break;
    }
    // evicted: (key >> shift) <= (prefix >> shift)
    thr = prefix | (shift ? ((1ull << shift) - 1) : 0ull);
  }
  // plan: holes (evicted, slot < B) take movers (kept, slot >= B) in order
  if (tid == 0) sh.nmoves = 0;
  int run0 = 0, run1 = 0;
#pragma unroll
  for (int k = 0; k < Keys::KMAX; ++k) {
    if (k >= kpt || k * ENT >= L) break;
    const int r = k * ENT + tid;
    bool ev = false;
    if (r < L) ev = keys.get(k) <= thr;
    const bool hole = r < B && ev;
    const bool mover = r >= B && r < L && !ev;
    int rk0, rk1, t0, t1;
    block_scan2(hole, mover, rk0, rk1, t0, t1, sh);
    if (hole) mv[2 * (run0 + rk0)] = r;
    if (mover) mv[2 * (run1 + rk1) + 1] = r;
    if (a.kept_out && r < B && !ev) a.kept_out[(size_t)u * B + r] = r;
    run0 += t0;
    run1 += t1;
  }
  __syncthreads();
  const int nm = run0;  // == run1
  // copy rows: one 16-lane group per move
  constexpr int N16 = D * ELT / 16;  // 16-byte chunks per row (8 or 16)
  const int grp = tid / 16, gl = tid % 16, ngrp = ENT / 16;
  for (int j = grp; j < nm; j += ngrp) {
    const int dst = mv[2 * j], src = mv[2 * j + 1];
    const size_t gd = ub + dst, gs = ub + src;
    char* kb = (char*)a.k;
    char* vb = (char*)a.v;
    for (int c = gl; c < N16; c += 16) {
      *reinterpret_cast<uint4*>(kb + gd * D * ELT + c * 16) = ldg16(kb + gs * D * ELT + c * 16);
      *reinterpret_cast<uint4*>(vb + gd * D * ELT + c * 16) = ldg16(vb + gs * D * ELT + c * 16);
    }
    if (gl == 0) {
      a.alpha[gd] = a.alpha[gs];
      a.num[gd] = a.num[gs];
      a.den[gd] = a.den[gs];
      a.pos[gd] = a.pos[gs];
      a.vnorm[gd] = a.vnorm[gs];
      if (a.kept_out) a.kept_out[(size_t)u * B + dst] = src;
    }
  }
}

// Fused path: scores in registers, one workgroup per unit.
template <int DTYPE, int D>
__global__ void __launch_bounds__(ENT) score_select_kernel(EvictArgs a) {
  extern __shared__ int dyn[];
  __shared__ SelShared sh;
  const int u = blockIdx.x, tid = threadIdx.x;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  RegKeys<REG_KPT> keys;
#pragma unroll
  for (int k = 0; k < REG_KPT; ++k) {
    const int r = k * ENT + tid;
    keys.key[k] = ~0ull;
    if (r < a.L) {
      float x[4];
      int32_t p;
      load_features(a, ub + r, invT, x, p);
      const float s = policy_score(a, x);
      if (a.scores_out) a.scores_out[(size_t)u * a.L + r] = s;
      keys.key[k] = row_key(s, p);
    }
  }
  if (!a.evict) {
    if (a.kept_out)
      for (int r = tid; r < a.L; r += ENT) a.kept_out[(size_t)u * a.L + r] = r;
    return;
  }
  select_compact<RegKeys<REG_KPT>, DTYPE, D>(a, u, keys, REG_KPT, sh, dyn);
}

// Long caches: scores to keys in the workspace (grid over rows) ...
__global__ void __launch_bounds__(256) score_kernel(EvictArgs a, uint64_t* keys, int kstride) {
  const int u = blockIdx.y;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  for (int r = blockIdx.x * 256 + threadIdx.x; r < a.L; r += gridDim.x * 256) {
    float x[4];
    int32_t p;
    load_features(a, ub + r, invT, x, p);
    const float s = policy_score(a, x);
    if (a.scores_out) a.scores_out[(size_t)u * a.L + r] = s;
    keys[(size_t)u * kstride + r] = row_key(s, p);
  }
}

// ... then one workgroup per unit selects and compacts.
template <int DTYPE, int D>
__global__ void __launch_bounds__(ENT) select_kernel(EvictArgs a, const uint64_t* keys, int kstride) {
  extern __shared__ int dyn[];
  __shared__ SelShared sh;
  const int u = blockIdx.x;
  MemKeys mk{keys + (size_t)u * kstride};
  select_compact<MemKeys, DTYPE, D>(a, u, mk, (a.L + ENT - 1) / ENT, sh, dyn);
}

__global__ void identity_kept_kernel(int32_t* kept, int units, int L) {
  const size_t n = (size_t)units * L;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    kept[i] = (int32_t)(i % L);
}

int evict_max_len() { return MAX_LEN; }

template <int DTYPE, int D>
static int launch_evict_t(const EvictArgs& a, uint64_t* ws_keys, hipStream_t s) {
  if (!a.evict && !a.scores_out && !a.kept_out) return 0;
  const int E = a.L - a.budget;
  const int nmv = a.evict ? (E < a.budget ? E : a.budget) : 0;
  const size_t dyn = (size_t)(2 * (nmv > 0 ? nmv : 1)) * sizeof(int);
  if (a.L <= ENT * REG_KPT) {
    auto k = score_select_kernel<DTYPE, D>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    hipLaunchKernelGGL(k, dim3(a.units), dim3(ENT), dyn, s, a);
  } else {
    const int kstride = (a.L + ENT - 1) / ENT * ENT;
    int gx = (a.L + 255) / 256;
    hipLaunchKernelGGL(score_kernel, dim3(gx, a.units), dim3(256), 0, s, a, ws_keys, kstride);
    if (a.evict) {
      auto k = select_kernel<DTYPE, D>;
      hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
      hipLaunchKernelGGL(k, dim3(a.units), dim3(ENT), dyn, s, a, (const uint64_t*)ws_keys, kstride);
    } else if (a.kept_out) {
      hipLaunchKernelGGL(identity_kept_kernel, dim3(1024), dim3(256), 0, s, a.kept_out, a.units, a.L);
    }
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

size_t evict_ws_bytes(int units, int L) {
  if (L <= ENT * REG_KPT) return 0;
  const size_t kstride = (size_t)(L + ENT - 1) / ENT * ENT;
  return (size_t)units * kstride * sizeof(uint64_t);
}

}  // namespace dc
