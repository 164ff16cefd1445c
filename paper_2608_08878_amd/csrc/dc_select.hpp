// Scoring, top-B selection and hole-filling compaction shared by the
// stand-alone score/evict kernels and the fused decode+evict kernel.
#pragma once
#include <type_traits>

#include "dc_device.hpp"
#include "dc_kernels.hpp"

namespace dc {

constexpr int ENT = 1024;            // threads of the stand-alone select workgroup
constexpr int ENW_MAX = 16;          // waves per workgroup, at most
constexpr int REG_KPT = 8;           // rows per thread kept in registers (L <= 8192)
constexpr int MAX_LEN = 40960;

__device__ __forceinline__ uint32_t score_key(float s) {
  uint32_t b = __float_as_uint(s);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return 0u;  // NaN ranks lowest
  if (b == 0x80000000u) b = 0u;                                           // -0 -> +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint64_t row_key(float s, int32_t pos) {
  return ((uint64_t)score_key(s) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)pos);
}

// Rows and budget of unit u (ragged caches, per-unit budgets), clamped to the
// host's bounds (rows to [1, L], budgets to [1, budget]) so that a bad device
// value cannot take an access out of the buffers.
__device__ __forceinline__ int unit_rows(const EvictArgs& a, int u) {
  if (!a.unit_len) return a.L;
  const int n = a.unit_len[u];
  return n < 1 ? 1 : n > a.L ? a.L : n;
}
__device__ __forceinline__ int unit_budget(const EvictArgs& a, int u) {
  if (!a.budgets) return a.budget;
  const int b = a.budgets[u];
  return b < 1 ? 1 : b > a.budget ? a.budget : b;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two 32x32
// multiplies with the key advanced by the Weyl constants; only the first output
// word is used.
__device__ __forceinline__ uint32_t philox4x32_10_w0(uint32_t c0, uint32_t c1, uint32_t c2,
                                                     uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t h0 = __umulhi(0xD2511F53u, c0), l0 = 0xD2511F53u * c0;
    const uint32_t h1 = __umulhi(0xCD9E8D57u, c2), l1 = 0xCD9E8D57u * c2;
    c0 = h1 ^ c1 ^ k0;
    c1 = l1;
    c2 = h0 ^ c3 ^ k1;
    c3 = l0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c0;
}

// Training-mode ranking score (Sec. 3.1.2 Gumbel perturbation, App. C
// temperature): s / tau + g with g = -ln(-ln U) a standard Gumbel draw, U
// taken from Philox with counter (position, unit, draw, 0) so that a token
// keeps its draw wherever its row sits.  U = (2 (x >> 9) + 1) 2^-24 is exact in
// float32 and strictly inside (0, 1).
__device__ __forceinline__ float sampled_score(const EvictArgs& a, float s, int32_t pos, int unit) {
  const uint32_t x = philox4x32_10_w0((uint32_t)pos, (uint32_t)unit, a.draw, 0u, a.seed0, a.seed1);
  const float U = (float)(2u * (x >> 9) + 1u) * 0x1p-24f;
  return s / a.tau - logf(-logf(U));
}

// Feature vector x = [alpha, ||v||, H = num/den (0 if den = 0), pos / T].
__device__ __forceinline__ void make_features(float alpha, float vnorm, double num, double den,
                                              int32_t p, float invT, float x[4]) {
  x[0] = alpha;
  x[1] = vnorm;
  x[2] = den > 0.0 ? (float)(num / den) : 0.0f;
  x[3] = (float)p * invT;
}

__device__ __forceinline__ void load_features(const EvictArgs& a, size_t gi, float invT, float x[4],
                                              int32_t& p) {
  p = a.pos[gi];
  make_features(a.alpha[gi], a.vnorm[gi], a.num[gi], a.den[gi], p, invT, x);
}

// Policy parameters are read through the constant address space: no kernel
// writes them, so each load is a scalar load issued once per wave instead of a
// vector load per lane (which would compete with the cache streams for the
// vector memory pipeline).
typedef __attribute__((address_space(4))) const float cfloat;

__device__ __forceinline__ const cfloat* const_params(const float* p) {
  return (const cfloat*)p;
}

// Extended one-hidden-layer policy (a fifth input sigma_i and/or LayerNorm,
// width up to 128): x has n_in inputs in the paper's order; z = W x + b,
// [z = gain (z - mean) / sqrt(var + 1e-5) + bias over the layer], h = relu(z);
// s = w_out . h + b_out.  Float32 with fixed evaluation order (bias first,
// inputs / units in order); LayerNorm moments accumulated in binary64.  The
// hidden layer lives in registers (128 slots); out of line so that they do not
// share the caller's register budget.  (Two hidden layers run on the matrix
// cores: dc_mlp.hip.)
constexpr int EXT_HMAX = 128;
constexpr float LN_EPS = 1e-5f;

__device__ __attribute__((noinline)) float mlp_ext(const float* params, int n_in, int h1, int ln,
                                                   float x0, float x1, float x2, float x3,
                                                   float x4) {
  const cfloat* W = const_params(params);
  const cfloat* b = W + h1 * n_in;
  const float xin[5] = {x0, x1, x2, x3, x4};
  float h[EXT_HMAX];
  double s1 = 0.0, s2 = 0.0;
#pragma unroll
  for (int i = 0; i < EXT_HMAX; ++i) {
    float z = 0.0f;
    if (i < h1) {
      z = b[i];
#pragma unroll
      for (int k = 0; k < 5; ++k)
        if (k < n_in) z = __builtin_fmaf(W[i * n_in + k], xin[k], z);
      s1 += (double)z;
      s2 += (double)z * (double)z;
    }
    h[i] = z;
  }
  const cfloat* next = b + h1;
  if (ln) {
    const cfloat* g = next;
    const cfloat* be = next + h1;
    next += 2 * h1;
    const double mean = s1 / h1;
    const double var = s2 / h1 - mean * mean;
    const float m = (float)mean;
    const float rs = (float)(1.0 / sqrt((var > 0.0 ? var : 0.0) + (double)LN_EPS));
#pragma unroll
    for (int i = 0; i < EXT_HMAX; ++i)
      if (i < h1) h[i] = __builtin_fmaf((h[i] - m) * rs, g[i], be[i]);
  }
#pragma unroll
  for (int i = 0; i < EXT_HMAX; ++i) h[i] = fmaxf(h[i], 0.0f);
  const cfloat* wo = next;
  float out = wo[h1];
#pragma unroll
  for (int i = 0; i < EXT_HMAX; ++i)
    if (i < h1) out = __builtin_fmaf(wo[i], h[i], out);
  return out;
}

// Score of row gi under the extended policy (features in the paper's order;
// sigma only with five inputs).
__device__ __forceinline__ float ext_score(const EvictArgs& a, size_t gi, float invT, int32_t& p) {
  p = a.pos[gi];
  const double num = a.num[gi], den = a.den[gi];
  const float H = den > 0.0 ? (float)(num / den) : 0.0f;
  const float al = a.alpha[gi], vn = a.vnorm[gi], ps = (float)p * invT;
  if (a.n_in == 5)
    return mlp_ext(a.params, 5, a.h1, a.ln, al, vn, a.sigma[gi], H, ps);
  return mlp_ext(a.params, 4, a.h1, a.ln, al, vn, H, ps, 0.0f);
}

// Policy weights staged in LDS are read through LDS-typed pointers, so the
// reads stay ds_read instructions even behind an optimisation barrier.
typedef __attribute__((address_space(3))) const float lfloat;

// One hidden unit of the one-hidden-layer MLP for KP rows.
template <int KP>
__device__ __forceinline__ void mlp1_unit(const cfloat* W1, const cfloat* b1, const cfloat* wo,
                                          int h, const float (&x)[KP][4], float (&out)[KP],
                                          int kact) {
  const float w0 = W1[4 * h], w1 = W1[4 * h + 1], w2 = W1[4 * h + 2], w3 = W1[4 * h + 3];
  const float bb = b1[h], ww = wo[h];
#pragma unroll
  for (int k = 0; k < KP; ++k) {
    if (k < kact) {
      float z = bb;
      z = __builtin_fmaf(w0, x[k][0], z);
      z = __builtin_fmaf(w1, x[k][1], z);
      z = __builtin_fmaf(w2, x[k][2], z);
      z = __builtin_fmaf(w3, x[k][3], z);
      out[k] = __builtin_fmaf(ww, fmaxf(z, 0.0f), out[k]);
    }
  }
}

// Scores of KP rows per thread, s = f_phi(x) for the one-hidden-layer policy
// in float32 with a fixed evaluation order: out = b_out, then for every hidden
// unit h in order
// out += w_out[h] relu(b1[h] + W1[h,0] x0 + W1[h,1] x1 + W1[h,2] x2 + W1[h,3] x3).
// Row slots k >= kact (uniform over the wave) are skipped.  The loops over the
// hidden units are uniform, so every weight is read once per wave and reused
// for all row slots.
template <int KP>
__device__ __forceinline__ void policy_scores(const EvictArgs& a, const float (&x)[KP][4],
                                              float (&out)[KP], int kact) {
  const cfloat* P = const_params(a.params);
  const int h1 = a.h1;
  const cfloat* W1 = P;
  const cfloat* b1 = P + 4 * h1;
  const cfloat* wo = b1 + h1;
  const float bo = wo[h1];
#pragma unroll
  for (int k = 0; k < KP; ++k) out[k] = bo;
  int h = 0;
  for (; h + 4 <= h1; h += 4) {       // four units per trip: the scalar loads batch up
#pragma unroll
    for (int q = 0; q < 4; ++q) mlp1_unit<KP>(W1, b1, wo, h + q, x, out, kact);
  }
  for (; h < h1; ++h) mlp1_unit<KP>(W1, b1, wo, h, x, out, kact);
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

// The keys of rows k*NT + tid for k in [k0, k0 + 8) from the workspace, requested
// together (eight loads in flight instead of one at a time); rows past L (and k
// past kpt) read as ~0, which no selection takes.
template <typename Keys, int NT>
__device__ __forceinline__ void key_batch(const Keys& keys, int k0, int kpt, int L, uint64_t (&x)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = (k0 + j) * NT + (int)threadIdx.x;
    x[j] = keys.key[r < L ? r : L - 1];                // unconditional, in bounds
  }
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (k0 + j >= kpt || (k0 + j) * NT + (int)threadIdx.x >= L) x[j] = ~0ull;
}

// ... or in LDS (fused decode+evict kernel).
// Keys in LDS at a row stride of `stride` u64 (rows k * NT + tid).
template <int KM, int NT>
struct LdsKeys {
  static constexpr int KMAX = KM;
  const uint64_t* key;
  int stride;
  __device__ uint64_t get(int k) const { return key[(size_t)(k * NT + threadIdx.x) * stride]; }
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
  uint64_t wmin[ENW_MAX];
  int hist[256];
  int sel[4];            // digit, count below, count in digit, evicted slot
  int wcnt[2][ENW_MAX];  // per-wave hole / mover counts
  int nmoves;
};

// Block exclusive scans of two flags over rows k*NT + tid (one k at a time).
template <int NT>
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
  for (int w = 0; w < NT / 64; ++w) {
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
// rows k*NT + tid for k < kpt (invalid rows beyond L are ignored); NT is the
// workgroup size.
// Keep the top B of unit u's L rows (B < L) and compact; kept_out rows have
// stride a.ld_kept.  Move j of the plan is the pair (hole, mover) at
// mv[MS j], mv[MS j + 1] (MS = 2: a dense list; a larger stride lets the list
// share row slots with the keys, move j beside row j's key).  BATCHED (the
// stand-alone selection, many moves per unit): the state fields of 16
// consecutive moves travel together, lane q of a 16-lane group carrying move
// q's, so each field's reads and writes coalesce (the movers and the holes
// both ascend); otherwise lane q of a group carries field q of one move.
template <typename Keys, int DTYPE, int D, int NT = ENT, int MS = 2, bool BATCHED = false>
__device__ void select_compact(const EvictArgs& a, int u, int L, int B, const Keys& keys, int kpt,
                               SelShared& sh, int* mv) {
  constexpr int ELT = DTYPE == 0 ? 4 : 2;
  constexpr bool GLOBAL_KEYS = std::is_same<Keys, MemKeys>::value;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = L - B;
  const size_t ub = (size_t)u * a.cap;
  // threshold: evicted rows are those with key <= thr
  uint64_t thr;
  if (E == 1) {
    uint64_t m = ~0ull;
    int mr = -1;                        // (global keys) the row of this thread's minimum
    if constexpr (GLOBAL_KEYS) {
      for (int k0 = 0; k0 < kpt; k0 += 8) {
        uint64_t x[8];
        key_batch<Keys, NT>(keys, k0, kpt, L, x);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (x[j] < m) {
            m = x[j];
            mr = (k0 + j) * NT + tid;
          }
      }
    } else {
#pragma unroll
      for (int k = 0; k < Keys::KMAX; ++k) {
        if (k >= kpt) break;
        const int r = k * NT + tid;
        if (r < L) {
          const uint64_t x = keys.get(k);
          m = x < m ? x : m;
        }
      }
    }
    const uint64_t mine = m;
    m = wave_min(m);
    if (lane == 0) sh.wmin[wave] = m;
    __syncthreads();
    thr = sh.wmin[0];
    for (int w = 1; w < NT / 64; ++w) thr = sh.wmin[w] < thr ? sh.wmin[w] : thr;
    // one row leaves: if it sits below B, the row in slot B (the only slot >= B)
    // fills it; no scans needed.  Keys are unique, so exactly one row holds thr.
    if constexpr (GLOBAL_KEYS) {
      if (mr >= 0 && mine == thr) sh.sel[3] = mr;
    } else {
#pragma unroll
      for (int k = 0; k < Keys::KMAX; ++k) {
        if (k >= kpt) break;
        const int r = k * NT + tid;
        if (r < L && keys.get(k) == thr) sh.sel[3] = r;
      }
    }
    __syncthreads();
    const int ev = sh.sel[3];
    if (a.kept_out)
      for (int r = tid; r < B; r += NT) a.kept_out[(size_t)u * a.ld_kept + r] = r == ev ? B : r;
    if (ev < B && tid < 64) {
      const size_t gd = ub + ev, gs = ub + B;
      constexpr int N16 = D * ELT / 16;
      char* kb = (char*)a.k;
      char* vb = (char*)a.v;
      for (int c = tid; c < 2 * N16; c += 64) {
        char* base = c < N16 ? kb : vb;
        const int cc = c < N16 ? c : c - N16;
        *reinterpret_cast<uint4*>(base + gd * D * ELT + cc * 16) = ldg16(base + gs * D * ELT + cc * 16);
      }
      if (tid == 0) {
        a.alpha[gd] = a.alpha[gs];
        a.num[gd] = a.num[gs];
        a.den[gd] = a.den[gs];
        a.pos[gd] = a.pos[gs];
        a.vnorm[gd] = a.vnorm[gs];
        if (a.sigma) a.sigma[gd] = a.sigma[gs];
      }
    }
    return;
  } else {
    uint64_t prefix = 0;
    int need = E;
    int shift = 56;
    for (;; shift -= 8) {
      const uint64_t hmask = shift + 8 >= 64 ? 0ull : (~0ull << (shift + 8));
      for (int i = tid; i < 256; i += NT) sh.hist[i] = 0;
      __syncthreads();
      if constexpr (GLOBAL_KEYS) {
        for (int k0 = 0; k0 < kpt; k0 += 8) {
          uint64_t x[8];
          key_batch<Keys, NT>(keys, k0, kpt, L, x);
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (k0 + j < kpt && (k0 + j) * NT + tid < L && (x[j] & hmask) == prefix)
              atomicAdd(&sh.hist[(int)((x[j] >> shift) & 255u)], 1);
        }
      } else {
#pragma unroll
        for (int k = 0; k < Keys::KMAX; ++k) {
          if (k >= kpt) break;
          const int r = k * NT + tid;
          if (r < L) {
            const uint64_t x = keys.get(k);
            if ((x & hmask) == prefix) atomicAdd(&sh.hist[(int)((x >> shift) & 255u)], 1);
          }
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
  auto plan_row = [&](int r, bool ev) {
    const bool hole = r < B && ev;
    const bool mover = r >= B && r < L && !ev;
    int rk0, rk1, t0, t1;
    block_scan2<NT>(hole, mover, rk0, rk1, t0, t1, sh);
    if (hole) mv[MS * (run0 + rk0)] = r;
    if (mover) mv[MS * (run1 + rk1) + 1] = r;
    if (a.kept_out && r < B && !ev) a.kept_out[(size_t)u * a.ld_kept + r] = r;
    run0 += t0;
    run1 += t1;
  };
  if constexpr (GLOBAL_KEYS) {
    for (int k0 = 0; k0 < kpt && k0 * NT < L; k0 += 8) {
      uint64_t x[8];
      key_batch<Keys, NT>(keys, k0, kpt, L, x);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = k0 + j;
        if (k >= kpt || k * NT >= L) break;
        const int r = k * NT + tid;
        plan_row(r, r < L && x[j] <= thr);
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < Keys::KMAX; ++k) {
      if (k >= kpt || k * NT >= L) break;
      const int r = k * NT + tid;
      bool ev = false;
      if (r < L) ev = keys.get(k) <= thr;
      plan_row(r, ev);
    }
  }
  __syncthreads();
  const int nm = run0;  // == run1
  // copy rows: one 16-lane group per move, MB moves per trip with every load
  // issued before the stores (moves are independent: sources and destinations
  // are disjoint); lane gl of a group also carries state field gl
  constexpr int N16 = D * ELT / 16;        // 16-byte chunks per row (8, 16 or 32)
  constexpr int CPL = (N16 + 15) / 16;     // chunks per lane
  constexpr int MB = 4;
  const int grp = tid / 16, gl = tid % 16, ngrp = NT / 16;
  char* kb = (char*)a.k;
  char* vb = (char*)a.v;
  if constexpr (BATCHED) {
    for (int b0 = 16 * grp; b0 < nm; b0 += 16 * ngrp) {
      // state of moves b0 .. b0 + 15, lane gl carrying move b0 + gl (past the
      // list: re-read move b0, no store); requested before the rows
      const bool sok = b0 + gl < nm;
      const int js = sok ? b0 + gl : b0;
      const size_t sd = ub + mv[MS * js], ss = ub + mv[MS * js + 1];
      const float s_al = a.alpha[ss], s_vn = a.vnorm[ss];
      const double s_nu = a.num[ss], s_de = a.den[ss];
      const int32_t s_po = a.pos[ss];
      const float s_sg = a.sigma ? a.sigma[ss] : 0.0f;
      // rows: all 16 lanes per move, MB moves per trip, every load before the stores
      const int mend = nm - b0 < 16 ? nm - b0 : 16;
      for (int m0 = 0; m0 < mend; m0 += MB) {
        size_t gd[MB], gs[MB];
        uint4 kx[MB][CPL], vx[MB][CPL];
#pragma unroll
        for (int q = 0; q < MB; ++q) {
          const int j = b0 + (m0 + q < mend ? m0 + q : m0);
          gd[q] = ub + mv[MS * j];
          gs[q] = ub + mv[MS * j + 1];
#pragma unroll
          for (int cc = 0; cc < CPL; ++cc) {
            const int c = gl + 16 * cc < N16 ? gl + 16 * cc : N16 - 1;
            kx[q][cc] = ldg16(kb + gs[q] * D * ELT + c * 16);
            vx[q][cc] = ldg16(vb + gs[q] * D * ELT + c * 16);
          }
        }
#pragma unroll
        for (int q = 0; q < MB; ++q) {
          if (m0 + q >= mend) continue;
#pragma unroll
          for (int cc = 0; cc < CPL; ++cc) {
            const int c = gl + 16 * cc;
            if (c < N16) {
              *reinterpret_cast<uint4*>(kb + gd[q] * D * ELT + c * 16) = kx[q][cc];
              *reinterpret_cast<uint4*>(vb + gd[q] * D * ELT + c * 16) = vx[q][cc];
            }
          }
        }
      }
      if (sok) {
        a.alpha[sd] = s_al;
        a.vnorm[sd] = s_vn;
        a.num[sd] = s_nu;
        a.den[sd] = s_de;
        a.pos[sd] = s_po;
        if (a.sigma) a.sigma[sd] = s_sg;
        if (a.kept_out) a.kept_out[(size_t)u * a.ld_kept + (int)(sd - ub)] = (int)(ss - ub);
      }
    }
    return;
  }
  for (int j0 = grp; j0 < nm; j0 += MB * ngrp) {
    size_t gd[MB], gs[MB];
    bool ok[MB];
    uint4 kx[MB][CPL], vx[MB][CPL];
    uint64_t sv[MB];
#pragma unroll
    for (int q = 0; q < MB; ++q) {
      const int j = j0 + q * ngrp;
      ok[q] = j < nm;
      const int jj = ok[q] ? j : j0;         // past the list: re-read a listed move, no store
      gd[q] = ub + mv[MS * jj];
      gs[q] = ub + mv[MS * jj + 1];
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int c = gl + 16 * cc < N16 ? gl + 16 * cc : N16 - 1;
        kx[q][cc] = ldg16(kb + gs[q] * D * ELT + c * 16);
        vx[q][cc] = ldg16(vb + gs[q] * D * ELT + c * 16);
      }
      sv[q] = 0;
      if (gl == 0) sv[q] = __float_as_uint(a.alpha[gs[q]]);
      else if (gl == 1) sv[q] = (uint64_t)__double_as_longlong(a.num[gs[q]]);
      else if (gl == 2) sv[q] = (uint64_t)__double_as_longlong(a.den[gs[q]]);
      else if (gl == 3) sv[q] = (uint32_t)a.pos[gs[q]];
      else if (gl == 4) sv[q] = __float_as_uint(a.vnorm[gs[q]]);
      else if (gl == 5 && a.sigma) sv[q] = __float_as_uint(a.sigma[gs[q]]);
    }
#pragma unroll
    for (int q = 0; q < MB; ++q) {
      if (!ok[q]) continue;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int c = gl + 16 * cc;
        if (c < N16) {
          *reinterpret_cast<uint4*>(kb + gd[q] * D * ELT + c * 16) = kx[q][cc];
          *reinterpret_cast<uint4*>(vb + gd[q] * D * ELT + c * 16) = vx[q][cc];
        }
      }
      if (gl == 0) a.alpha[gd[q]] = __uint_as_float((uint32_t)sv[q]);
      else if (gl == 1) a.num[gd[q]] = __longlong_as_double((long long)sv[q]);
      else if (gl == 2) a.den[gd[q]] = __longlong_as_double((long long)sv[q]);
      else if (gl == 3) a.pos[gd[q]] = (int32_t)(uint32_t)sv[q];
      else if (gl == 4) a.vnorm[gd[q]] = __uint_as_float((uint32_t)sv[q]);
      else if (gl == 5 && a.sigma) a.sigma[gd[q]] = __uint_as_float((uint32_t)sv[q]);
      else if (gl == 6 && a.kept_out)
        a.kept_out[(size_t)u * a.ld_kept + (int)(gd[q] - ub)] = (int)(gs[q] - ub);
    }
  }
}

}  // namespace dc
