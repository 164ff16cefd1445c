// Exact log-partition of the size-B subset law and the log-probability of a
// kept set (App. C, policy-gradient derivation for Gumbel-top-B), gfx950.
//
// For the scores s_i of one unit's L rows and r_i = s_i / tau:
//   log Z(s, B, tau) = log sum over size-B subsets a of exp(sum_{i in a} r_i)
//                    = log e_B(exp(r_1), ..., exp(r_L)),
// e_B the elementary symmetric polynomial of degree B, and
//   log pi(a | s) = sum_{i in a} r_i - log Z.
//
// Design.  e_B satisfies e_B(x) = (prod x) e_{L-B}(1 / x), so the programme
// runs over K = min(B, L - B) entries instead of B: a step that evicts one
// token costs O(L), not O(L B).  With x_i = exp(+-r_i - shift) (shift = the
// largest exponent, so every weight is at most 1) the recursion
//   E_i[j] = E_{i-1}[j] + x_i E_{i-1}[j - 1],   E[0] = 1,
// adds positive terms only, so it runs in linear space: each entry is a
// float32 mantissa in [0.5, 1) with its own int32 exponent (the entries span
// far more than any floating-point exponent range), renormalised with frexp
// once per 64 updates.  One update is one fused multiply-add plus exponent
// alignment (seven VALU instructions, no transcendental), and it is more
// accurate than log-space float32: every term is positive, so the relative
// error of E_L[K] stays below about (K + L) 2^-24 (rounding of the weights plus
// one rounding per update).
//
// Two layouts, one wave (64 lanes) per unit:
//  - K <= 8 (row split): every lane folds the rows i = lane (mod 64) into its
//    own truncated polynomial, then six butterfly levels multiply the lanes'
//    polynomials (truncated convolution, the lower lane's factor first, so
//    that both partners compute identical bits).
//  - K > 8 (column): lane l holds entries 1 + l C .. (l + 1) C and all lanes
//    take the rows in order; entry l C + 1 needs the previous value of entry
//    l C from lane l - 1 (one cross-lane shift per row).  K > 64 C_MAX is done
//    in bands of 64 C_MAX entries: a band records, for every row, the previous
//    value of its top entry in the caller's workspace and the next band reads
//    it as its entry below.
//
// Weights below 2^-16384 of the largest are clamped to 2^-16384 (so the
// exponent bookkeeping stays in int32 range for K up to 20480); scores whose
// ratio to tau spans more than about 11000 are outside exact coverage.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dc_kernels.hpp"

#pragma clang fp contract(off)

namespace dc {

namespace {

constexpr int KZERO = -(1 << 30);        // exponent of an exact zero entry (mantissa 0)
constexpr int KMIN_W = -16384;           // smallest weight exponent kept
constexpr int C_MAX = 64;                // entries per lane in the column layout
constexpr int BAND = 64 * C_MAX;
constexpr double LN2 = 0x1.62e42fefa39efp-1;
constexpr double LN2_HI = 0x1.62e42fee00000p-1;   // Cody-Waite split of ln 2
constexpr double LN2_LO = 0x1.a39ef35793c76p-33;
constexpr double INV_LN2 = 0x1.71547652b82fep+0;

__device__ __forceinline__ float rdl(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}
__device__ __forceinline__ int rdl(int x, int l) { return __builtin_amdgcn_readlane(x, l); }

// (m, k) = v with v = m 2^k, m in [0.5, 1) (or m = 0), exponent offset kn.
__device__ __forceinline__ void norm(float v, int kn, float& m, int& k) {
  m = __builtin_amdgcn_frexp_mantf(v);
  k = kn + __builtin_amdgcn_frexp_expf(v);
}

// E[j] <- E[j] + x E[j-1]  (x = xm 2^xk, xm in [0.5, 1); (pm, pk) the previous
// E[j-1]).  Both terms are aligned to the larger exponent and the sum keeps
// that exponent without renormalising: the mantissa of the aligned-to term is
// at most halved (x's mantissa) and the sum at most doubled per update, so
// after at most RENORM updates from [0.5, 1) every mantissa lies in
// [2^-65, 2^64], far inside float32's normal range, and a term shifted below
// float32's range is under 2^-61 of the sum it joins.
__device__ __forceinline__ void upd(float& m, int& k, float pm, int pk, float xm, int xk) {
  const int kb = pk + xk;
  const int kn = k > kb ? k : kb;
  const float a = __builtin_amdgcn_ldexpf(m, k - kn);
  const float b = __builtin_amdgcn_ldexpf(pm, kb - kn);
  m = __builtin_fmaf(xm, b, a);
  k = kn;
}

constexpr int RENORM = 64;   // updates between renormalisations (one row batch)

__device__ __forceinline__ void renorm(float& m, int& k) { norm(m, k, m, k); }

// Weight exp(z), z <= 0, as (m, k): z = n ln2 + f with f in [0, ln2) (Cody-Waite).
__device__ __forceinline__ void weight(double z, float& m, int& k) {
  double n = floor(z * INV_LN2);
  n = n < (double)KMIN_W ? (double)KMIN_W : n;
  const double f = (z - n * LN2_HI) - n * LN2_LO;
  const float e = (float)exp(f > 0.0 ? f : 0.0);   // z below the clamp gives f < 0: weight 2^n
  norm(e, (int)n, m, k);
}

// Sizes of unit u (ragged caches and per-unit budgets: per unit; the host
// chose the kernel for an upper bound of K).
struct UnitDims {
  int L, B, nk, K, neg;
};

__device__ __forceinline__ UnitDims unit_dims(const LogzArgs& a, int u) {
  UnitDims d;
  // device values clamped to the host's bounds (rows [1, L], budgets [1, B])
  d.L = a.unit_len ? (a.unit_len[u] < 1 ? 1 : a.unit_len[u] > a.L ? a.L : a.unit_len[u]) : a.L;
  d.B = a.budgets ? (a.budgets[u] < 1 ? 1 : a.budgets[u] > a.B ? a.B : a.budgets[u]) : a.B;
  d.nk = d.B < d.L ? d.B : d.L;
  d.K = d.B >= d.L ? 0 : (d.B <= d.L - d.B ? d.B : d.L - d.B);
  d.neg = d.B < d.L && d.L - d.B < d.B;
  return d;
}

struct UnitStats {
  double shift;    // max over rows of (neg ? -r : r)
  double sumr;     // sum of r
  double kept;     // sum of r over the kept rows
  int bad;         // a non-finite r, or a kept index outside [0, L)
};

__device__ __forceinline__ double wave_max(double x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    const double y = __shfl_xor(x, d);
    x = x > y ? x : y;
  }
  return x;
}
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d);
  return x;
}
__device__ __forceinline__ int wave_or(int x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x |= __shfl_xor(x, d);
  return x;
}

__device__ __forceinline__ double r_of(const LogzArgs& a, float s) { return (double)s / (double)a.tau; }

__device__ UnitStats unit_stats(const LogzArgs& a, const UnitDims& d, const float* s,
                                const int32_t* kept, int lane) {
  double mx = -INFINITY, sum = 0.0, ks = 0.0;
  int bad = 0;
  // (unrolled so that eight iterations' loads are in flight together; the
  // sums keep their order)
#pragma unroll 8
  for (int i = lane; i < d.L; i += 64) {
    const double r = r_of(a, s[i]);
    bad |= !isfinite(r);
    const double x = d.neg ? -r : r;
    mx = x > mx ? x : mx;
    sum += r;
  }
  if (kept) {
#pragma unroll 8
    for (int t = lane; t < d.nk; t += 64) {
      const int idx = kept[t];
      if (idx < 0 || idx >= d.L) bad = 1;
      else ks += r_of(a, s[idx]);
    }
  }
  UnitStats st;
  st.shift = wave_max(mx);
  st.sumr = wave_sum(sum);
  st.kept = wave_sum(ks);
  st.bad = wave_or(bad);
  return st;
}

__device__ __forceinline__ void row_weight(const LogzArgs& a, const UnitDims& d, float s,
                                           double shift, float& m, int& k) {
  const double r = r_of(a, s);
  weight((d.neg ? -r : r) - shift, m, k);
}

__device__ void finish(const LogzArgs& a, const UnitDims& d, int u, const UnitStats& st, float mK,
                       int kK, int lane) {
  if (lane) return;
  double logz;
  if (d.K == 0) logz = st.sumr;                  // one subset: the whole cache
  else logz = (double)d.K * st.shift + (d.neg ? st.sumr : 0.0) + log((double)mK) + (double)kK * LN2;
  double logp = d.B >= d.L ? 0.0 : st.kept - logz;
  if (st.bad) logz = logp = __builtin_nan("");
  if (a.logz) a.logz[u] = logz;
  if (a.logp) a.logp[u] = logp;
}

// Truncated product c = lo * hi of two polynomials with c_0 = lo_0 = hi_0 = 1
// (entries 1..KS stored), terms in the fixed order t = 0..j.
template <int KS>
__device__ __forceinline__ void poly_mul(const float* lm, const int* lk, const float* hm,
                                         const int* hk, float* cm, int* ck) {
#pragma unroll
  for (int j = 1; j <= KS; ++j) {
    int kt[KS + 1];
    float mt[KS + 1];
    int kn = KZERO;
#pragma unroll
    for (int t = 0; t <= j; ++t) {
      const float am = t == 0 ? 0.5f : lm[t - 1];
      const int ak = t == 0 ? 1 : lk[t - 1];
      const float bm = t == j ? 0.5f : hm[j - t - 1];
      const int bk = t == j ? 1 : hk[j - t - 1];
      int e = ak + bk;                            // both >= -2^30: no overflow
      e = e > KZERO ? e : KZERO;
      kt[t] = e;
      mt[t] = am * bm;
      kn = e > kn ? e : kn;
    }
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t <= j; ++t) acc += __builtin_amdgcn_ldexpf(mt[t], kt[t] - kn);
    norm(acc, kn, cm[j - 1], ck[j - 1]);
  }
}

template <int KS>
__global__ void __launch_bounds__(64) logz_rows_kernel(LogzArgs a) {
  const int u = blockIdx.x, lane = threadIdx.x;
  const UnitDims d = unit_dims(a, u);
  const float* s = a.scores + (size_t)u * a.L;
  const UnitStats st = unit_stats(a, d, s, a.kept ? a.kept + (size_t)u * a.nk : nullptr, lane);
  float m[KS];
  int k[KS];
#pragma unroll
  for (int j = 0; j < KS; ++j) {
    m[j] = 0.0f;
    k[j] = KZERO;
  }
  for (int i0 = 0; i0 < d.L; i0 += 64 * RENORM) {
    const int iend = d.L < i0 + 64 * RENORM ? d.L : i0 + 64 * RENORM;
#pragma unroll 8
    for (int i = i0 + lane; i < iend; i += 64) {
      float xm;
      int xk;
      row_weight(a, d, s[i], st.shift, xm, xk);
#pragma unroll
      for (int j = KS - 1; j >= 1; --j) upd(m[j], k[j], m[j - 1], k[j - 1], xm, xk);
      upd(m[0], k[0], 0.5f, 1, xm, xk);
    }
#pragma unroll
    for (int j = 0; j < KS; ++j) renorm(m[j], k[j]);
  }
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    float pm[KS], lm[KS], hm[KS];
    int pk[KS], lk[KS], hk[KS];
    const bool low = !(lane & d);
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      pm[j] = __shfl_xor(m[j], d);
      pk[j] = __shfl_xor(k[j], d);
      lm[j] = low ? m[j] : pm[j];
      lk[j] = low ? k[j] : pk[j];
      hm[j] = low ? pm[j] : m[j];
      hk[j] = low ? pk[j] : k[j];
    }
    poly_mul<KS>(lm, lk, hm, hk, m, k);
  }
  float mK = 0.5f;
  int kK = 1;
#pragma unroll
  for (int j = 0; j < KS; ++j)
    if (j == d.K - 1) {
      mK = m[j];
      kK = k[j];
    }
  finish(a, d, u, st, mK, kK, lane);
}

template <int C>
__global__ void __launch_bounds__(64) logz_col_kernel(LogzArgs a) {
  const int u = blockIdx.x, lane = threadIdx.x;
  const UnitDims d = unit_dims(a, u);
  const float* s = a.scores + (size_t)u * a.L;
  const UnitStats st = unit_stats(a, d, s, a.kept ? a.kept + (size_t)u * a.nk : nullptr, lane);
  float mK = 0.5f;
  int kK = 1;
  if (d.K > 0) {
    const int nb = (d.K + 64 * C - 1) / (64 * C);
    float* cm = a.col_m ? a.col_m + (size_t)u * a.L : nullptr;
    int* ck = a.col_k ? a.col_k + (size_t)u * a.L : nullptr;
    for (int band = 0; band < nb; ++band) {
      const bool rd = band > 0, wr = band + 1 < nb;
      float m[C];
      int k[C];
#pragma unroll
      for (int t = 0; t < C; ++t) {
        m[t] = 0.0f;
        k[t] = KZERO;
      }
      for (int i0 = 0; i0 < d.L; i0 += 64) {
        const int n = d.L - i0 < 64 ? d.L - i0 : 64;
        float xm = 0.0f, inm = 0.5f, outm = 0.0f;
        int xk = KZERO, ink = 1, outk = KZERO;
        if (lane < n) {
          row_weight(a, d, s[i0 + lane], st.shift, xm, xk);
          if (rd) {
            inm = cm[i0 + lane];
            ink = ck[i0 + lane];
          }
        }
        // one row: entry l C + 1 takes lane l - 1's top entry (lane 0: the band
        // column, or E[0] = 1); the band's top entry is recorded before the update
        auto row = [&](int r) {
          const float sxm = rdl(xm, r);
          const int sxk = rdl(xk, r);
          float nm = __shfl_up(m[C - 1], 1);
          int nk = __shfl_up(k[C - 1], 1);
          if (lane == 0) {
            nm = rdl(inm, r);
            nk = rdl(ink, r);
          }
          if (wr) {
            const float tm = rdl(m[C - 1], 63);
            const int tk = rdl(k[C - 1], 63);
            if (lane == r) {
              outm = tm;
              outk = tk;
            }
          }
#pragma unroll
          for (int t = C - 1; t >= 1; --t) upd(m[t], k[t], m[t - 1], k[t - 1], sxm, sxk);
          upd(m[0], k[0], nm, nk, sxm, sxk);
        };
        // two rows per trip (written out: the loop holds cross-lane operations,
        // which the compiler does not unroll), so that the exponents alternate
        // between two register sets instead of being copied back every row
        int r = 0;
        for (; r + 1 < n; r += 2) {
          row(r);
          row(r + 1);
        }
        if (r < n) row(r);
        static_assert(RENORM >= 64, "one renormalisation per row batch");
#pragma unroll
        for (int t = 0; t < C; ++t) renorm(m[t], k[t]);
        if (wr && lane < n) {
          cm[i0 + lane] = outm;
          ck[i0 + lane] = outk;
        }
      }
      const int jj = d.K - 1 - band * 64 * C;     // entry K within this band
      if (jj >= 0 && jj < 64 * C) {
        float pm = 0.0f;
        int pk = KZERO;
#pragma unroll
        for (int t = 0; t < C; ++t)
          if (t == jj % C) {
            pm = m[t];
            pk = k[t];
          }
        mK = rdl(pm, jj / C);
        kK = rdl(pk, jj / C);
      }
    }
  }
  finish(a, d, u, st, mK, kK, lane);
}

template <typename F>
int launch1(F kern, const LogzArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(kern, dim3(a.units), dim3(64), 0, s, a);
  return (int)hipGetLastError();
}

}  // namespace

int logz_band_entries() { return BAND; }

size_t logz_ws_bytes(int units, int L, int B) {
  const int K = B >= L ? 0 : (B < L - B ? B : L - B);
  return K > BAND ? (size_t)units * L * (sizeof(float) + sizeof(int)) : 0;
}

int launch_logz(const LogzArgs& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int K = a.K;
  if (K <= 1) return launch1(logz_rows_kernel<1>, a, s);
  if (K <= 2) return launch1(logz_rows_kernel<2>, a, s);
  if (K <= 4) return launch1(logz_rows_kernel<4>, a, s);
  if (K <= 8) return launch1(logz_rows_kernel<8>, a, s);
  const int c = (K + 63) / 64;
  if (c <= 1) return launch1(logz_col_kernel<1>, a, s);
  if (c <= 2) return launch1(logz_col_kernel<2>, a, s);
  if (c <= 4) return launch1(logz_col_kernel<4>, a, s);
  if (c <= 8) return launch1(logz_col_kernel<8>, a, s);
  if (c <= 12) return launch1(logz_col_kernel<12>, a, s);
  if (c <= 16) return launch1(logz_col_kernel<16>, a, s);
  if (c <= 24) return launch1(logz_col_kernel<24>, a, s);
  if (c <= 32) return launch1(logz_col_kernel<32>, a, s);
  if (c <= 48) return launch1(logz_col_kernel<48>, a, s);
  return launch1(logz_col_kernel<C_MAX>, a, s);
}

}  // namespace dc
