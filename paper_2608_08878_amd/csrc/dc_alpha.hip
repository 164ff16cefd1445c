// The paper's alpha (Sec. 3.1.1, state space): the attention mass a token
// received in the most recent forward pass averaged over all heads and layers,
// formed from every KV unit's recent mass (the G-head mean its decode step
// left in alpha), gfx950.
//
// For sequence b (units b * per_seq .. b * per_seq + per_seq - 1: every layer
// and KV head) and position p:
//     A_b(p) = (1 / per_seq) sum_{units u of b} alpha_u(p),
// alpha_u(p) = 0 when unit u does not hold p.  Every unit has the same number
// of query heads, so this is the mean over all the sequence's heads.  The sums
// are 64-bit fixed point (2^-52 per unit of alpha): integer sums do not depend
// on their order, so the result is deterministic.
//   1. ga_add_kernel: a workgroup takes a group of GA_UG units of one sequence
//      and a window of positions, adds its rows' alpha into an LDS histogram of
//      the window and stores it as the group's partial sums;
//   2. ga_sum_kernel: the partial sums of a sequence's groups, in group order;
//   3. ga_write_kernel: every row takes its position's sum / per_seq.
// Rows are read once per window (two windows cover 32768 positions).
#include <hip/hip_runtime.h>

#include "dc_kernels.hpp"

namespace dc {

namespace {

constexpr double GA_ONE = 0x1p52;     // fixed-point 1.0; per_seq <= 2048 keeps sums below 2^63
constexpr int GA_T = 256;             // threads of the sum and write kernels
constexpr int GA_AT = 1024;           // threads of the add kernel
constexpr int GA_UG = 16;             // units per add workgroup
constexpr int GA_UNROLL = 4;          // rows per thread in flight
constexpr int GA_PWMAX = 16384;       // positions per window, at most (128 KB of LDS sums)

__device__ __forceinline__ int ga_rows(const GlobalAlphaArgs& a, int u) {
  if (!a.unit_len) return a.len;
  const int n = a.unit_len[u];
  return n < 1 ? 1 : (n > a.len ? a.len : n);
}

// grid: (windows, sequences x groups); dynamic LDS: pw sums
__global__ void __launch_bounds__(GA_AT) ga_add_kernel(GlobalAlphaArgs a, uint64_t* part, int pw,
                                                       int ngrp) {
  extern __shared__ unsigned long long hist[];
  const int tid = threadIdx.x;
  const int y = a.y0 + blockIdx.y;
  const int b = y / ngrp, g = y - b * ngrp;
  const int p0 = blockIdx.x * pw;
  for (int i = tid; i < pw; i += GA_AT) hist[i] = 0ull;
  __syncthreads();
  const int u0 = b * a.per_seq + g * GA_UG;
  const int u1 = u0 + GA_UG < (b + 1) * a.per_seq ? u0 + GA_UG : (b + 1) * a.per_seq;
  for (int u = u0; u < u1; ++u) {
    const int L = ga_rows(a, u);
    const size_t ub = (size_t)u * a.cap;
    for (int r0 = tid; r0 < L; r0 += GA_UNROLL * GA_AT) {
      int p[GA_UNROLL];
      float al[GA_UNROLL];
#pragma unroll
      for (int k = 0; k < GA_UNROLL; ++k) {      // unconditional loads (clamped row)
        const int r = r0 + k * GA_AT;
        const size_t gi = ub + (r < L ? r : L - 1);
        p[k] = r < L ? a.pos[gi] : -1;
        al[k] = a.alpha[gi];
      }
#pragma unroll
      for (int k = 0; k < GA_UNROLL; ++k) {
        const int q = p[k] - p0;
        if (q >= 0 && q < pw && p[k] < a.T) {
          const float x = fminf(fmaxf(al[k], 0.0f), 1.0f);     // NaN -> 0
          atomicAdd(&hist[q], (unsigned long long)((double)x * GA_ONE + 0.5));
        }
      }
    }
  }
  __syncthreads();
  uint64_t* dst = part + ((size_t)b * ngrp + g) * a.T + p0;
  for (int i = tid; i < pw && p0 + i < a.T; i += GA_AT) dst[i] = hist[i];
}

__global__ void __launch_bounds__(GA_T) ga_sum_kernel(GlobalAlphaArgs a, const uint64_t* part,
                                                      int ngrp) {
  const size_t n = (size_t)(a.units / a.per_seq) * a.T;
  for (size_t i = (size_t)blockIdx.x * GA_T + threadIdx.x; i < n; i += (size_t)gridDim.x * GA_T) {
    const size_t b = i / a.T, p = i - b * a.T;
    const uint64_t* src = part + b * ngrp * a.T + p;
    uint64_t s = 0;
    for (int g = 0; g < ngrp; ++g) s += src[(size_t)g * a.T];
    a.acc[i] = s;
  }
}

__global__ void __launch_bounds__(GA_T) ga_write_kernel(GlobalAlphaArgs a) {
  const int u = a.y0 + blockIdx.y;
  const int L = ga_rows(a, u);
  const uint64_t* acc = a.acc + (size_t)(u / a.per_seq) * a.T;
  const double inv = 1.0 / (GA_ONE * (double)a.per_seq);
  for (int r = blockIdx.x * GA_T + threadIdx.x; r < L; r += gridDim.x * GA_T) {
    const size_t gi = (size_t)u * a.cap + r;
    const int p = a.pos[gi];
    if (p < 0 || p >= a.T) continue;
    a.alpha[gi] = (float)((double)acc[p] * inv);
  }
}

}  // namespace

int global_alpha_groups(int per_seq) { return (per_seq + GA_UG - 1) / GA_UG; }

int launch_global_alpha(const GlobalAlphaArgs& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int nseq = a.units / a.per_seq;
  const int ngrp = global_alpha_groups(a.per_seq);
  // a.acc: [nseq][T] sums, then [nseq][ngrp][T] partial sums
  uint64_t* part = a.acc + (size_t)nseq * a.T;
  const int nwin = (a.T + GA_PWMAX - 1) / GA_PWMAX;
  const int pw = ((a.T + nwin - 1) / nwin + 255) / 256 * 256;     // <= GA_PWMAX
  const int lds = pw * (int)sizeof(unsigned long long);
  hipFuncSetAttribute((const void*)ga_add_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  for_grid_y(nseq * ngrp, [&](int y0, int ny) {
    GlobalAlphaArgs b = a;
    b.y0 = y0;
    hipLaunchKernelGGL(ga_add_kernel, dim3(nwin, ny), dim3(GA_AT), lds, s, b, part, pw, ngrp);
  });
  const size_t n = (size_t)nseq * a.T;
  const size_t nb = (n + GA_T - 1) / GA_T;
  hipLaunchKernelGGL(ga_sum_kernel, dim3(nb < 8192 ? nb : 8192), dim3(GA_T), 0, s, a,
                     (const uint64_t*)part, ngrp);
  const int gx = (a.len + GA_T - 1) / GA_T;
  for_grid_y(a.units, [&](int y0, int ny) {
    GlobalAlphaArgs b = a;
    b.y0 = y0;
    hipLaunchKernelGGL(ga_write_kernel, dim3(gx < 64 ? gx : 64, ny), dim3(GA_T), 0, s, b);
  });
  return (int)hipGetLastError();
}

}  // namespace dc
