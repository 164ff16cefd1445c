// Rollout reward math of the REINFORCE update (Sec. 3.2), gfx950.
//
// For T decode steps and K sampled rollouts (row-major [T][K] arrays):
//   G[t][k] = R[t][k] + gamma G[t+1][k]            (discounted return, G[T] = 0)
//   b[t][k] = (sum_k' G[t][k'] - G[t][k]) / (K-1)    (leave-one-out, K >= 2)
//           = e                                      (EMA baseline, K = 1)
//   A = G - b,  H^ = -log pi,  w = -(A - beta) / (T K)
//   loss = -mean(log pi A + beta H^),  e <- d e + (1 - d) mean(G).
// Everything is float64 in one workgroup: a thread per rollout runs the
// backward scan, then a thread per step forms the baselines, then a fixed-order
// tree reduces the loss terms, so results are deterministic.  The arrays are
// small (T x K is a rollout's steps times its batch), so the kernel is a few
// microseconds of latency, not throughput.
#include <hip/hip_runtime.h>

#include "dc_kernels.hpp"

#pragma clang fp contract(off)

namespace dc {

namespace {

constexpr int RT = 256;

__global__ void __launch_bounds__(RT) reinforce_kernel(ReinforceArgs a) {
  __shared__ double red[3][RT];
  const int tid = threadIdx.x;
  const int T = a.steps, K = a.rollouts;
  const double ema0 = *a.ema;     // read before thread 0 rewrites it at the end
  for (int k = tid; k < K; k += RT) {
    double g = 0.0;
    for (int t = T - 1; t >= 0; --t) {
      g = (double)a.rewards[(size_t)t * K + k] + a.gamma * g;
      a.returns[(size_t)t * K + k] = g;
    }
  }
  __syncthreads();
  const double n = (double)T * (double)K;
  double lsum = 0.0, hsum = 0.0, gsum = 0.0;
  for (int t = tid; t < T; t += RT) {
    const double* G = a.returns + (size_t)t * K;
    double S = 0.0;
    for (int k = 0; k < K; ++k) S += G[k];
    gsum += S;
    for (int k = 0; k < K; ++k) {
      const size_t i = (size_t)t * K + k;
      const double b = K >= 2 ? (S - G[k]) / (double)(K - 1) : ema0;
      const double A = G[k] - b;
      const double lp = a.logp[i];
      lsum += lp * A + a.beta * -lp;
      hsum += -lp;
      if (a.baseline) a.baseline[i] = b;
      if (a.adv) a.adv[i] = A;
      if (a.weight) a.weight[i] = -(A - a.beta) / n;
    }
  }
  red[0][tid] = lsum;
  red[1][tid] = hsum;
  red[2][tid] = gsum;
  __syncthreads();
  for (int w = RT / 2; w > 0; w >>= 1) {
    if (tid < w)
      for (int j = 0; j < 3; ++j) red[j][tid] += red[j][tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    const double mean_g = red[2][0] / n;
    if (a.stats) {
      a.stats[0] = -red[0][0] / n;   // loss
      a.stats[1] = red[1][0] / n;    // mean entropy surrogate
      a.stats[2] = mean_g;           // mean return
    }
    *a.ema = a.ema_decay * ema0 + (1.0 - a.ema_decay) * mean_g;
  }
}

}  // namespace

int launch_reinforce(const ReinforceArgs& a, void* stream) {
  hipLaunchKernelGGL(reinforce_kernel, dim3(1), dim3(RT), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

}  // namespace dc
