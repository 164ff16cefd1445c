// Decode attention fused with the eviction-feature update (gfx950).
//
// One decode step of one unit (Algorithm 1 forward pass + feature extraction):
//   s_{j,i} = scale * q_j . k_i,  a_j = softmax(s_j),  o_j = sum_i a_{j,i} v_i,
//   H_j = -sum_i a_{j,i} ln a_{j,i}                      (entropy of query j)
//   alpha_i += (1/G) sum_j a_{j,i}                        (cumulative attention)
//   den_i += sum_j a_{j,i} - [retired step],  num_i += sum_j a_{j,i} H_j - [retired step]
// where the retired step is the one leaving the w-step entropy window; its
// weights are recomputed from the query ring with exactly the arithmetic that
// added them, so the window sums stay exact to binary64 rounding.
//
// Layout of the work: K and V are streamed once, 16 bytes per lane, one row per
// LPR-lane group (LPR = 16 for bf16 d=128).  Each group keeps an online softmax
// (m, l, and u = sum p (s - m) for the entropy) and a partial output; logits,
// retired contributions and value norms go to LDS (unit path, one workgroup per
// unit) or to the workspace (chunked path, several workgroups per unit) so that
// the feature pass after the softmax reduction never touches K/V again.
#include "dc_device.hpp"
#include "dc_kernels.hpp"

#pragma clang fp contract(off)

namespace dc {

constexpr int NTH = 1024;             // threads per workgroup
constexpr int NWAVE = NTH / 64;
constexpr int CHUNK = 2048;           // rows per workgroup on the chunked path
constexpr int LDS_LIMIT = 160 * 1024;

template <int DTYPE, int D, int G>
struct Geo {
  using R = RowT<DTYPE, D>;
  static constexpr int ELT = R::ELT, EPL = R::EPL, LPR = R::LPR;
  static constexpr int NG = NTH / LPR;      // row groups per workgroup
  static constexpr int PART = 3 * G + G * D;  // floats in one softmax partial
};

template <int G, int EPL>
struct Acc {
  float m[G], l[G], u[G];
  float o[G][EPL];
};

// ---------------------------------------------------------------- phase A
// Stream rows [r0, r1) of unit u: logits, retired contributions, value norms to
// the sinks (index i - sink0), online softmax into acc.
template <int DTYPE, int D, int G, bool FEAT, bool LDS_SINK>
__device__ __forceinline__ void phase_a(const DecodeArgs& a, int u, int r0, int r1, float* s_sink,
                                        float* r_sink, float* v_sink, int sink0,
                                        Acc<G, Geo<DTYPE, D, G>::EPL>& acc) {
  using Q = Geo<DTYPE, D, G>;
  constexpr int EPL = Q::EPL, LPR = Q::LPR, NG = Q::NG, ELT = Q::ELT;
  constexpr int PF = 2;
  const int tid = threadIdx.x, grp = tid / LPR, lam = tid % LPR;
  const char* kc = (const char*)a.k + (size_t)u * a.cap * D * ELT;
  const char* vc = (const char*)a.v + (size_t)u * a.cap * D * ELT;
  const char* kn = a.append ? (const char*)a.k_new + (size_t)u * D * ELT : nullptr;
  const char* vn = a.append ? (const char*)a.v_new + (size_t)u * D * ELT : nullptr;
  const int newrow = a.append ? a.len_old : -1;

  uint4 qs[G];
  const char* qp = (const char*)a.q + (size_t)u * G * D * ELT;
#pragma unroll
  for (int j = 0; j < G; ++j) qs[j] = ldg16(qp + (size_t)j * D * ELT + lam * 16);

  uint4 qr[G];
  float mret[G], ilret[G], hret[G];
  const bool retire = FEAT && a.retire;
  if (retire) {
    const char* rp = (const char*)a.qring + ((size_t)u * a.window + a.slot) * G * D * ELT;
    const float* st = a.qstat + ((size_t)u * a.window + a.slot) * G * 3;
#pragma unroll
    for (int j = 0; j < G; ++j) {
      qr[j] = ldg16(rp + (size_t)j * D * ELT + lam * 16);
      mret[j] = st[3 * j];
      ilret[j] = st[3 * j + 1];
      hret[j] = st[3 * j + 2];
    }
  }

#pragma unroll
  for (int j = 0; j < G; ++j) {
    acc.m[j] = NEG_BIG;
    acc.l[j] = 0.0f;
    acc.u[j] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc.o[j][e] = 0.0f;
  }

  auto kptr = [&](int i) { return i == newrow ? kn : kc + (size_t)i * D * ELT; };
  auto vptr = [&](int i) { return i == newrow ? vn : vc + (size_t)i * D * ELT; };

  uint4 kb[PF], vb[PF];
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    int row = r0 + grp + p * NG;
    if (row < r1) {
      kb[p] = ldg16_nt(kptr(row) + lam * 16);
      vb[p] = ldg16_nt(vptr(row) + lam * 16);
    }
  }

  for (int base = r0 + grp; base < r1; base += PF * NG) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int row = base + p * NG;
      if (row < r1) {
        const uint4 kv = kb[p], vv = vb[p];
        const int nrow = row + PF * NG;
        if (nrow < r1) {
          kb[p] = ldg16_nt(kptr(nrow) + lam * 16);
          vb[p] = ldg16_nt(vptr(nrow) + lam * 16);
        }
        float s[G];
#pragma unroll
        for (int j = 0; j < G; ++j) s[j] = row_sum<LPR>(dot_slice<DTYPE>(qs[j], kv)) * a.scale;
        float vf[EPL];
        unpack_slice<DTYPE>(vv, vf);
        if constexpr (FEAT) {
          const int si = row - sink0;
          if (retire) {
            float sr[G];
#pragma unroll
            for (int j = 0; j < G; ++j) sr[j] = row_sum<LPR>(dot_slice<DTYPE>(qr[j], kv)) * a.scale;
            float cz, cn;
            row_contrib<G>(sr, mret, ilret, hret, cz, cn);
            if (lam == 0) {
              r_sink[2 * si] = cz;
              r_sink[2 * si + 1] = cn;
            }
          }
          float v2 = vf[0] * vf[0];
#pragma unroll
          for (int e = 1; e < EPL; ++e) v2 = __builtin_fmaf(vf[e], vf[e], v2);
          v2 = row_sum<LPR>(v2);
          if (lam == 0) {
            v_sink[si] = __builtin_sqrtf(v2);
#pragma unroll
            for (int j = 0; j < G; ++j) s_sink[si * G + j] = s[j];
          }
        }
#pragma unroll
        for (int j = 0; j < G; ++j) {
          const float mn = fmaxf(acc.m[j], s[j]);
          if (mn > acc.m[j]) {
            const float dm = acc.m[j] - mn;
            const float c = __builtin_amdgcn_exp2f(dm * LOG2E);
            acc.u[j] = c * (acc.u[j] + dm * acc.l[j]);
            acc.l[j] = acc.l[j] * c;
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc.o[j][e] = acc.o[j][e] * c;
            acc.m[j] = mn;
          }
          const float d = s[j] - acc.m[j];
          const float p = __builtin_amdgcn_exp2f(d * LOG2E);
          acc.l[j] = acc.l[j] + p;
          acc.u[j] = acc.u[j] + p * d;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc.o[j][e] = __builtin_fmaf(p, vf[e], acc.o[j][e]);
        }
      }
    }
  }
}

// Merge two softmax partials (m, l, u, o) into the first.
__device__ __forceinline__ void merge_stats(float& m, float& l, float& u, float mo, float lo,
                                            float uo, float& c1, float& c2) {
  const float mn = fmaxf(m, mo);
  c1 = __builtin_amdgcn_exp2f((m - mn) * LOG2E);
  c2 = __builtin_amdgcn_exp2f((mo - mn) * LOG2E);
  u = c1 * (u + (m - mn) * l) + c2 * (uo + (mo - mn) * lo);
  l = c1 * l + c2 * lo;
  m = mn;
}

// Combine the row groups of one wave (all lanes end with the wave's partial).
template <int G, int EPL, int LPR>
__device__ __forceinline__ void wave_combine(Acc<G, EPL>& acc) {
#pragma unroll
  for (int off = LPR; off < 64; off *= 2) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const float mo = __shfl_xor(acc.m[j], off), lo = __shfl_xor(acc.l[j], off),
                  uo = __shfl_xor(acc.u[j], off);
      float c1, c2;
      merge_stats(acc.m[j], acc.l[j], acc.u[j], mo, lo, uo, c1, c2);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float oo = __shfl_xor(acc.o[j][e], off);
        acc.o[j][e] = c1 * acc.o[j][e] + c2 * oo;
      }
    }
  }
}

// Combine the waves of a workgroup.  On return every thread holds the final
// (m, l, u) per head in fm/fl/fu, and its wave's rescale factor cw[j]; stat is
// LDS scratch of NWAVE * 3G + 3G floats.  A few threads merge the per-wave
// partials (fixed order) and broadcast the result through LDS.
template <int G>
__device__ __forceinline__ void block_stats(float (&m)[G], float (&l)[G], float (&u)[G],
                                            float* stat, float (&fm)[G], float (&fl)[G],
                                            float (&fu)[G], float (&cw)[G]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      stat[(wave * G + j) * 3 + 0] = m[j];
      stat[(wave * G + j) * 3 + 1] = l[j];
      stat[(wave * G + j) * 3 + 2] = u[j];
    }
  }
  __syncthreads();
  if (threadIdx.x < G) {
    const int j = threadIdx.x;
    float M = stat[j * 3], Lx = stat[j * 3 + 1], U = stat[j * 3 + 2];
    for (int w = 1; w < NWAVE; ++w) {
      float c1, c2;
      merge_stats(M, Lx, U, stat[(w * G + j) * 3], stat[(w * G + j) * 3 + 1],
                  stat[(w * G + j) * 3 + 2], c1, c2);
    }
    stat[NWAVE * 3 * G + 3 * j] = M;
    stat[NWAVE * 3 * G + 3 * j + 1] = Lx;
    stat[NWAVE * 3 * G + 3 * j + 2] = U;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < G; ++j) {
    fm[j] = stat[NWAVE * 3 * G + 3 * j];
    fl[j] = stat[NWAVE * 3 * G + 3 * j + 1];
    fu[j] = stat[NWAVE * 3 * G + 3 * j + 2];
    cw[j] = __builtin_amdgcn_exp2f((m[j] - fm[j]) * LOG2E);
  }
}

template <int G>
__device__ __forceinline__ void final_head_stats(const float (&fl)[G], const float (&fu)[G],
                                                 float (&invl)[G], float (&H)[G]) {
#pragma unroll
  for (int j = 0; j < G; ++j) {
    invl[j] = 1.0f / fl[j];
    H[j] = __logf(fl[j]) - fu[j] * invl[j];
  }
}

// Feature update of rows [r0, r1) (thread per row), logits/retired/vnorm from
// the sinks at index i - sink0.
template <int G>
__device__ __forceinline__ void phase_d(const DecodeArgs& a, int u, int r0, int r1,
                                        const float* s_src, const float* r_src,
                                        const float* v_src, int sink0, const float (&M)[G],
                                        const float (&invl)[G], const float (&H)[G]) {
  const size_t ub = (size_t)u * a.cap;
  const int newrow = a.append ? a.len_old : -1;
  constexpr float invG = 1.0f / G;
  for (int i = r0 + threadIdx.x; i < r1; i += NTH) {
    const int si = i - sink0;
    float w[G];
#pragma unroll
    for (int j = 0; j < G; ++j) w[j] = attn_weight(s_src[si * G + j], M[j], invl[j]);
    float cz, cn;
    contrib_from_weights<G>(w, H, cz, cn);
    const size_t gi = ub + i;
    if (a.sigma) a.sigma[gi] = head_variance<G>(w);
    if (i == newrow) {
      a.alpha[gi] = cz * invG;
      a.den[gi] = (double)cz;
      a.num[gi] = (double)cn;
      a.pos[gi] = a.T - 1;
    } else {
      a.alpha[gi] = (a.arec ? 0.0f : a.alpha[gi]) + cz * invG;
      double z = a.den[gi] + (double)cz;
      double n = a.num[gi] + (double)cn;
      if (a.retire && a.pos[gi] <= a.pmax_ret) {
        z = z - (double)r_src[2 * si];
        n = n - (double)r_src[2 * si + 1];
      }
      a.den[gi] = z;
      a.num[gi] = n;
    }
    a.vnorm[gi] = v_src[si];
  }
}

template <int DTYPE>
__device__ __forceinline__ void store_elem(void* base, size_t idx, float x) {
  if constexpr (DTYPE == 1) ((uint16_t*)base)[idx] = (uint16_t)f32_to_bf16_bits(x);
  else ((float*)base)[idx] = x;
}

// Append the new key/value rows to slot len_old (read back only from k_new/v_new
// within the step, so no intra-kernel ordering is needed).
template <int DTYPE, int D>
__device__ __forceinline__ void write_append(const DecodeArgs& a, int u) {
  constexpr int ELT = DTYPE == 0 ? 4 : 2;
  constexpr int N16 = D * ELT / 16;
  const int t = threadIdx.x;
  if (t < 2 * N16) {
    const bool isv = t >= N16;
    const int c = isv ? t - N16 : t;
    const char* src = (const char*)(isv ? a.v_new : a.k_new) + (size_t)u * D * ELT;
    char* dst = (char*)(isv ? a.v : a.k) + ((size_t)u * a.cap + a.len_old) * D * ELT;
    *reinterpret_cast<uint4*>(dst + c * 16) = ldg16(src + c * 16);
  }
}

// Record this step's queries and statistics in the ring slot.
template <int DTYPE, int D, int G>
__device__ __forceinline__ void write_ring(const DecodeArgs& a, int u, const float (&M)[G],
                                           const float (&invl)[G], const float (&H)[G]) {
  constexpr int ELT = DTYPE == 0 ? 4 : 2;
  constexpr int N16 = G * D * ELT / 16;
  const int t = threadIdx.x;
  const size_t rs = (size_t)u * a.window + a.slot;
  if (t < N16) {
    const char* src = (const char*)a.q + (size_t)u * G * D * ELT;
    char* dst = (char*)a.qring + rs * G * D * ELT;
    *reinterpret_cast<uint4*>(dst + t * 16) = ldg16(src + t * 16);
  }
  if (t < G) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      if (j == t) {
        a.qstat[(rs * G + j) * 3 + 0] = M[j];
        a.qstat[(rs * G + j) * 3 + 1] = invl[j];
        a.qstat[(rs * G + j) * 3 + 2] = H[j];
      }
    }
  }
}

// ---------------------------------------------------------------- unit path
// One workgroup per unit; logits, retired contributions and value norms of all
// L rows live in LDS.
template <int DTYPE, int D, int G, bool FEAT>
__global__ void __launch_bounds__(NTH) decode_unit_kernel(DecodeArgs a) {
  using Q = Geo<DTYPE, D, G>;
  extern __shared__ float lds[];
  const int u = blockIdx.x;
  float* stat = lds;                          // NWAVE * 3G + 3G
  float* sbuf = lds + NWAVE * 3 * G + 3 * G;  // L * G
  float* rbuf = sbuf + (FEAT ? a.L * G : 0);  // L * 2
  float* vbuf = rbuf + (FEAT ? a.L * 2 : 0);  // L
  float* obuf = sbuf;                         // NWAVE * G * D, after the feature pass

  if (FEAT && a.append) write_append<DTYPE, D>(a, u);
  Acc<G, Q::EPL> acc;
  phase_a<DTYPE, D, G, FEAT, true>(a, u, 0, a.L, sbuf, rbuf, vbuf, 0, acc);
  wave_combine<G, Q::EPL, Q::LPR>(acc);
  float fm[G], fl[G], fu[G], cw[G], invl[G], H[G];
  block_stats<G>(acc.m, acc.l, acc.u, stat, fm, fl, fu, cw);
  final_head_stats<G>(fl, fu, invl, H);
  if constexpr (FEAT) phase_d<G>(a, u, 0, a.L, sbuf, rbuf, vbuf, 0, fm, invl, H);
  __syncthreads();
  // output: sum of the rescaled wave partials
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane < Q::LPR) {
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < Q::EPL; ++e)
        obuf[(wave * G + j) * D + lane * Q::EPL + e] = acc.o[j][e] * cw[j];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < G * D; t += NTH) {
    const int j = t / D;
    float o = 0.0f;
    for (int w = 0; w < NWAVE; ++w) o = o + obuf[w * G * D + t];
    float il = invl[0];
#pragma unroll
    for (int jj = 1; jj < G; ++jj) il = (jj == j) ? invl[jj] : il;
    store_elem<DTYPE>(a.out, (size_t)u * G * D + t, o * il);
  }
  if (!FEAT && a.append) write_append<DTYPE, D>(a, u);
  if (FEAT && a.window > 0) write_ring<DTYPE, D, G>(a, u, fm, invl, H);
}

// ---------------------------------------------------------------- chunked path
// Pass 1: workgroup (chunk c, unit u) streams rows [c*CHUNK, ...), writes logits /
// retired contributions / value norms to the workspace and its softmax partial.
template <int DTYPE, int D, int G, bool FEAT>
__global__ void __launch_bounds__(NTH) decode_split1_kernel(DecodeArgs a) {
  using Q = Geo<DTYPE, D, G>;
  __shared__ float lds[NWAVE * 3 * G + 3 * G + NWAVE * G * D];
  float* stat = lds;
  float* obuf = lds + NWAVE * 3 * G + 3 * G;
  const int c = blockIdx.x, u = a.y0 + blockIdx.y;
  const int r0 = c * a.chunk, r1 = min(a.L, r0 + a.chunk);
  if (c == 0 && a.append) write_append<DTYPE, D>(a, u);
  float* s_sink = FEAT ? a.ws_s + (size_t)u * a.lmax * G : nullptr;
  float* r_sink = FEAT ? a.ws_r + (size_t)u * a.lmax * 2 : nullptr;
  float* v_sink = FEAT ? a.ws_v + (size_t)u * a.lmax : nullptr;
  Acc<G, Q::EPL> acc;
  phase_a<DTYPE, D, G, FEAT, false>(a, u, r0, r1, s_sink, r_sink, v_sink, 0, acc);
  wave_combine<G, Q::EPL, Q::LPR>(acc);
  float fm[G], fl[G], fu[G], cw[G];
  block_stats<G>(acc.m, acc.l, acc.u, stat, fm, fl, fu, cw);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane < Q::LPR) {
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < Q::EPL; ++e)
        obuf[(wave * G + j) * D + lane * Q::EPL + e] = acc.o[j][e] * cw[j];
  }
  __syncthreads();
  float* part = a.ws_part + ((size_t)u * a.nchunks + c) * Q::PART;
  for (int t = threadIdx.x; t < G * D; t += NTH) {
    float o = 0.0f;
    for (int w = 0; w < NWAVE; ++w) o = o + obuf[w * G * D + t];
    part[3 * G + t] = o;
  }
  if (threadIdx.x < G) {
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (j == (int)threadIdx.x) {
        part[3 * j] = fm[j];
        part[3 * j + 1] = fl[j];
        part[3 * j + 2] = fu[j];
      }
  }
}

// Pass 2: workgroup (chunk c, unit u) merges the unit's partials, updates the
// features of its chunk; chunk 0 also writes the output and the ring slot.
template <int DTYPE, int D, int G, bool FEAT>
__global__ void __launch_bounds__(NTH) decode_split2_kernel(DecodeArgs a) {
  using Q = Geo<DTYPE, D, G>;
  const int c = blockIdx.x, u = a.y0 + blockIdx.y;
  const float* parts = a.ws_part + (size_t)u * a.nchunks * Q::PART;
  float fm[G], fl[G], fu[G], invl[G], H[G];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    float M = parts[3 * j], Lx = parts[3 * j + 1], U = parts[3 * j + 2];
    for (int cc = 1; cc < a.nchunks; ++cc) {
      const float* p = parts + (size_t)cc * Q::PART;
      float c1, c2;
      merge_stats(M, Lx, U, p[3 * j], p[3 * j + 1], p[3 * j + 2], c1, c2);
    }
    fm[j] = M;
    fl[j] = Lx;
    fu[j] = U;
  }
  final_head_stats<G>(fl, fu, invl, H);
  if constexpr (FEAT) {
    const int r0 = c * a.chunk, r1 = min(a.L, r0 + a.chunk);
    phase_d<G>(a, u, r0, r1, a.ws_s + (size_t)u * a.lmax * G, a.ws_r + (size_t)u * a.lmax * 2,
               a.ws_v + (size_t)u * a.lmax, 0, fm, invl, H);
  }
  if (c != 0) return;
  for (int t = threadIdx.x; t < G * D; t += NTH) {
    const int j = t / D;
    float M = fm[0], il = invl[0];
#pragma unroll
    for (int jj = 1; jj < G; ++jj) {
      M = (jj == j) ? fm[jj] : M;
      il = (jj == j) ? invl[jj] : il;
    }
    float o = 0.0f;
    for (int cc = 0; cc < a.nchunks; ++cc) {
      const float* p = parts + (size_t)cc * Q::PART;
      o = o + p[3 * G + t] * __builtin_amdgcn_exp2f((p[3 * j] - M) * LOG2E);
    }
    store_elem<DTYPE>(a.out, (size_t)u * G * D + t, o * il);
  }
  if (FEAT && a.window > 0) write_ring<DTYPE, D, G>(a, u, fm, invl, H);
}

// ---------------------------------------------------------------- feature init
template <int DTYPE, int D>
__global__ void __launch_bounds__(256) feat_init_kernel(DecodeArgs a, int first_pos) {
  using R = RowT<DTYPE, D>;
  constexpr int LPR = R::LPR, EPL = R::EPL, ELT = R::ELT;
  const int u = a.y0 + blockIdx.y;
  const int grp = (blockIdx.x * 256 + threadIdx.x) / LPR, lam = threadIdx.x % LPR;
  const int ngrp = gridDim.x * 256 / LPR;
  for (int i = grp; i < a.L; i += ngrp) {
    const size_t gi = (size_t)u * a.cap + i;
    float vf[EPL];
    unpack_slice<DTYPE>(ldg16((const char*)a.v + gi * D * ELT + lam * 16), vf);
    float v2 = vf[0] * vf[0];
#pragma unroll
    for (int e = 1; e < EPL; ++e) v2 = __builtin_fmaf(vf[e], vf[e], v2);
    v2 = row_sum<LPR>(v2);
    if (lam == 0) {
      a.vnorm[gi] = __builtin_sqrtf(v2);
      a.alpha[gi] = 0.0f;
      if (a.sigma) a.sigma[gi] = 0.0f;
      a.num[gi] = 0.0;
      a.den[gi] = 0.0;
      a.pos[gi] = first_pos + i;
    }
  }
}

// ---------------------------------------------------------------- dispatch
size_t decode_lds_bytes(int L, int G, int D, bool feat) {
  size_t stat = (size_t)NWAVE * 3 * G + 3 * G;
  size_t rows = feat ? (size_t)L * (G + 3) : 0;
  size_t ob = (size_t)NWAVE * G * D;
  return (stat + (rows > ob ? rows : ob)) * sizeof(float);
}

bool decode_fits_lds(int L, int G, int D) { return decode_lds_bytes(L, G, D, true) <= LDS_LIMIT; }

int decode_chunk_rows() { return CHUNK; }

template <int DTYPE, int D, int G>
static int launch_t(const DecodeArgs& a, bool feat, bool split, hipStream_t s) {
  if (!split) {
    size_t lds = decode_lds_bytes(a.L, G, D, feat);
    if (feat) {
      auto k = decode_unit_kernel<DTYPE, D, G, true>;
      hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hipLaunchKernelGGL(k, dim3(a.units), dim3(NTH), lds, s, a);
    } else {
      auto k = decode_unit_kernel<DTYPE, D, G, false>;
      hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hipLaunchKernelGGL(k, dim3(a.units), dim3(NTH), lds, s, a);
    }
  } else {
    // every slice of pass 1 before pass 2 (stream order)
    for_grid_y(a.units, [&](int y0, int ny) {
      DecodeArgs b = a;
      b.y0 = y0;
      if (feat) hipLaunchKernelGGL((decode_split1_kernel<DTYPE, D, G, true>), dim3(a.nchunks, ny), dim3(NTH), 0, s, b);
      else hipLaunchKernelGGL((decode_split1_kernel<DTYPE, D, G, false>), dim3(a.nchunks, ny), dim3(NTH), 0, s, b);
    });
    for_grid_y(a.units, [&](int y0, int ny) {
      DecodeArgs b = a;
      b.y0 = y0;
      if (feat) hipLaunchKernelGGL((decode_split2_kernel<DTYPE, D, G, true>), dim3(a.nchunks, ny), dim3(NTH), 0, s, b);
      else hipLaunchKernelGGL((decode_split2_kernel<DTYPE, D, G, false>), dim3(a.nchunks, ny), dim3(NTH), 0, s, b);
    });
  }
  return (int)hipGetLastError();
}

template <int DTYPE, int D>
static int launch_g(const DecodeArgs& a, int G, bool feat, bool split, hipStream_t s) {
  switch (G) {
    case 1: return launch_t<DTYPE, D, 1>(a, feat, split, s);
    case 2: return launch_t<DTYPE, D, 2>(a, feat, split, s);
    case 4: return launch_t<DTYPE, D, 4>(a, feat, split, s);
    case 8: return launch_t<DTYPE, D, 8>(a, feat, split, s);
  }
  return (int)hipErrorInvalidValue;
}

int launch_decode(const DecodeArgs& a, int dtype, int D, int G, bool feat, bool split,
                  void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (dtype == 1 && D == 128) return launch_g<1, 128>(a, G, feat, split, s);
  if (dtype == 1 && D == 64) return launch_g<1, 64>(a, G, feat, split, s);
  if (dtype == 0 && D == 128) return launch_g<0, 128>(a, G, feat, split, s);
  if (dtype == 0 && D == 64) return launch_g<0, 64>(a, G, feat, split, s);
  return (int)hipErrorInvalidValue;
}

int launch_feat_init(const DecodeArgs& a, int dtype, int D, int first_pos, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  int gx = (a.L + 255) / 256;
  if (gx > 64) gx = 64;
  if (gx < 1) gx = 1;
  if (!((dtype == 0 || dtype == 1) && (D == 64 || D == 128))) return (int)hipErrorInvalidValue;
  for_grid_y(a.units, [&](int y0, int ny) {
    DecodeArgs b = a;
    b.y0 = y0;
    const dim3 grid(gx, ny);
    if (dtype == 1 && D == 128) hipLaunchKernelGGL((feat_init_kernel<1, 128>), grid, dim3(256), 0, s, b, first_pos);
    else if (dtype == 1 && D == 64) hipLaunchKernelGGL((feat_init_kernel<1, 64>), grid, dim3(256), 0, s, b, first_pos);
    else if (dtype == 0 && D == 128) hipLaunchKernelGGL((feat_init_kernel<0, 128>), grid, dim3(256), 0, s, b, first_pos);
    else hipLaunchKernelGGL((feat_init_kernel<0, 64>), grid, dim3(256), 0, s, b, first_pos);
  });
  return (int)hipGetLastError();
}

}  // namespace dc
