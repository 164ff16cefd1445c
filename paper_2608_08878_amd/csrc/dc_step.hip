// Decode step for bfloat16 caches on gfx950 matrix cores, optionally fused with
// scoring, top-B selection and compaction (the whole of one Algorithm 1 step).
//
// Per unit (G query heads sharing one KV head, head_dim D):
//   pass A  stream K once.  One v_mfma_f32_16x16x32_bf16 chain per 16 keys gives
//           the logits of up to 16 query rows: rows 0..G-1 are this step's
//           queries, rows 8..8+G-1 the queries of the step leaving the entropy
//           window (from the ring), so the retired weights come out of the same
//           instructions that produced them w steps ago.  Logits s = scale q.k
//           go to LDS, the retired contributions are reduced per key.
//   pass P  with the block-wide max M_j: p = exp(s - M) (stored over s),
//           l_j = sum p, u_j = sum p (s - M);  H_j = ln l_j - u_j / l_j.
//   pass B  stream V once: o_j = sum_i p_ji v_i (fp32), one 16-lane group per row.
//   pass D  features per key (thread per key): alpha += mean_j a_ji,
//           den += sum_j a_ji - retired, num += sum_j a_ji H_j - retired,
//           a_ji = p_ji / l_j; with eviction fused, the policy score and the
//           64-bit ranking key of every row are formed here and the unit is
//           compacted before the workgroup exits.
// Caches too long for LDS use the chunked form of the same passes (two
// kernels, logits in the workspace).
#include "dc_select.hpp"

#pragma clang fp contract(off)

namespace dc {

constexpr int SNT = 512;              // threads per workgroup (two workgroups per CU)
constexpr int SNW = SNT / 64;
constexpr int SCHUNK = 2048;          // rows per workgroup on the chunked path
constexpr int S_KMAX = 10;            // fused step: row slots per thread (L <= 5120)
constexpr int S_LDS = 160 * 1024 - 4 * 1024;  // dynamic LDS budget (static LDS aside)

template <int D>
struct MG {
  static constexpr int NT = D / 32;   // MFMA k-steps per 16-key tile
  static constexpr int LB = D / 2;    // bytes of a key row one lane loads
  static constexpr int LPR = D / 8;   // lanes per row in the value pass (16 bytes each)
};

__device__ __forceinline__ float max16(float x) {
  x = fmaxf(x, dpp<DPP_XOR1>(x));
  x = fmaxf(x, dpp<DPP_XOR2>(x));
  x = fmaxf(x, dpp<DPP_HALF_MIRROR>(x));
  x = fmaxf(x, dpp<DPP_MIRROR>(x));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// A-operand fragments: lane l holds row i = l & 15 and, for MFMA t, the 8 dims
// of 16-byte chunk 4t + g (g = l >> 4) of that row.  The key rows are read
// with the same chunk assignment (so each load instruction covers 64
// contiguous bytes of 16 rows); which dims a lane contributes to an MFMA's
// reduction is free as long as both operands agree.  Rows 0..G-1 hold the
// current queries, rows 8..8+G-1 the retiring queries, other rows zero.
template <int D, int G>
__device__ __forceinline__ void load_qfrag(uint4 (&qa)[MG<D>::NT], const DecodeArgs& a, int u,
                                           bool retire) {
  const int lane = threadIdx.x & 63, i = lane & 15, g = lane >> 4;
  const char* src = nullptr;
  if (i < G) src = (const char*)a.q + ((size_t)u * G + i) * D * 2;
  else if (retire && i >= 8 && i < 8 + G)
    src = (const char*)a.qring + (((size_t)u * a.window + a.slot) * G + (i - 8)) * D * 2;
#pragma unroll
  for (int t = 0; t < MG<D>::NT; ++t)
    qa[t] = src ? ldg16(src + 16 * (4 * t + g)) : make_uint4(0, 0, 0, 0);
}

// Retiring step's statistics (uniform over the workgroup).
template <int G>
struct RetStats {
  float m[G], il[G], h[G];
};

template <int G>
__device__ __forceinline__ void load_ret(RetStats<G>& r, const DecodeArgs& a, int u) {
  const float* st = a.qstat + ((size_t)u * a.window + a.slot) * G * 3;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    r.m[j] = st[3 * j];
    r.il[j] = st[3 * j + 1];
    r.h[j] = st[3 * j + 2];
  }
}

// ---------------------------------------------------------------- pass A
// Rows [r0, r1) of unit u in 16-key tiles.  Logits of the current heads go to
// s_sink[(i - sink0) * RS + j], running maxima per current head into mrun.  The
// retired contributions (z, n) of each key are either stored to
// r_sink[2 (i - sink0)] (tiles round-robin over the waves; chunked path) or, with
// GROUPED, kept in registers: rows then go in groups of 64 (four tiles), group
// b to wave b mod SNW, and after a group lane l of the wave holds the pair of
// the group's row l, in zr[k] / nr[k] for the wave's k-th group.
constexpr int S_GMAX = S_KMAX;        // 64-row groups per wave, at most (L <= 5120)

// Rows of unit u before this step (per unit for ragged caches).
// (Device lengths are clamped to [0, len_old], the host's bound, so that a bad
// value cannot take an access out of the buffers.)
__device__ __forceinline__ int len_old_of(const DecodeArgs& a, int u) {
  if (!a.unit_len) return a.len_old;
  const int n = a.unit_len[u];
  return n < 0 ? 0 : n > a.len_old ? a.len_old : n;
}

template <int D, int G, bool FEAT, bool GROUPED, int RS = G>
__device__ __forceinline__ void pass_a(const DecodeArgs& a, int u, int r0, int r1, float* s_sink,
                                       float* r_sink, int sink0, const uint4 (&qa)[MG<D>::NT],
                                       bool retire, const RetStats<G>& rs, float (&mrun)[4],
                                       float (&zr)[S_GMAX], float (&nr)[S_GMAX]) {
  constexpr int NT = MG<D>::NT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, i = lane & 15, g = lane >> 4;
  const char* kc = (const char*)a.k + (size_t)u * a.cap * D * 2;
  const char* kn = a.append ? (const char*)a.k_new + (size_t)u * D * 2 : nullptr;
  const int newrow = a.append ? len_old_of(a, u) : -1;
  const int ntiles = (r1 - r0 + 15) / 16;
#pragma unroll
  for (int r = 0; r < 4; ++r) mrun[r] = NEG_BIG;
  auto clamp_tile = [&](int t) { return t < ntiles ? t : ntiles - 1; };
  auto load_tile = [&](int tile, uint4 (&kb)[NT]) {
    int key = r0 + tile * 16 + i;
    key = key < r1 ? key : r1 - 1;
    const char* kp = key == newrow ? kn : kc + (size_t)key * D * 2;
    // plain loads: instructions t and t+1 read the two halves of the same 128-byte
    // line, so the second one should find it in the vector L1
#pragma unroll
    for (int t = 0; t < NT; ++t) kb[t] = ldg16(kp + 16 * (4 * t + g));
  };
  // logits of tile tt; returns the retired pair of key (tile row i) in lanes
  // 32 + i (zero elsewhere or without a retiring step)
  auto process = [&](int tt, const uint4 (&kb)[NT], float& z, float& n) {
    f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int t = 0; t < NT; ++t)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, qa[t]),
                                                    __builtin_bit_cast(bf16x8_t, kb[t]), acc, 0,
                                                    0, 0);
    const int key = r0 + tt * 16 + i;
    const bool valid = key < r1;
    float s[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) s[r] = acc[r] * a.scale;
    // rows 4g + r: current heads in groups g < 2, retiring heads in groups 2, 3
    if (4 * g < G && valid) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (4 * g + r < G) mrun[r] = fmaxf(mrun[r], s[r]);
      float* dst = s_sink + (size_t)(key - sink0) * RS + 4 * g;
      if constexpr (G >= 4) {
        *reinterpret_cast<f32x4_t*>(dst) = f32x4_t{s[0], s[1], s[2], s[3]};
      } else {
#pragma unroll
        for (int r = 0; r < G; ++r) dst[r] = s[r];
      }
    }
    z = 0.0f;
    n = 0.0f;
    if constexpr (FEAT) {
      if (retire && g >= 2 && 4 * (g - 2) < G) {
        const bool hi = G > 4 && g == 3;        // heads 4..7 (only when G == 8)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          constexpr int last = G - 1;
          const int jl = r < G ? r : last, jh = 4 + r < G ? 4 + r : last;
          if ((hi ? 4 + r : r) < G) {
            const float mm = hi ? rs.m[jh] : rs.m[jl];
            const float il = hi ? rs.il[jh] : rs.il[jl];
            const float hh = hi ? rs.h[jh] : rs.h[jl];
            const float w = attn_weight(s[r], mm, il);
            z = z + w;
            n = n + w * hh;
          }
        }
      }
      if constexpr (G > 4) {     // heads 4..7 live in group 3: add the blocks in order
        const float z1 = __shfl_down(z, 16), n1 = __shfl_down(n, 16);
        z = z + z1;
        n = n + n1;
      }
    }
  };
  // Two tiles in flight per wave: consume a buffer, then refill it.  Every load
  // is issued unconditionally (a tile past the end re-reads the last tile, which
  // the cache serves), so the wait before a tile's MFMAs covers only that
  // tile's loads and never drains the other buffer.
  if constexpr (GROUPED) {
    const int ngrp = (ntiles + 3) / 4;
    const int ngw = wave < ngrp ? (ngrp - 1 - wave) / SNW + 1 : 0;
#pragma unroll
    for (int k = 0; k < S_GMAX; ++k) {
      zr[k] = 0.0f;
      nr[k] = 0.0f;
    }
    if (ngw > 0) {
      uint4 kb0[NT], kb1[NT];
      load_tile(4 * wave, kb0);
      load_tile(clamp_tile(4 * wave + 1), kb1);
      for (int k = 0; k < ngw; ++k) {
        const int t0 = 4 * (wave + SNW * k), tn = t0 + 4 * SNW;
        float zz = 0.0f, nn = 0.0f;
        // tile j's pairs (lanes 32..47) move to lanes 16 j .. 16 j + 15
        auto take = [&](int j, float z, float n) {
          const float zj = __shfl(z, 32 + i), nj = __shfl(n, 32 + i);
          zz = g == j ? zj : zz;
          nn = g == j ? nj : nn;
        };
        float z, n;
        process(t0, kb0, z, n);
        if constexpr (FEAT) take(0, z, n);
        load_tile(clamp_tile(t0 + 2), kb0);
        process(t0 + 1, kb1, z, n);
        if constexpr (FEAT) take(1, z, n);
        load_tile(clamp_tile(t0 + 3), kb1);
        process(t0 + 2, kb0, z, n);
        if constexpr (FEAT) take(2, z, n);
        load_tile(clamp_tile(tn), kb0);
        process(t0 + 3, kb1, z, n);
        if constexpr (FEAT) take(3, z, n);
        load_tile(clamp_tile(tn + 1), kb1);
        if constexpr (FEAT) {
#pragma unroll
          for (int s2 = 0; s2 < S_GMAX; ++s2) {
            zr[s2] = s2 == k ? zz : zr[s2];
            nr[s2] = s2 == k ? nn : nr[s2];
          }
        }
      }
    }
  } else if (wave < ntiles) {
    uint4 kb0[NT], kb1[NT];
    load_tile(wave, kb0);
    // the loop stores one retired pair per tile between the two buffers' loads;
    // a store to the padding row here gives the loop's first wait the same
    // sequence of outstanding operations as every later one
    if constexpr (FEAT) *reinterpret_cast<float2*>(r_sink + 2 * (size_t)(a.lmax - 1 - sink0)) = make_float2(0.0f, 0.0f);
    load_tile(clamp_tile(wave + SNW), kb1);
    // every lane stores (a store under a branch would make the wait before the
    // next tile's matrix ops cover it too); lanes without a retired row of their
    // own write the padding row past the unit
    auto sink = [&](int tt, float z, float n) {
      if constexpr (FEAT) {
        const int key = r0 + tt * 16 + i;
        const int slot = (retire && g == 2 && key < r1) ? key - sink0 : a.lmax - 1 - sink0;
        *reinterpret_cast<float2*>(r_sink + 2 * (size_t)slot) = make_float2(z, n);
      }
    };
    for (int tile = wave; tile < ntiles; tile += 2 * SNW) {
      float z, n;
      process(tile, kb0, z, n);
      sink(tile, z, n);
      load_tile(clamp_tile(tile + 2 * SNW), kb0);
      // unconditional: a tile past the end has no valid key, so it writes no
      // logits and sends its retired pair to the padding row
      process(tile + SNW, kb1, z, n);
      sink(tile + SNW, z, n);
      load_tile(clamp_tile(tile + 3 * SNW), kb1);
    }
  }
}

// Block-wide max of the current heads' logits; stat: SNW * G + G floats of LDS.
// A few threads reduce over the waves (fixed order) and broadcast through LDS,
// so no thread holds all the per-wave partials at once.
template <int G>
__device__ __forceinline__ void block_max(const float (&mrun)[4], float* stat, float (&M)[G]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 4;
  float mm[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) mm[r] = max16(mrun[r]);
  if ((lane & 15) == 0 && 4 * g < G) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * g + r < G) stat[wave * G + 4 * g + r] = mm[r];
  }
  __syncthreads();
  if (threadIdx.x < G) {
    float m = stat[threadIdx.x];
    for (int w = 1; w < SNW; ++w) m = fmaxf(m, stat[w * G + threadIdx.x]);
    stat[SNW * G + threadIdx.x] = m;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < G; ++j) M[j] = stat[SNW * G + j];
}

// pass P over LDS rows [0, n): p = exp(s - M) in place; returns the per-thread
// partial sums of p and p (s - M).
template <int G, int RS = G>
__device__ __forceinline__ void pass_p(float* sbuf, int n, const float (&M)[G], float (&ls)[G],
                                       float (&us)[G]) {
#pragma unroll
  for (int j = 0; j < G; ++j) {
    ls[j] = 0.0f;
    us[j] = 0.0f;
  }
  for (int i = threadIdx.x; i < n; i += SNT) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const float d = sbuf[i * RS + j] - M[j];
      const float p = __builtin_amdgcn_exp2f(d * LOG2E);
      sbuf[i * RS + j] = p;
      ls[j] = ls[j] + p;
      us[j] = us[j] + p * d;
    }
  }
}

// Block sums of G-vectors (fixed order); stat: SNW * 2G + 2G floats of LDS.
template <int G>
__device__ __forceinline__ void block_sum2(float (&x)[G], float (&y)[G], float* stat) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    x[j] = wave_sum(x[j]);
    y[j] = wave_sum(y[j]);
  }
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      stat[wave * 2 * G + j] = x[j];
      stat[wave * 2 * G + G + j] = y[j];
    }
  }
  __syncthreads();
  if (threadIdx.x < 2 * G) {
    float acc = 0.0f;
    for (int w = 0; w < SNW; ++w) acc = acc + stat[w * 2 * G + threadIdx.x];
    stat[SNW * 2 * G + threadIdx.x] = acc;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < G; ++j) {
    x[j] = stat[SNW * 2 * G + j];
    y[j] = stat[SNW * 2 * G + G + j];
  }
}

// pass B: rows [r0, r1), p from pbuf[(i - p0) * G + j]; per-wave partial output
// o[j][e] for the lane's 8 dims (lanes 0..LPR-1 hold the wave total).
template <int D, int G, int RS = G>
__device__ __forceinline__ void pass_b(const DecodeArgs& a, int u, int r0, int r1,
                                       const float* pbuf, int p0, float (&o)[G][8]) {
  constexpr int LPR = MG<D>::LPR, NG = SNT / LPR;
  constexpr int PF = 8;
  const int tid = threadIdx.x, grp = tid / LPR, lam = tid % LPR;
  const char* vc = (const char*)a.v + (size_t)u * a.cap * D * 2;
  const char* vn = a.append ? (const char*)a.v_new + (size_t)u * D * 2 : nullptr;
  const int newrow = a.append ? len_old_of(a, u) : -1;
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[j][e] = 0.0f;
  // rows past r1 load row r1 - 1 again and are given weight 0 (no divergent loads)
  auto load_row = [&](int row) {
    const int rc = row < r1 ? row : r1 - 1;
    return ldg16_nt((rc == newrow ? vn : vc + (size_t)rc * D * 2) + lam * 16);
  };
  auto accumulate = [&](int row, const uint4& vv) {
    const bool ok = row < r1;
    const int rc = ok ? row : r1 - 1;
    float pj[G];
    if constexpr (RS == 4 && G == 4) {
      const f32x4_t w = *reinterpret_cast<const f32x4_t*>(pbuf + (size_t)(rc - p0) * RS);
#pragma unroll
      for (int j = 0; j < G; ++j) pj[j] = ok ? w[j] : 0.0f;
    } else {
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float w = pbuf[(size_t)(rc - p0) * RS + j];
        pj[j] = ok ? w : 0.0f;
      }
    }
    float vf[8];
    unpack_slice<1>(vv, vf);
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[j][e] = __builtin_fmaf(pj[j], vf[e], o[j][e]);
  };
  const int nrows = r1 - r0;
  const int iters = (nrows + NG - 1) / NG;      // row slots per group (uniform)
  // Two halves of PF/2 rows per group in flight.  The loads are unconditional
  // (past the end they re-read the last row), and the scheduling barrier keeps
  // each half's refill between the halves, so while one half is consumed the
  // other half's loads are still outstanding; the last iters % PF rows are
  // consumed after the loop without new loads.
  constexpr int HF = PF / 2;
  uint4 vb[PF];
#pragma unroll
  for (int p = 0; p < PF; ++p) vb[p] = load_row(r0 + grp + p * NG);
  const int full = iters / PF;
  for (int f = 0; f < full; ++f) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int q = 0; q < HF; ++q) accumulate(r0 + grp + (f * PF + h * HF + q) * NG, vb[h * HF + q]);
#pragma unroll
      for (int q = 0; q < HF; ++q) vb[h * HF + q] = load_row(r0 + grp + ((f + 1) * PF + h * HF + q) * NG);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (full * PF + p < iters) accumulate(r0 + grp + (full * PF + p) * NG, vb[p]);
#pragma unroll
  for (int off = LPR; off < 64; off *= 2)
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[j][e] = o[j][e] + __shfl_xor(o[j][e], off);
}

// Norm of the appended value row (every thread receives it through LDS).
template <int D>
__device__ __forceinline__ float new_row_vnorm(const DecodeArgs& a, int u, float* slot) {
  constexpr int LPR = MG<D>::LPR;
  if (threadIdx.x < LPR) {
    float vf[8];
    unpack_slice<1>(ldg16((const char*)a.v_new + (size_t)u * D * 2 + threadIdx.x * 16), vf);
    float v2 = vf[0] * vf[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) v2 = __builtin_fmaf(vf[e], vf[e], v2);
    v2 = row_sum<LPR>(v2);
    if (threadIdx.x == 0) *slot = __builtin_sqrtf(v2);
  }
  __syncthreads();
  return *slot;
}

// Feature update of one row from its weights; returns the updated state.
template <int G>
__device__ __forceinline__ void update_row(const DecodeArgs& a, size_t gi, bool is_new,
                                           const float (&pj)[G], const float (&invl)[G],
                                           const float (&H)[G], const float* ret, float newnorm,
                                           float& alpha, double& num, double& den, int32_t& pos,
                                           float& vn) {
  constexpr float invG = 1.0f / G;
  float w[G];
#pragma unroll
  for (int j = 0; j < G; ++j) w[j] = pj[j] * invl[j];
  float cz, cn;
  contrib_from_weights<G>(w, H, cz, cn);
  if (is_new) {
    alpha = cz * invG;
    den = (double)cz;
    num = (double)cn;
    pos = a.T - 1;
    vn = newnorm;
    a.pos[gi] = pos;
    a.vnorm[gi] = vn;
  } else {
    alpha = (a.arec ? 0.0f : a.alpha[gi]) + cz * invG;
    double z = a.den[gi] + (double)cz;
    double n = a.num[gi] + (double)cn;
    pos = a.pos[gi];
    if (a.retire && pos <= a.pmax_ret) {
      z = z - (double)ret[0];
      n = n - (double)ret[1];
    }
    den = z;
    num = n;
    vn = a.vnorm[gi];
  }
  a.alpha[gi] = alpha;
  a.den[gi] = den;
  a.num[gi] = num;
  if (a.sigma) a.sigma[gi] = head_variance<G>(w);
}

template <int D, int G>
__device__ __forceinline__ void write_ring2(const DecodeArgs& a, int u, const float (&M)[G],
                                            const float (&invl)[G], const float (&H)[G]) {
  constexpr int N16 = G * D * 2 / 16;
  const int t = threadIdx.x;
  const size_t rs = (size_t)u * a.window + a.slot;
  if (t < N16) {
    const char* src = (const char*)a.q + (size_t)u * G * D * 2;
    char* dst = (char*)a.qring + rs * G * D * 2;
    *reinterpret_cast<uint4*>(dst + t * 16) = ldg16(src + t * 16);
  }
  if (t < G) {
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (j == t) {
        a.qstat[(rs * G + j) * 3 + 0] = M[j];
        a.qstat[(rs * G + j) * 3 + 1] = invl[j];
        a.qstat[(rs * G + j) * 3 + 2] = H[j];
      }
  }
}

template <int D>
__device__ __forceinline__ void append_rows(const DecodeArgs& a, int u) {
  constexpr int N16 = D * 2 / 16;
  const int t = threadIdx.x;
  if (t < 2 * N16) {
    const bool isv = t >= N16;
    const int c = isv ? t - N16 : t;
    const char* src = (const char*)(isv ? a.v_new : a.k_new) + (size_t)u * D * 2;
    char* dst = (char*)(isv ? a.v : a.k) + ((size_t)u * a.cap + len_old_of(a, u)) * D * 2;
    *reinterpret_cast<uint4*>(dst + c * 16) = ldg16(src + c * 16);
  }
}

// ---------------------------------------------------------------- unit kernel
// One workgroup per unit, sized so that two fit on a CU (one computes while the
// other streams).  Dynamic LDS: [L * RS floats: logits -> weights -> u64 keys]
// [SNW/2 * G * D output partials][2 ints per compaction move]; the retired
// contributions (cz, cn) of pass A stay in registers (lane l holds those of
// row l of each of its wave's 64-row groups) until the feature pass.
template <int G>
struct RowStride {
  static constexpr int RS = G < 2 ? 2 : G;     // floats per row in LDS (a u64 key must fit)
  static constexpr int KS = RS / 2;            // u64 per row
};

// SMP: training-mode ranking by the Gumbel-perturbed score; the unperturbed
// score is kept in the row's LDS slot beside its key (needs RS >= 4, G >= 4).
// RAG: ragged cache with per-unit budgets (e.budgets).  Unit u has its own rows
// (unit_len[u] + the append) and budget; a.L bounds the rows a workgroup serves
// (it sizes the LDS), and a unit with more rows leaves at once (the chunked
// kernels serve it).  The compaction plan sits in the free half of the rows'
// LDS slots beside the keys (move j beside row j's key: at most L / 2 moves,
// however many rows the unit evicts), so it needs RS >= 4 (G >= 4).
template <int D, int G, bool FEAT, bool EVICT, bool SIG = false, bool SMP = false, bool RAG = false>
__global__ void __launch_bounds__(SNT, G > 4 ? 2 : 4) step_unit_kernel(DecodeArgs a, EvictArgs e) {
  static_assert(!SIG || (FEAT && !EVICT), "sigma is stored by the decode-only variant");
  static_assert(!SMP || (EVICT && RowStride<G>::RS >= 4), "sampling keeps the score beside the key");
  static_assert(!RAG || (FEAT && EVICT && !SIG && !SMP && RowStride<G>::RS >= 4),
                "the ragged variant plans its moves beside the keys");
  constexpr int LPR = MG<D>::LPR;
  constexpr int RS = RowStride<G>::RS, KS = RowStride<G>::KS;
  extern __shared__ float lds[];
  __shared__ SelShared sh;
  __shared__ float stat[SNW * 2 * G + 2 * G];
  __shared__ float newnorm_slot;
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = RAG ? len_old_of(a, u) + a.append : a.L;
  if constexpr (RAG) {
    if (L > a.L || L < 1) return;                     // whole workgroup: the chunked kernels' unit
  }
  float* sbuf = lds;                                  // row stride RS
  float* obuf = lds + (size_t)L * RS;                 // (SNW / 2) * G * D
  int* mv = (int*)(obuf + (SNW / 2) * G * D);
  const size_t ub = (size_t)u * a.cap;

  if (a.append) append_rows<D>(a, u);
  const bool retire = FEAT && a.retire;
  float M[G], invl[G], H[G];
  float zr[S_GMAX], nr[S_GMAX];     // retired pairs of the wave's 64-row groups (lane = row)
  {
    uint4 qa[MG<D>::NT];
    load_qfrag<D, G>(qa, a, u, retire);
    RetStats<G> rs;
    if (retire) load_ret<G>(rs, a, u);
    float mrun[4];
    pass_a<D, G, FEAT, true, RS>(a, u, 0, L, sbuf, nullptr, 0, qa, retire, rs, mrun, zr, nr);
    block_max<G>(mrun, stat, M);
  }
  {
    float ls[G], us[G];
    pass_p<G, RS>(sbuf, L, M, ls, us);
    __syncthreads();
    block_sum2<G>(ls, us, stat);
#pragma unroll
    for (int j = 0; j < G; ++j) {
      invl[j] = 1.0f / ls[j];
      H[j] = __logf(ls[j]) - us[j] * invl[j];
    }
  }
  {
    float o[G][8];
    pass_b<D, G, RS>(a, u, 0, L, sbuf, 0, o);
    // tree over the waves through SNW/2 partial slots
    if (wave >= SNW / 2 && lane < LPR) {
#pragma unroll
      for (int j = 0; j < G; ++j)
#pragma unroll
        for (int x = 0; x < 8; ++x) obuf[((wave - SNW / 2) * G + j) * D + lane * 8 + x] = o[j][x];
    }
    __syncthreads();
    if (wave < SNW / 2 && lane < LPR) {
#pragma unroll
      for (int j = 0; j < G; ++j)
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          float* slot = &obuf[(wave * G + j) * D + lane * 8 + x];
          *slot = o[j][x] + *slot;
        }
    }
  }
  __syncthreads();
  for (int t = tid; t < G * D; t += SNT) {
    const int j = t / D;
    float acc = obuf[t];
    for (int w = 1; w < SNW / 2; ++w) acc = acc + obuf[w * G * D + t];
    float il = invl[0];
#pragma unroll
    for (int jj = 1; jj < G; ++jj) il = (jj == j) ? invl[jj] : il;
    ((uint16_t*)a.out)[(size_t)u * G * D + t] = (uint16_t)f32_to_bf16_bits(acc * il);
  }
  if constexpr (FEAT) {
    const float newnorm = a.append ? new_row_vnorm<D>(a, u, &newnorm_slot) : 0.0f;
    const int newrow = a.append ? len_old_of(a, u) : -1;
    const float invT = 1.0f / (float)a.T;
    constexpr float invG = 1.0f / G;
    uint64_t* keys = reinterpret_cast<uint64_t*>(sbuf);   // row i's key replaces its weights
    // The rows of pass A's 64-row groups, one per lane: group b (wave b mod SNW)
    // row 64 b + lane, whose retired pair this lane kept in registers.  The next
    // group's state is requested before the current one is updated; in full
    // groups every load and store is unconditional, only the unit's partial last
    // group (one wave) guards its stores.
    const int ngrp = (L + 63) / 64;
    const int ngw = wave < ngrp ? (ngrp - 1 - wave) / SNW + 1 : 0;
    const bool part = ngw > 0 && wave + SNW * (ngw - 1) == ngrp - 1 && (L & 63) != 0;
    const int nfull = ngw - (part ? 1 : 0);
    struct Row {
      float al, vn;
      double nu, de;
      int32_t p;
    };
    auto load_row = [&](int k, Row& x) {
      const int r = 64 * (wave + SNW * k) + lane;
      const size_t gi = ub + (r < L ? r : L - 1);
      x.al = a.alpha[gi];
      x.nu = a.num[gi];
      x.de = a.den[gi];
      x.p = a.pos[gi];
      x.vn = a.vnorm[gi];
    };
    auto update = [&](int k, const Row& x, bool guard) {
      const int r = 64 * (wave + SNW * k) + lane;
      const bool valid = r < L;
      const int ic = valid ? r : L - 1;
      const size_t gi = ub + ic;
      float w[G];
#pragma unroll
      for (int j = 0; j < G; ++j) w[j] = sbuf[ic * RS + j] * invl[j];
      float cz, cn;
      contrib_from_weights<G>(w, H, cz, cn);
      float rz = zr[0], rn = nr[0];
#pragma unroll
      for (int s2 = 1; s2 < S_GMAX; ++s2) {
        rz = s2 == k ? zr[s2] : rz;
        rn = s2 == k ? nr[s2] : rn;
      }
      float al = (a.arec ? 0.0f : x.al) + cz * invG;
      double de = x.de + (double)cz;
      double nu = x.nu + (double)cn;
      int32_t ps = x.p;
      float vn = x.vn;
      if (retire && ps <= a.pmax_ret) {
        de = de - (double)rz;
        nu = nu - (double)rn;
      }
      if (ic == newrow) {
        al = cz * invG;
        de = (double)cz;
        nu = (double)cn;
        ps = a.T - 1;
        vn = newnorm;
      }
      if (!guard || valid) {
        a.alpha[gi] = al;
        a.den[gi] = de;
        a.num[gi] = nu;
        if constexpr (SIG) a.sigma[gi] = head_variance<G>(w);
      }
      if constexpr (EVICT) {
        float f[1][4], sc[1];
        make_features(al, vn, nu, de, ps, invT, f[0]);
        policy_scores<1>(e, f, sc, 1);
        if constexpr (SMP) {
          const float ks = sampled_score(e, sc[0], ps, u);
          if (!guard || valid) {
            keys[(size_t)r * KS] = row_key(ks, ps);
            sbuf[(size_t)r * RS + 2] = sc[0];
          }
        } else {
          if (!guard || valid) keys[(size_t)r * KS] = row_key(sc[0], ps);
        }
      }
    };
    if (ngw > 0) {
      Row cur, nxt;
      load_row(0, cur);
      for (int k = 0; k < nfull; ++k) {
        load_row(k + 1 < ngw ? k + 1 : k, nxt);
        update(k, cur, false);
        cur = nxt;
      }
      if (part) update(nfull, cur, true);
    }
    // the appended row's position and value norm (the other rows keep theirs)
    if (a.append && tid == 0) {
      a.pos[ub + newrow] = a.T - 1;
      a.vnorm[ub + newrow] = newnorm;
    }
    if (a.window > 0) write_ring2<D, G>(a, u, M, invl, H);
    if constexpr (EVICT) {
      __syncthreads();
      // row stride of scores_out: the unit's rows, or the bound of a ragged cache
      const size_t lso = RAG ? (size_t)e.L : (size_t)L;
      if (e.scores_out) {
        // the scores: beside the keys when sampling, else recovered from the
        // ranking keys (-0 reads back as +0)
        for (int r = tid; r < L; r += SNT) {
          if constexpr (SMP) {
            e.scores_out[(size_t)u * lso + r] = sbuf[(size_t)r * RS + 2];
          } else {
            const uint32_t k = (uint32_t)(keys[(size_t)r * KS] >> 32);
            const uint32_t bits = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
            e.scores_out[(size_t)u * lso + r] = __uint_as_float(bits);
          }
        }
      }
      const int nslots = (L + SNT - 1) / SNT;
      LdsKeys<S_KMAX, SNT> lk{keys, KS};
      if constexpr (RAG) {
        const int Bu = unit_budget(e, u);
        if (Bu < L) {
          select_compact<LdsKeys<S_KMAX, SNT>, 1, D, SNT, RS>(e, u, L, Bu, lk, nslots, sh,
                                                             reinterpret_cast<int*>(sbuf) + 2);
          if (e.kept_out)     // slots past this unit's budget
            for (int r = Bu + tid; r < e.ld_kept; r += SNT) e.kept_out[(size_t)u * e.ld_kept + r] = -1;
        } else if (e.kept_out) {
          for (int r = tid; r < e.ld_kept; r += SNT) e.kept_out[(size_t)u * e.ld_kept + r] = r < L ? r : -1;
        }
      } else if (e.evict) {
        select_compact<LdsKeys<S_KMAX, SNT>, 1, D, SNT>(e, u, L, e.budget, lk, nslots, sh, mv);
      } else if (e.kept_out) {
        for (int r = tid; r < L; r += SNT) e.kept_out[(size_t)u * L + r] = r;
      }
    }
  }
}

// ---------------------------------------------------------------- chunked path
// ws_part per (unit, chunk): [G] chunk max m_c, [G] l_c, [G] u_c, [G*D] o_c, the
// sums taken relative to the chunk's own maximum (stepc_d rescales them).
template <int G>
__device__ __forceinline__ void chunk_max(const DecodeArgs& a, int u, int D, float (&M)[G]) {
  const float* parts = a.ws_part + (size_t)u * a.nchunks * (3 * G + G * D);
#pragma unroll
  for (int j = 0; j < G; ++j) {
    float m = parts[j];
    for (int c = 1; c < a.nchunks; ++c) m = fmaxf(m, parts[(size_t)c * (3 * G + G * D) + j]);
    M[j] = m;
  }
}

// Passes A, P and B of one chunk in one workgroup: K streamed once (logits and
// retired pairs to the workspace), p = exp(s - m_c) against the chunk maximum,
// then V streamed once.  The chunk's logits come back from the workspace
// while still in L2 (this workgroup stored them moments before).  RET: the
// step retires a step leaving the window; without one no retired pair is
// stored (the feature pass reads them only when the step retires).
template <int D, int G, bool FEAT, bool RET>
__global__ void __launch_bounds__(SNT) stepc_ab_kernel(DecodeArgs a) {
  constexpr int LPR = MG<D>::LPR;
  __shared__ float pbuf[SCHUNK * G];
  __shared__ float obuf[SNW * G * D];
  __shared__ float stat[SNW * 2 * G + 2 * G];
  const int c = blockIdx.x, u = a.y0 + blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Lu = len_old_of(a, u) + a.append;       // this unit's rows (ragged caches: per unit)
  if (Lu <= a.fused_rows) return;                   // served by the single-launch kernel
  const int r0 = c * a.chunk, r1 = min(Lu, r0 + a.chunk), n = r1 - r0;
  if (c == 0 && a.append) append_rows<D>(a, u);
  float* part = a.ws_part + ((size_t)u * a.nchunks + c) * (3 * G + G * D);
  if (n <= 0) {
    // a chunk past this unit's rows: neutral partials (max -inf, sums 0, no output)
    for (int t = tid; t < 3 * G + G * D; t += SNT) part[t] = t < G ? NEG_BIG : 0.0f;
    return;
  }
  constexpr bool FR = FEAT && RET;
  const bool retire = FR && a.retire;
  uint4 qa[MG<D>::NT];
  load_qfrag<D, G>(qa, a, u, retire);
  RetStats<G> rs;
  if (retire) load_ret<G>(rs, a, u);
  float mrun[4];
  float zr[S_GMAX], nr[S_GMAX];   // unused on this path
  pass_a<D, G, FR, false>(a, u, r0, r1, a.ws_s + (size_t)u * a.lmax * G,
                          FR ? a.ws_r + (size_t)u * a.lmax * 2 : nullptr, 0, qa, retire, rs,
                          mrun, zr, nr);
  float M[G];
  block_max<G>(mrun, stat, M);    // (its barriers also order the logit stores before the reads)
  const float* src = a.ws_s + ((size_t)u * a.lmax + r0) * G;
  for (int t = tid; t < n * G; t += SNT) pbuf[t] = src[t];
  __syncthreads();
  float ls[G], us[G];
  pass_p<G>(pbuf, n, M, ls, us);
  __syncthreads();
  block_sum2<G>(ls, us, stat);
  float o[G][8];
  pass_b<D, G>(a, u, r0, r1, pbuf, r0, o);
  if (lane < LPR) {
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int x = 0; x < 8; ++x) obuf[(wave * G + j) * D + lane * 8 + x] = o[j][x];
  }
  __syncthreads();
  for (int t = tid; t < G * D; t += SNT) {
    float acc = 0.0f;
    for (int w = 0; w < SNW; ++w) acc = acc + obuf[w * G * D + t];
    part[3 * G + t] = acc;
  }
  if (tid < G) {
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (j == tid) {
        part[j] = M[j];
        part[G + j] = ls[j];
        part[2 * G + j] = us[j];
      }
  }
}

template <int D, int G, bool FEAT>
__global__ void __launch_bounds__(SNT) stepc_d_kernel(DecodeArgs a) {
  __shared__ float newnorm_slot;
  const int c = blockIdx.x, u = a.y0 + blockIdx.y, tid = threadIdx.x;
  const int Lu = len_old_of(a, u) + a.append;
  if (Lu <= a.fused_rows) return;                   // served by the single-launch kernel
  const int r0 = c * a.chunk, r1 = min(Lu, r0 + a.chunk);
  const int PART = 3 * G + G * D;
  const float* parts = a.ws_part + (size_t)u * a.nchunks * PART;
  float M[G], ls[G], us[G], invl[G], H[G];
  chunk_max<G>(a, u, D, M);
  // chunk c's sums move to the common maximum M: with f = e^(m_c - M),
  // l += f l_c, u += f (u_c + (m_c - M) l_c), o += f o_c (a neutral chunk: f = 0)
#pragma unroll
  for (int j = 0; j < G; ++j) {
    float l = 0.0f, uu = 0.0f;
    for (int cc = 0; cc < a.nchunks; ++cc) {
      const float* pc = parts + (size_t)cc * PART;
      const float dm = pc[j] - M[j];
      const float f = __builtin_amdgcn_exp2f(dm * LOG2E);
      l = l + f * pc[G + j];
      uu = uu + f * (pc[2 * G + j] + dm * pc[G + j]);
    }
    ls[j] = l;
    us[j] = uu;
    invl[j] = 1.0f / l;
    H[j] = __logf(l) - uu * invl[j];
  }
  if constexpr (FEAT) {
    const int newrow = a.append ? len_old_of(a, u) : -1;
    const float newnorm = (a.append && newrow >= r0 && newrow < r1)
                              ? new_row_vnorm<D>(a, u, &newnorm_slot) : 0.0f;
    const float* s_src = a.ws_s + (size_t)u * a.lmax * G;
    const float* r_src = a.ws_r + (size_t)u * a.lmax * 2;
    const size_t ub = (size_t)u * a.cap;
    for (int i = r0 + tid; i < r1; i += SNT) {
      float pj[G];
#pragma unroll
      for (int j = 0; j < G; ++j)
        pj[j] = __builtin_amdgcn_exp2f((s_src[(size_t)i * G + j] - M[j]) * LOG2E);
      float al, vn;
      double nu, de;
      int32_t ps;
      update_row<G>(a, ub + i, i == newrow, pj, invl, H, r_src + 2 * (size_t)i, newnorm, al, nu,
                    de, ps, vn);
    }
  }
  if (c != 0) return;
  for (int t = tid; t < G * D; t += SNT) {
    const int j = t / D;
    float mj = M[0];
#pragma unroll
    for (int jj = 1; jj < G; ++jj) mj = (jj == j) ? M[jj] : mj;
    float acc = 0.0f;
    for (int cc = 0; cc < a.nchunks; ++cc) {
      const float* pc = parts + (size_t)cc * PART;
      acc = acc + __builtin_amdgcn_exp2f((pc[j] - mj) * LOG2E) * pc[3 * G + t];
    }
    float il = invl[0];
#pragma unroll
    for (int jj = 1; jj < G; ++jj) il = (jj == j) ? invl[jj] : il;
    ((uint16_t*)a.out)[(size_t)u * G * D + t] = (uint16_t)f32_to_bf16_bits(acc * il);
  }
  if (FEAT && a.window > 0) write_ring2<D, G>(a, u, M, invl, H);
}

// ---------------------------------------------------------------- ragged caches
__global__ void unit_len_add_kernel(int32_t* len, int units, int add) {
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u < units) len[u] += add;
}

__global__ void unit_len_min_kernel(int32_t* len, const int32_t* budgets, int b, int units) {
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u < units) {
    int bu = budgets ? budgets[u] : b;
    bu = bu < 1 ? 1 : bu > b ? b : bu;            // the clamp the selection applies
    len[u] = bu < len[u] ? bu : len[u];
  }
}

int launch_unit_len_add(int32_t* len, int units, int add, void* stream) {
  hipLaunchKernelGGL(unit_len_add_kernel, dim3((units + 255) / 256), dim3(256), 0,
                     (hipStream_t)stream, len, units, add);
  return (int)hipGetLastError();
}

int launch_unit_len_min(int32_t* len, const int32_t* budgets, int b, int units, void* stream) {
  hipLaunchKernelGGL(unit_len_min_kernel, dim3((units + 255) / 256), dim3(256), 0,
                     (hipStream_t)stream, len, budgets, b, units);
  return (int)hipGetLastError();
}

// ---------------------------------------------------------------- dispatch
// ints of the compaction move list (a multiple of four, so what follows it in
// LDS stays 16-byte aligned)
static int move_list_ints(int nmoves) { return (2 * (nmoves > 0 ? nmoves : 1) + 3) / 4 * 4; }

size_t step_lds_bytes(int L, int G, int D, bool feat, int nmoves) {
  const size_t rs = G < 2 ? 2 : G;
  const size_t b = ((size_t)L * rs + (size_t)(SNW / 2) * G * D) * sizeof(float);
  return b + (size_t)move_list_ints(nmoves) * sizeof(int);
}

bool step_fits(int L, int G, int D, bool feat, int nmoves) {
  return (!feat || L <= S_KMAX * SNT) && step_lds_bytes(L, G, D, feat, nmoves) <= (size_t)S_LDS;
}

int step_chunk_rows() { return SCHUNK; }

int step_ragged_rows(int G, int D) {
  if (G < 4) return 0;                            // keys fill the row slots: no room for the plan
  // two workgroups per CU: half the dynamic LDS budget; rows in registers: S_KMAX per thread
  int L = S_KMAX * SNT;
  while (L > 0 && step_lds_bytes(L, G, D, true, 0) > (size_t)S_LDS / 2) --L;
  return L;
}

template <int D, int G>
static int launch_step_t(const DecodeArgs& a, const EvictArgs* e, bool feat, bool chunked,
                         hipStream_t s) {
  if (!chunked) {
    // (the ragged variant plans its moves beside the keys: no separate list)
    const int nm = e && e->evict && !a.unit_len ? (a.L - e->budget < e->budget ? a.L - e->budget : e->budget) : 0;
    EvictArgs ee;
    if (e) ee = *e;
    else __builtin_memset(&ee, 0, sizeof(ee));
    ee.mv_ints = move_list_ints(nm);
    const size_t lds = step_lds_bytes(a.L, G, D, feat, nm);
    auto pick = [&](auto kern) {
      hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hipLaunchKernelGGL(kern, dim3(a.units), dim3(SNT), lds, s, a, ee);
    };
    // (the fused evicting variants serve the one-hidden-layer four-input policy)
    if (!feat) pick(step_unit_kernel<D, G, false, false>);
    else if (e && e->sample) {
      if constexpr (RowStride<G>::RS >= 4) pick(step_unit_kernel<D, G, true, true, false, true>);
      else return (int)hipErrorInvalidValue;     // the caller takes the separate path
    }
    else if (e && a.unit_len) {
      if constexpr (RowStride<G>::RS >= 4) pick(step_unit_kernel<D, G, true, true, false, false, true>);
      else return (int)hipErrorInvalidValue;     // the caller takes the separate path
    }
    else if (e) pick(step_unit_kernel<D, G, true, true>);
    else if (a.sigma) pick(step_unit_kernel<D, G, true, false, true>);
    else pick(step_unit_kernel<D, G, true, false>);
  } else {
    // every slice of one pass before the next (stream order)
    for_grid_y(a.units, [&](int y0, int ny) {
      DecodeArgs b = a;
      b.y0 = y0;
      if (feat && a.retire)
        hipLaunchKernelGGL((stepc_ab_kernel<D, G, true, true>), dim3(a.nchunks, ny), dim3(SNT), 0, s, b);
      else if (feat)
        hipLaunchKernelGGL((stepc_ab_kernel<D, G, true, false>), dim3(a.nchunks, ny), dim3(SNT), 0, s, b);
      else
        hipLaunchKernelGGL((stepc_ab_kernel<D, G, false, false>), dim3(a.nchunks, ny), dim3(SNT), 0, s, b);
    });
    for_grid_y(a.units, [&](int y0, int ny) {
      DecodeArgs b = a;
      b.y0 = y0;
      if (feat) hipLaunchKernelGGL((stepc_d_kernel<D, G, true>), dim3(a.nchunks, ny), dim3(SNT), 0, s, b);
      else hipLaunchKernelGGL((stepc_d_kernel<D, G, false>), dim3(a.nchunks, ny), dim3(SNT), 0, s, b);
    });
  }
  return (int)hipGetLastError();
}

template <int D>
static int launch_step_g(const DecodeArgs& a, const EvictArgs* e, int G, bool feat, bool chunked,
                         hipStream_t s) {
  switch (G) {
    case 1: return launch_step_t<D, 1>(a, e, feat, chunked, s);
    case 2: return launch_step_t<D, 2>(a, e, feat, chunked, s);
    case 4: return launch_step_t<D, 4>(a, e, feat, chunked, s);
    case 8: return launch_step_t<D, 8>(a, e, feat, chunked, s);
  }
  return (int)hipErrorInvalidValue;
}

int launch_step(const DecodeArgs& a, const EvictArgs* e, int D, int G, bool feat, bool chunked,
                void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (D == 128) return launch_step_g<128>(a, e, G, feat, chunked, s);
  if (D == 64) return launch_step_g<64>(a, e, G, feat, chunked, s);
  return (int)hipErrorInvalidValue;
}

}  // namespace dc
