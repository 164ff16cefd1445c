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
// Caches too long for LDS use the chunked form of the same passes (three
// kernels, logits in the workspace).
#include "dc_select.hpp"

#pragma clang fp contract(off)

namespace dc {

constexpr int SNT = 512;              // threads per workgroup (two workgroups per CU)
constexpr int SNW = SNT / 64;
constexpr int SCHUNK = 2048;          // rows per workgroup on the chunked path
constexpr int S_KMAX = 10;            // fused step: row slots per thread (L <= 5120)
constexpr int S_KB = 3;               // row slots per thread handled per feature batch
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
// Rows [r0, r1) of unit u, 16-key tiles distributed over the waves.  Logits of
// the current heads go to s_sink[(i - sink0) * G + j], retired contributions to
// r_sink[2 (i - sink0)], running maxima per current head into mrun.
template <int D, int G, bool FEAT, int RS = G>
__device__ __forceinline__ void pass_a(const DecodeArgs& a, int u, int r0, int r1, float* s_sink,
                                       float* r_sink, int sink0, const uint4 (&qa)[MG<D>::NT],
                                       bool retire, const RetStats<G>& rs, float (&mrun)[4]) {
  constexpr int NT = MG<D>::NT, LB = MG<D>::LB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, i = lane & 15, g = lane >> 4;
  const char* kc = (const char*)a.k + (size_t)u * a.cap * D * 2;
  const char* kn = a.append ? (const char*)a.k_new + (size_t)u * D * 2 : nullptr;
  const int newrow = a.append ? a.len_old : -1;
  const int ntiles = (r1 - r0 + 15) / 16;
#pragma unroll
  for (int r = 0; r < 4; ++r) mrun[r] = NEG_BIG;
  auto load_tile = [&](int tile, uint4 (&kb)[NT]) {
    int key = r0 + tile * 16 + i;
    key = key < r1 ? key : r1 - 1;
    const char* kp = key == newrow ? kn : kc + (size_t)key * D * 2;
    // plain loads: instructions t and t+1 read the two halves of the same 128-byte
    // line, so the second one should find it in the vector L1
#pragma unroll
    for (int t = 0; t < NT; ++t) kb[t] = ldg16(kp + 16 * (4 * t + g));
  };
  auto process = [&](int tt, const uint4 (&kb)[NT]) {
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
    if constexpr (FEAT) {
      if (retire && g >= 2 && 4 * (g - 2) < G) {
        const bool hi = G > 4 && g == 3;        // heads 4..7 (only when G == 8)
        float z = 0.0f, n = 0.0f;
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
        if constexpr (G > 4) {   // heads 4..7 live in group 3: add the blocks in order
          const float z1 = __shfl_down(z, 16), n1 = __shfl_down(n, 16);
          z = z + z1;
          n = n + n1;
        }
        if (g == 2 && valid) {
          r_sink[2 * (key - sink0)] = z;
          r_sink[2 * (key - sink0) + 1] = n;
        }
      }
    }
  };
  // two tiles in flight per wave: consume a buffer, then refill it
  uint4 kb0[NT], kb1[NT];
  if (wave < ntiles) load_tile(wave, kb0);
  if (wave + SNW < ntiles) load_tile(wave + SNW, kb1);
  for (int tile = wave; tile < ntiles; tile += 2 * SNW) {
    process(tile, kb0);
    if (tile + 2 * SNW < ntiles) load_tile(tile + 2 * SNW, kb0);
    if (tile + SNW < ntiles) {
      process(tile + SNW, kb1);
      if (tile + 3 * SNW < ntiles) load_tile(tile + 3 * SNW, kb1);
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
  constexpr int PF = 4;
  const int tid = threadIdx.x, grp = tid / LPR, lam = tid % LPR;
  const char* vc = (const char*)a.v + (size_t)u * a.cap * D * 2;
  const char* vn = a.append ? (const char*)a.v_new + (size_t)u * D * 2 : nullptr;
  const int newrow = a.append ? a.len_old : -1;
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
#pragma unroll
    for (int j = 0; j < G; ++j) pj[j] = ok ? pbuf[(size_t)(rc - p0) * RS + j] : 0.0f;
    float vf[8];
    unpack_slice<1>(vv, vf);
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[j][e] = __builtin_fmaf(pj[j], vf[e], o[j][e]);
  };
  const int nrows = r1 - r0;
  const int iters = (nrows + NG - 1) / NG;      // row slots per group (uniform)
  uint4 vb[PF];
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (p < iters) vb[p] = load_row(r0 + grp + p * NG);
  for (int it = 0; it < iters; it += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      if (it + p < iters) {
        accumulate(r0 + grp + (it + p) * NG, vb[p]);
        if (it + p + PF < iters) vb[p] = load_row(r0 + grp + (it + p + PF) * NG);
      }
    }
  }
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
    alpha = a.alpha[gi] + cz * invG;
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
    char* dst = (char*)(isv ? a.v : a.k) + ((size_t)u * a.cap + a.len_old) * D * 2;
    *reinterpret_cast<uint4*>(dst + c * 16) = ldg16(src + c * 16);
  }
}

// ---------------------------------------------------------------- unit kernel
// One workgroup per unit, sized so that two fit on a CU (one computes while the
// other streams).  Dynamic LDS: [L * RS floats: logits -> weights -> u64 keys]
// [SNW/2 * G * D output partials][2 ints per compaction move]; the retired
// contributions (cz, cn) of pass A go to the workspace (ws_r) and come back in
// the feature pass.
template <int G>
struct RowStride {
  static constexpr int RS = G < 2 ? 2 : G;     // floats per row in LDS (a u64 key must fit)
  static constexpr int KS = RS / 2;            // u64 per row
};

template <int D, int G, bool FEAT, bool EVICT, int NH>
__global__ void __launch_bounds__(SNT, 2) step_unit_kernel(DecodeArgs a, EvictArgs e) {
  constexpr int LPR = MG<D>::LPR;
  constexpr int RS = RowStride<G>::RS, KS = RowStride<G>::KS;
  extern __shared__ float lds[];
  __shared__ SelShared sh;
  __shared__ float stat[SNW * 2 * G + 2 * G];
  __shared__ float newnorm_slot;
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = a.L;
  float* sbuf = lds;                                  // row stride RS
  float* obuf = lds + (size_t)L * RS;                 // (SNW / 2) * G * D
  int* mv = (int*)(obuf + (SNW / 2) * G * D);
  float* rws = FEAT ? a.ws_r + (size_t)u * a.lmax * 2 : nullptr;
  const size_t ub = (size_t)u * a.cap;

  if (a.append) append_rows<D>(a, u);
  const bool retire = FEAT && a.retire;
  float M[G], invl[G], H[G];
  {
    uint4 qa[MG<D>::NT];
    load_qfrag<D, G>(qa, a, u, retire);
    RetStats<G> rs;
    if (retire) load_ret<G>(rs, a, u);
    float mrun[4];
    pass_a<D, G, FEAT, RS>(a, u, 0, L, sbuf, rws, 0, qa, retire, rs, mrun);
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
    const int newrow = a.append ? a.len_old : -1;
    const float invT = 1.0f / (float)a.T;
    constexpr float invG = 1.0f / G;
    uint64_t* keys = reinterpret_cast<uint64_t*>(sbuf);   // row i's key replaces its weights
    const int nslots = (L + SNT - 1) / SNT;
    struct Batch {
      float al[S_KB], vn[S_KB], rz[S_KB], rn[S_KB];
      double nu[S_KB], de[S_KB];
      int32_t p[S_KB];
    };
    auto kact_of = [&](int kb) {
      const int rem = L - kb * SNT - wave * 64;   // slots with a valid row in this wave
      return rem > 0 ? min(S_KB, (rem + SNT - 1) / SNT) : 0;
    };
    auto load_batch = [&](int kb, Batch& b) {
      const int kact = kact_of(kb);
#pragma unroll
      for (int k = 0; k < S_KB; ++k) {
        if (k < kact) {
          const int i = (kb + k) * SNT + tid;
          const int ic = i < L ? i : L - 1;
          const size_t gi = ub + ic;
          b.al[k] = a.alpha[gi];
          b.nu[k] = a.num[gi];
          b.de[k] = a.den[gi];
          b.p[k] = a.pos[gi];
          b.vn[k] = a.vnorm[gi];
          if (retire) {
            b.rz[k] = rws[2 * ic];
            b.rn[k] = rws[2 * ic + 1];
          }
        }
      }
    };
    Batch cur, nxt;
    load_batch(0, cur);
    for (int kb = 0; kb < nslots; kb += S_KB) {
      if (kb + S_KB < nslots) load_batch(kb + S_KB, nxt);
      const int kact = kact_of(kb);
      float x[S_KB][4];
      int32_t pk[S_KB];
#pragma unroll
      for (int k = 0; k < S_KB; ++k) {
        if (k < kact) {
          const int i = (kb + k) * SNT + tid;
          const bool valid = i < L;
          const int ic = valid ? i : L - 1;
          const size_t gi = ub + ic;
          float w[G];
#pragma unroll
          for (int j = 0; j < G; ++j) w[j] = sbuf[ic * RS + j] * invl[j];
          float cz, cn;
          contrib_from_weights<G>(w, H, cz, cn);
          float al, vn;
          double nu, de;
          int32_t ps;
          if (ic == newrow) {
            al = cz * invG;
            de = (double)cz;
            nu = (double)cn;
            ps = a.T - 1;
            vn = newnorm;
          } else {
            al = cur.al[k] + cz * invG;
            de = cur.de[k] + (double)cz;
            nu = cur.nu[k] + (double)cn;
            ps = cur.p[k];
            vn = cur.vn[k];
            if (retire && ps <= a.pmax_ret) {
              de = de - (double)cur.rz[k];
              nu = nu - (double)cur.rn[k];
            }
          }
          if (valid) {
            a.alpha[gi] = al;
            a.den[gi] = de;
            a.num[gi] = nu;
            if (ic == newrow) {
              a.pos[gi] = ps;
              a.vnorm[gi] = vn;
            }
          }
          make_features(al, vn, nu, de, ps, invT, x[k]);
          pk[k] = ps;
        }
      }
      if constexpr (EVICT) {
        float sc[S_KB];
        policy_scores<S_KB, NH>(e, x, sc, kact);
#pragma unroll
        for (int k = 0; k < S_KB; ++k) {
          const int i = (kb + k) * SNT + tid;
          if (k < kact && i < L) {
            if (e.scores_out) e.scores_out[(size_t)u * L + i] = sc[k];
            keys[(size_t)i * KS] = row_key(sc[k], pk[k]);
          }
        }
      }
      cur = nxt;
    }
    if (a.window > 0) write_ring2<D, G>(a, u, M, invl, H);
    if constexpr (EVICT) {
      __syncthreads();
      if (e.evict) {
        LdsKeys<S_KMAX, SNT> lk{keys, KS};
        select_compact<LdsKeys<S_KMAX, SNT>, 1, D, SNT>(e, u, lk, nslots, sh, mv);
      } else if (e.kept_out) {
        for (int r = tid; r < L; r += SNT) e.kept_out[(size_t)u * L + r] = r;
      }
    }
  }
}

// ---------------------------------------------------------------- chunked path
// ws_part per (unit, chunk): [G] max, [G] l, [G] u, [G*D] o.
template <int D, int G, bool FEAT>
__global__ void __launch_bounds__(SNT) stepc_a_kernel(DecodeArgs a) {
  __shared__ float stat[SNW * 2 * G + 2 * G];
  const int c = blockIdx.x, u = blockIdx.y;
  const int r0 = c * a.chunk, r1 = min(a.L, r0 + a.chunk);
  if (c == 0 && a.append) append_rows<D>(a, u);
  const bool retire = FEAT && a.retire;
  uint4 qa[MG<D>::NT];
  load_qfrag<D, G>(qa, a, u, retire);
  RetStats<G> rs;
  if (retire) load_ret<G>(rs, a, u);
  float mrun[4];
  pass_a<D, G, FEAT>(a, u, r0, r1, a.ws_s + (size_t)u * a.lmax * G,
                     FEAT ? a.ws_r + (size_t)u * a.lmax * 2 : nullptr, 0, qa, retire, rs, mrun);
  float M[G];
  block_max<G>(mrun, stat, M);
  if (threadIdx.x < G) {
    float* part = a.ws_part + ((size_t)u * a.nchunks + c) * (3 * G + G * D);
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (j == (int)threadIdx.x) part[j] = M[j];
  }
}

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

template <int D, int G>
__global__ void __launch_bounds__(SNT) stepc_b_kernel(DecodeArgs a) {
  constexpr int LPR = MG<D>::LPR;
  __shared__ float pbuf[SCHUNK * G];
  __shared__ float obuf[SNW * G * D];
  __shared__ float stat[SNW * 2 * G + 2 * G];
  const int c = blockIdx.x, u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = c * a.chunk, r1 = min(a.L, r0 + a.chunk), n = r1 - r0;
  float M[G];
  chunk_max<G>(a, u, D, M);
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
  float* part = a.ws_part + ((size_t)u * a.nchunks + c) * (3 * G + G * D);
  for (int t = tid; t < G * D; t += SNT) {
    float acc = 0.0f;
    for (int w = 0; w < SNW; ++w) acc = acc + obuf[w * G * D + t];
    part[3 * G + t] = acc;
  }
  if (tid < G) {
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (j == tid) {
        part[G + j] = ls[j];
        part[2 * G + j] = us[j];
      }
  }
}

template <int D, int G, bool FEAT>
__global__ void __launch_bounds__(SNT) stepc_d_kernel(DecodeArgs a) {
  __shared__ float newnorm_slot;
  const int c = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  const int r0 = c * a.chunk, r1 = min(a.L, r0 + a.chunk);
  const int PART = 3 * G + G * D;
  const float* parts = a.ws_part + (size_t)u * a.nchunks * PART;
  float M[G], ls[G], us[G], invl[G], H[G];
  chunk_max<G>(a, u, D, M);
#pragma unroll
  for (int j = 0; j < G; ++j) {
    float l = 0.0f, uu = 0.0f;
    for (int cc = 0; cc < a.nchunks; ++cc) {
      l = l + parts[(size_t)cc * PART + G + j];
      uu = uu + parts[(size_t)cc * PART + 2 * G + j];
    }
    ls[j] = l;
    us[j] = uu;
    invl[j] = 1.0f / l;
    H[j] = __logf(l) - uu * invl[j];
  }
  if constexpr (FEAT) {
    const int newrow = a.append ? a.len_old : -1;
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
    float acc = 0.0f;
    for (int cc = 0; cc < a.nchunks; ++cc) acc = acc + parts[(size_t)cc * PART + 3 * G + t];
    const int j = t / D;
    float il = invl[0];
#pragma unroll
    for (int jj = 1; jj < G; ++jj) il = (jj == j) ? invl[jj] : il;
    ((uint16_t*)a.out)[(size_t)u * G * D + t] = (uint16_t)f32_to_bf16_bits(acc * il);
  }
  if (FEAT && a.window > 0) write_ring2<D, G>(a, u, M, invl, H);
}

// ---------------------------------------------------------------- dispatch
size_t step_lds_bytes(int L, int G, int D, bool feat, int nmoves) {
  const size_t rs = G < 2 ? 2 : G;
  const size_t b = ((size_t)L * rs + (size_t)(SNW / 2) * G * D) * sizeof(float);
  return b + (size_t)2 * (nmoves > 0 ? nmoves : 1) * sizeof(int);
}

bool step_fits(int L, int G, int D, bool feat, int nmoves) {
  return (!feat || L <= S_KMAX * SNT) && step_lds_bytes(L, G, D, feat, nmoves) <= (size_t)S_LDS;
}

int step_chunk_rows() { return SCHUNK; }

template <int D, int G>
static int launch_step_t(const DecodeArgs& a, const EvictArgs* e, bool feat, bool chunked,
                         hipStream_t s) {
  if (!chunked) {
    const int nm = e && e->evict ? (a.L - e->budget < e->budget ? a.L - e->budget : e->budget) : 0;
    const size_t lds = step_lds_bytes(a.L, G, D, feat, nm);
    EvictArgs ee;
    if (e) ee = *e;
    else __builtin_memset(&ee, 0, sizeof(ee));
    auto pick = [&](auto kern) {
      hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hipLaunchKernelGGL(kern, dim3(a.units), dim3(SNT), lds, s, a, ee);
    };
    if (!feat) pick(step_unit_kernel<D, G, false, false, 1>);
    else if (e && e->nh == 2) pick(step_unit_kernel<D, G, true, true, 2>);
    else if (e) pick(step_unit_kernel<D, G, true, true, 1>);
    else pick(step_unit_kernel<D, G, true, false, 1>);
  } else {
    dim3 grid(a.nchunks, a.units);
    if (feat) hipLaunchKernelGGL((stepc_a_kernel<D, G, true>), grid, dim3(SNT), 0, s, a);
    else hipLaunchKernelGGL((stepc_a_kernel<D, G, false>), grid, dim3(SNT), 0, s, a);
    hipLaunchKernelGGL((stepc_b_kernel<D, G>), grid, dim3(SNT), 0, s, a);
    if (feat) hipLaunchKernelGGL((stepc_d_kernel<D, G, true>), grid, dim3(SNT), 0, s, a);
    else hipLaunchKernelGGL((stepc_d_kernel<D, G, false>), grid, dim3(SNT), 0, s, a);
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
