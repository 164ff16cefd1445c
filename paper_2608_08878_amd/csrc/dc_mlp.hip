// Two-hidden-layer policy on matrix cores (Sec. 3.1.2 scoring with the App. D
// network: n_in -> h1 -> h2 -> 1, optional LayerNorm, widths up to 128), gfx950.
//
// Scoring every cached row with a wide second hidden layer is a dense
// contraction, [rows x h1] x [h1 x h2], so it runs on v_mfma_f32_16x16x4_f32
// (float32 operands and accumulation: the same precision as the scalar path).
// The hidden widths are padded to HP = 64 (both at most 64) or 128.  One wave
// takes 16 rows at a time:
//   layer 1 (VALU): lane l computes, for row l % 16, the units k = 4 s + l / 16
//     (s < HP / 4) -- exactly the A operand MFMA step s needs from that lane --
//     with LayerNorm moments reduced over the four lanes that share the row;
//   layer 2 (MFMA): HP / 16 column blocks x HP / 4 k-steps; B comes from W2
//     staged in LDS as [k][n] with a row stride of HP + 16 floats (the four k
//     rows one instruction reads fall in different bank quarters);
//   the accumulators hold row 4 (l / 16) + i, column 16 cb + l % 16: LayerNorm
//     moments, ReLU and the output dot product reduce over the 16 lanes of a
//     DPP row.
// 512-thread workgroups: at HP = 128 the 78 KB of staged weights allow two per
// CU, so eight waves share each copy (four per SIMD); at HP = 64 (23 KB) three.
// Padded units (k >= h1, n >= h2) are exact zeros and are left out of the
// LayerNorm moments.
#include <hip/hip_runtime.h>

#include "dc_mlp.hpp"
#include "dc_select.hpp"

#pragma clang fp contract(off)

namespace dc {

namespace {

constexpr int MT = 512;              // 8 waves share one staged copy of the weights
constexpr int MW = MT / 64;
constexpr int NX = 5;                // padded input width
typedef float f32x4_v __attribute__((ext_vector_type(4)));

// LDS layout (floats) for hidden widths padded to HP (64 or 128); the small
// arrays first, so that every per-lane read of them is a constant offset within
// the 64 KB reach of an LDS instruction
template <int HP>
struct Lay {
  static constexpr int W2S = HP + 16;                 // row stride of W2
  static constexpr int O_W1 = 0;                      // [NX][HP]  W1 transposed (unit-contiguous)
  static constexpr int O_B1 = O_W1 + HP * NX;         // b1, g1, be1       [HP] each
  static constexpr int O_B2 = O_B1 + 3 * HP;          // b2, g2, be2, wo   [HP] each
  static constexpr int O_W2 = O_B2 + 4 * HP;          // [HP][W2S]  W2 as [k][n]
  static constexpr int FLOATS = O_W2 + HP * W2S;
};

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float sum16(float x) {    // over the 16 lanes of a DPP row
  x += dpp_f<0xB1>(x);    // quad_perm [1,0,3,2]
  x += dpp_f<0x4E>(x);    // quad_perm [2,3,0,1]
  x += dpp_f<0x141>(x);   // row_half_mirror
  x += dpp_f<0x140>(x);   // row_mirror
  return x;
}
__device__ __forceinline__ float sum4rows(float x) {  // over lanes l, l^16, l^32, l^48
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

template <int HP>
__device__ void stage(const EvictArgs& a, float* sm) {
  using Y = Lay<HP>;
  constexpr int W2S = Y::W2S, O_W1 = Y::O_W1, O_B1 = Y::O_B1, O_B2 = Y::O_B2, O_W2 = Y::O_W2;
  const cfloat* P = const_params(a.params);
  const int h1 = a.h1, h2 = a.h2, nin = a.n_in, ln = a.ln;
  const cfloat* W1 = P;
  const cfloat* b1 = W1 + h1 * nin;
  const cfloat* g1 = b1 + h1;
  const cfloat* be1 = g1 + h1;
  const cfloat* W2 = b1 + h1 + (ln ? 2 * h1 : 0);
  const cfloat* b2 = W2 + h2 * h1;
  const cfloat* g2 = b2 + h2;
  const cfloat* be2 = g2 + h2;
  const cfloat* wo = b2 + h2 + (ln ? 2 * h2 : 0);
  for (int i = threadIdx.x; i < HP * W2S; i += MT) {
    const int k = i / W2S, n = i % W2S;
    sm[O_W2 + i] = (k < h1 && n < h2) ? W2[n * h1 + k] : 0.0f;
  }
  for (int i = threadIdx.x; i < HP; i += MT) {
    const bool v2 = i < h2, v1 = i < h1;
    sm[O_B2 + i] = v2 ? b2[i] : 0.0f;
    sm[O_B2 + HP + i] = v2 ? (ln ? g2[i] : 1.0f) : 0.0f;
    sm[O_B2 + 2 * HP + i] = v2 && ln ? be2[i] : 0.0f;
    sm[O_B2 + 3 * HP + i] = v2 ? wo[i] : 0.0f;
    sm[O_B1 + i] = v1 ? b1[i] : 0.0f;
    sm[O_B1 + HP + i] = v1 ? (ln ? g1[i] : 1.0f) : 0.0f;
    sm[O_B1 + 2 * HP + i] = v1 && ln ? be1[i] : 0.0f;
#pragma unroll
    for (int x = 0; x < NX; ++x) sm[O_W1 + x * HP + i] = (v1 && x < nin) ? W1[i * nin + x] : 0.0f;
  }
}

template <int HP, int MINB>
__global__ void __launch_bounds__(MT, MINB) score_mlp2_kernel(EvictArgs a, uint64_t* keys, int kstride) {
  using Y = Lay<HP>;
  constexpr int W2S = Y::W2S, O_W1 = Y::O_W1, O_B1 = Y::O_B1, O_B2 = Y::O_B2, O_W2 = Y::O_W2;
  constexpr int NS = HP / 4;     // MFMA k-steps (4 units each)
  constexpr int NC = HP / 16;    // 16-column blocks of layer 2
  extern __shared__ float sm[];
  // a unit that keeps every row reads no key (the whole workgroup leaves)
  if (unit_rows(a, a.y0 + blockIdx.y) <= a.fused_rows) return;    // served by the single-launch step
  if (!a.scores_out && unit_budget(a, a.y0 + blockIdx.y) >= unit_rows(a, a.y0 + blockIdx.y)) return;
  stage<HP>(a, sm);
  __syncthreads();
  const int u = a.y0 + blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ri = lane & 15, kg = lane >> 4;
  const int h1 = a.h1, h2 = a.h2, ln = a.ln;
  const int L = unit_rows(a, u);   // this unit's rows (scores_out keeps stride a.L)
  // LayerNorm: the moments multiply by 1 / width (one rounding more than a
  // division, far inside the score tolerance) and the scale uses the
  // hardware reciprocal square root: the IEEE division sequences cost about a
  // tenth of the kernel's VALU work, which adds to the matrix-core time here
  const float ih1 = 1.0f / (float)h1, ih2 = 1.0f / (float)h2;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  const float bout = const_params(a.params)[h1 * a.n_in + h1 + (ln ? 2 * h1 : 0) + h2 * h1 + h2 +
                                            (ln ? 2 * h2 : 0) + h2];
  // features of this lane's A row (the four lanes of a row load the same row);
  // the next row block's are requested while the current one is computed
  struct Feat {
    double num, den;
    int32_t pos;
    float al, vn, sg;
  };
  const float* sig = a.n_in == 5 ? a.sigma : a.alpha;   // (a dummy read for four inputs)
  auto fetch = [&](int rbx, Feat& f) {
    const int r = rbx + ri;
    const size_t gi = ub + (r < L ? r : L - 1);             // past the end: re-read, unused
    f.num = a.num[gi];
    f.den = a.den[gi];
    f.pos = a.pos[gi];
    f.al = a.alpha[gi];
    f.vn = a.vnorm[gi];
    f.sg = sig[gi];
  };
  const int stride = gridDim.x * MW * 16;
  int rb = (blockIdx.x * MW + wave) * 16;
  Feat nxt;
  fetch(rb, nxt);
  for (; rb < L; rb += stride) {
    const Feat f = nxt;
    fetch(rb + stride, nxt);
    float x[NX];
    {
      const float H = f.den > 0.0 ? (float)(f.num / f.den) : 0.0f;
      const float ps = (float)f.pos * invT;
      x[0] = f.al;
      x[1] = f.vn;
      if (a.n_in == 5) {
        x[2] = f.sg;
        x[3] = H;
        x[4] = ps;
      } else {
        x[2] = H;
        x[3] = ps;
        x[4] = 0.0f;
      }
    }
    // layer 1: units k = 4 s + kg (the weights are re-read from LDS per row
    // block: held across blocks they would take 256 registers)
    const lfloat* p1 = (const lfloat*)sm + kg;  // LDS, this lane's unit offset; all reads below
    asm volatile("" : "+v"(p1));                // are constant offsets from it
    float h[NS];
    float s1 = 0.0f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int k = 4 * s + kg;
      float z = p1[O_B1 + 4 * s];
#pragma unroll
      for (int i = 0; i < NX; ++i) z = __builtin_fmaf(p1[O_W1 + i * HP + 4 * s], x[i], z);
      h[s] = z;
      s1 += k < h1 ? z : 0.0f;
    }
    if (ln) {
      const float mean = sum4rows(s1) * ih1;
      float s2 = 0.0f;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const float d = h[s] - mean;
        s2 += (4 * s + kg) < h1 ? d * d : 0.0f;
      }
      const float rs = __builtin_amdgcn_rsqf(__builtin_fmaf(sum4rows(s2), ih1, LN_EPS));
#pragma unroll
      for (int s = 0; s < NS; ++s)
        h[s] = __builtin_fmaf((h[s] - mean) * rs, p1[O_B1 + HP + 4 * s], p1[O_B1 + 2 * HP + 4 * s]);
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) h[s] = (4 * s + kg) < h1 ? fmaxf(h[s], 0.0f) : 0.0f;
    // layer 2 on MFMA
    f32x4_v acc[NC];
#pragma unroll
    for (int cb = 0; cb < NC; ++cb) acc[cb] = (f32x4_v){0.0f, 0.0f, 0.0f, 0.0f};
    // B of step s + 1 is read while step s's MFMAs run (an opaque pointer per step
    // keeps the reads from being hoisted further ahead: the whole of W2 would not fit)
    float bq[2][NC];
    {
      const lfloat* br = (const lfloat*)sm + O_W2 + kg * W2S + ri;
      asm volatile("" : "+v"(br));
#pragma unroll
      for (int cb = 0; cb < NC; ++cb) bq[0][cb] = br[16 * cb];
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (s + 1 < NS) {
        const lfloat* br = (const lfloat*)sm + O_W2 + (4 * (s + 1) + kg) * W2S + ri;
        asm volatile("" : "+v"(br));
#pragma unroll
        for (int cb = 0; cb < NC; ++cb) bq[(s + 1) & 1][cb] = br[16 * cb];
      }
#pragma unroll
      for (int cb = 0; cb < NC; ++cb)
        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(h[s], bq[s & 1][cb], acc[cb], 0, 0, 0);
    }
    // rows 4 kg + i of the block, columns 16 cb + ri
    float score[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float z[NC];
      float t1 = 0.0f;
#pragma unroll
      for (int cb = 0; cb < NC; ++cb) {
        const int n = 16 * cb + ri;
        z[cb] = acc[cb][i] + sm[O_B2 + n];
        t1 += n < h2 ? z[cb] : 0.0f;
      }
      float mean = 0.0f, rs = 1.0f;
      if (ln) {
        mean = sum16(t1) * ih2;
        float t2 = 0.0f;
#pragma unroll
        for (int cb = 0; cb < NC; ++cb) {
          const float d = z[cb] - mean;
          t2 += (16 * cb + ri) < h2 ? d * d : 0.0f;
        }
        rs = __builtin_amdgcn_rsqf(__builtin_fmaf(sum16(t2), ih2, LN_EPS));
      }
      float o = 0.0f;
#pragma unroll
      for (int cb = 0; cb < NC; ++cb) {
        const int n = 16 * cb + ri;
        float y = ln ? __builtin_fmaf((z[cb] - mean) * rs, sm[O_B2 + HP + n], sm[O_B2 + 2 * HP + n])
                     : z[cb];
        o = __builtin_fmaf(sm[O_B2 + 3 * HP + n], fmaxf(y, 0.0f), o);   // padded units: wo = 0
      }
      score[i] = sum16(o) + bout;
    }
    // lanes ri < 4 of each row group write rows 4 kg + ri; lane 4 kg + ri
    // loaded that row's position with its features
    const int32_t p = __shfl(f.pos, 4 * kg + (ri & 3));
    if (ri < 4) {
      const int row = rb + 4 * kg + ri;
      float sc = score[0];
#pragma unroll
      for (int i = 1; i < 4; ++i) sc = ri == i ? score[i] : sc;
      if (row < L) {
        if (a.scores_out) a.scores_out[(size_t)u * a.L + row] = sc;
        keys[(size_t)u * kstride + row] = row_key(a.sample ? sampled_score(a, sc, p, u) : sc, p);
      }
    }
  }
}

}  // namespace

int launch_score_mlp2(const EvictArgs& a, uint64_t* keys, int kstride, void* stream) {
  const int nblk = (a.L + MW * 16 - 1) / (MW * 16);
  const int gx = nblk < 8 ? nblk : 8;
  // hidden widths up to 64 pad to 64: a quarter of the layer-2 work of 128
  const bool narrow = a.h1 <= 64 && a.h2 <= 64;
  const void* k = narrow ? (const void*)score_mlp2_kernel<64, 3> : (const void*)score_mlp2_kernel<128, 2>;
  const size_t lds = (size_t)(narrow ? Lay<64>::FLOATS : Lay<128>::FLOATS) * sizeof(float);
  hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  for_grid_y(a.units, [&](int y0, int ny) {
    EvictArgs b = a;
    b.y0 = y0;
    if (narrow)
      hipLaunchKernelGGL((score_mlp2_kernel<64, 3>), dim3(gx, ny), dim3(MT), lds, (hipStream_t)stream,
                         b, keys, kstride);
    else
      hipLaunchKernelGGL((score_mlp2_kernel<128, 2>), dim3(gx, ny), dim3(MT), lds, (hipStream_t)stream,
                         b, keys, kstride);
  });
  return (int)hipGetLastError();
}

}  // namespace dc
