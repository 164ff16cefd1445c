// Two-hidden-layer policy on matrix cores (Sec. 3.1.2 scoring with the App. D
// network: n_in -> h1 -> h2 -> 1, optional LayerNorm, widths up to 128), gfx950.
//
// Scoring every cached row is two dense contractions, [rows x n_in] x
// [n_in x h1] and [rows x h1] x [h1 x h2].  On this part the float32 matrix
// instructions run at the float32 vector rate and do not overlap the vector
// work around them, so both run on the bf16 matrix cores instead,
// at float32 accuracy: every float32 operand x is split exactly into three
// bf16 parts x = xh + xm + xl (8 significand bits each: 24 in all; |xm| and
// |xl| about 2^-8 and 2^-16 of |x|), and the product of an activation h and a
// weight w keeps the six part products down to about 2^-16 of it,
// hl wh + hm wm + hh wl + hm wh + hh wm + hh wh (each exact in float32,
// accumulated in float32 by v_mfma_f32_16x16x32_bf16); the three dropped ones
// (hm wl, hl wm, hl wl) come to about 2^-23 of the product, one float32
// rounding.  The hidden widths are padded to HP = 64 (both at most 64) or
// 128.  One wave takes 16 rows at a time:
//   layer 1 (MFMA, the same split, inputs padded to 32): per 16-unit block b,
//     W1 (16 units x 32 inputs) times the rows' features (32 x 16 rows), so
//     lane (i, g) receives units 16 b + 4 g + r (r < 4) of row i, with
//     LayerNorm moments reduced over the four lanes that share the row;
//   layer 2 (MFMA): HP / 16 column blocks x HP / 32 k-steps x 6 part products;
//     k-step t takes from lane (i, g) the units 32 t + 4 g + r and
//     32 t + 16 + 4 g + r (r < 4) that layer 1 left in it, and the weight
//     parts sit in LDS as three [n][k] bf16 arrays in that unit order, with
//     a row stride of 2 HP + 16 bytes (the 16 rows one read touches start 16
//     bytes apart in the banks); all weight parts are split once per
//     workgroup;
//   the accumulators hold row 4 (l / 16) + i, column 16 cb + l % 16: LayerNorm
//     moments, ReLU and the output dot product reduce over the 16 lanes of a
//     DPP row.
// HP = 128: 1024-thread workgroups (138 KB of LDS, one per CU, four waves per
// SIMD); HP = 64: 512 threads (44 KB, two per CU).  Padded units (k >= h1,
// n >= h2) are exact zeros and are left out of the LayerNorm moments.
#include <hip/hip_runtime.h>

#include "dc_mlp.hpp"
#include "dc_select.hpp"

#pragma clang fp contract(off)

namespace dc {

namespace {

constexpr int NX = 5;                // features per row (the fifth is 0 for four-input policies)
typedef float f32x4_v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) const char lchar;

template <int HP>
struct Cfg {
  static constexpr int MT = HP == 128 ? 1024 : 512;    // threads per workgroup
  static constexpr int MINB = HP == 128 ? 1 : 2;       // workgroups per CU
  static constexpr int MW = MT / 64;                   // waves
};

// LDS layout for hidden widths padded to HP (64 or 128): the float arrays
// first, so that every per-lane read of them is a constant offset within the
// 64 KB reach of an LDS instruction, then the three bf16 parts of W2
template <int HP>
struct Lay {
  static constexpr int RS = 2 * HP + 16;              // bytes per W2 row (unit n, k in k-step order)
  static constexpr int RS1 = 64 + 16;                 // bytes per W1 row (unit, 32 padded inputs)
  static constexpr int O_B1 = 0;                      // floats: b1, g1, be1       [HP] each
  static constexpr int O_B2 = O_B1 + 3 * HP;          // b2, g2, be2, wo   [HP] each
  static constexpr int FLOATS = O_B2 + 4 * HP;
  static constexpr int O_W2 = FLOATS * 4;             // bytes: parts h, m, l, [3][HP][RS]
  static constexpr int O_W1 = O_W2 + 3 * HP * RS;     // bytes: parts h, m, l, [3][HP][RS1]
  static constexpr int BYTES = O_W1 + 3 * HP * RS1;
};

// position, within its row of W2's parts, of unit k: k-step t = k / 32 holds
// lane group g's units 32 t + 4 g + r and 32 t + 16 + 4 g + r (r < 4) at
// bytes 2 (32 t + 8 g) .. + 16
__host__ __device__ constexpr int w2_pos(int k) {
  return (k & ~31) + ((k & 31) < 16 ? 8 * ((k & 15) >> 2) + (k & 3) : 8 * ((k & 15) >> 2) + 4 + (k & 3));
}

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

// x = h + m + l exactly (three round-to-nearest bf16 parts; each residual is
// exact in float32: it holds at most the 16, then 8, bits below the part taken)
__device__ __forceinline__ void split3(float x, __bf16& h, __bf16& m, __bf16& l) {
  h = (__bf16)x;
  const float r1 = x - (float)h;
  m = (__bf16)r1;
  const float r2 = r1 - (float)m;
  l = (__bf16)r2;
}

// the same for eight values, two at a time (one packed conversion per part
// and pair)
typedef float f32x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void split3x8(const float (&v)[8], bf16x8_t& h, bf16x8_t& m, bf16x8_t& l) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const f32x2_v x = {v[2 * p], v[2 * p + 1]};
    const bf16x2_t xh = __builtin_convertvector(x, bf16x2_t);
    const f32x2_v r1 = x - __builtin_convertvector(xh, f32x2_v);
    const bf16x2_t xm = __builtin_convertvector(r1, bf16x2_t);
    const f32x2_v r2 = r1 - __builtin_convertvector(xm, f32x2_v);
    const bf16x2_t xl = __builtin_convertvector(r2, bf16x2_t);
    h[2 * p] = xh[0];
    h[2 * p + 1] = xh[1];
    m[2 * p] = xm[0];
    m[2 * p + 1] = xm[1];
    l[2 * p] = xl[0];
    l[2 * p + 1] = xl[1];
  }
}

template <int HP>
__device__ void stage(const EvictArgs& a, float* sm) {
  using Y = Lay<HP>;
  constexpr int MT = Cfg<HP>::MT, RS = Y::RS, RS1 = Y::RS1, O_B1 = Y::O_B1, O_B2 = Y::O_B2;
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
  char* w2 = reinterpret_cast<char*>(sm) + Y::O_W2;
  for (int e = threadIdx.x; e < HP * HP; e += MT) {
    const int n = e / HP, k = e % HP;
    __bf16 wh, wm, wl;
    split3((k < h1 && n < h2) ? W2[n * h1 + k] : 0.0f, wh, wm, wl);
    const int q = 2 * w2_pos(k);
    *reinterpret_cast<__bf16*>(w2 + n * RS + q) = wh;
    *reinterpret_cast<__bf16*>(w2 + (HP + n) * RS + q) = wm;
    *reinterpret_cast<__bf16*>(w2 + (2 * HP + n) * RS + q) = wl;
  }
  char* w1 = reinterpret_cast<char*>(sm) + Y::O_W1;
  for (int e = threadIdx.x; e < HP * 32; e += MT) {
    const int k = e / 32, x = e % 32;
    __bf16 wh, wm, wl;
    split3((k < h1 && x < nin) ? W1[k * nin + x] : 0.0f, wh, wm, wl);
    *reinterpret_cast<__bf16*>(w1 + k * RS1 + 2 * x) = wh;
    *reinterpret_cast<__bf16*>(w1 + (HP + k) * RS1 + 2 * x) = wm;
    *reinterpret_cast<__bf16*>(w1 + (2 * HP + k) * RS1 + 2 * x) = wl;
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
  }
}

// FULL: both hidden widths equal HP (no padded units, no masks)
template <int HP, bool LN, bool FULL>
__global__ void __launch_bounds__(Cfg<HP>::MT, Cfg<HP>::MINB)
score_mlp2_kernel(EvictArgs a, uint64_t* keys, int kstride) {
  using Y = Lay<HP>;
  constexpr int MW = Cfg<HP>::MW, RS = Y::RS, RS1 = Y::RS1, O_B1 = Y::O_B1, O_B2 = Y::O_B2;
  constexpr int NT = HP / 32;    // MFMA k-steps (32 units each)
  constexpr int NB = HP / 16;    // 16-unit blocks of layer 1
  constexpr int NC = HP / 16;    // 16-column blocks of layer 2
  extern __shared__ float sm[];
  // a unit that keeps every row reads no key (the whole workgroup leaves)
  if (unit_rows(a, a.y0 + blockIdx.y) <= a.fused_rows) return;    // served by the single-launch step
  if (!a.scores_out && unit_budget(a, a.y0 + blockIdx.y) >= unit_rows(a, a.y0 + blockIdx.y)) return;
  stage<HP>(a, sm);
  __syncthreads();
  const int u = a.y0 + blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ri = lane & 15, kg = lane >> 4;
  const int h1 = a.h1, h2 = a.h2;
  const int L = unit_rows(a, u);   // this unit's rows (scores_out keeps stride a.L)
  // LayerNorm: the moments multiply by 1 / width (one rounding more than a
  // division, far inside the score tolerance) and the scale uses the
  // hardware reciprocal square root
  const float ih1 = 1.0f / (float)h1, ih2 = 1.0f / (float)h2;
  const size_t ub = (size_t)u * a.cap;
  const float invT = 1.0f / (float)a.T;
  const float bout = const_params(a.params)[h1 * a.n_in + h1 + (LN ? 2 * h1 : 0) + h2 * h1 + h2 +
                                            (LN ? 2 * h2 : 0) + h2];
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
    // layer 1 on the matrix cores: per 16-unit block b, D = W1 x X^T with the
    // inputs padded to 32 (lanes kg > 0 supply zeros), so lane (ri, kg) gets
    // units 16 b + 4 kg + r of its row ri, accumulated onto their biases.
    // Padded units (k >= h1) have zero weights, bias, gain and shift, so they
    // come out exactly 0 here, after the LayerNorm and after the ReLU: only
    // the variance sum needs a mask (none when FULL).
    typedef __attribute__((address_space(3))) const f32x4_v lfloat4;
    typedef __attribute__((address_space(3))) const bf16x8_t lbf16x8;
    bf16x8_t xh, xm, xl;
    {
      float v[8] = {x[0], x[1], x[2], x[3], x[4], 0.0f, 0.0f, 0.0f};
      split3x8(v, xh, xm, xl);
      if (kg != 0) {
        const bf16x8_t zero = {};
        xh = zero;
        xm = zero;
        xl = zero;
      }
    }
    const lfloat* p1 = (const lfloat*)sm + 4 * kg;   // LDS, this lane's unit offset in a block
    const lchar* w1 = (const lchar*)sm + Y::O_W1 + ri * RS1 + 16 * kg;
    asm volatile("" : "+v"(p1), "+v"(w1));
    f32x4_v hv[NB];
    float s1 = 0.0f;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const lchar* wb = w1 + 16 * b * RS1;
      const bf16x8_t wh = *reinterpret_cast<lbf16x8*>(wb);
      const bf16x8_t wm = *reinterpret_cast<lbf16x8*>(wb + HP * RS1);
      const bf16x8_t wl = *reinterpret_cast<lbf16x8*>(wb + 2 * HP * RS1);
      f32x4_v c = *reinterpret_cast<lfloat4*>(p1 + O_B1 + 16 * b);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wl, xh, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wm, xm, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wh, xl, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wm, xh, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wh, xm, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wh, xh, c, 0, 0, 0);
      hv[b] = c;
#pragma unroll
      for (int r = 0; r < 4; ++r) s1 += c[r];
    }
    if (LN) {
      const float mean = sum4rows(s1) * ih1;
      float s2 = 0.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = hv[b][r] - mean;
          hv[b][r] = d;
          if (FULL || (16 * b + 4 * kg + r) < h1) s2 = __builtin_fmaf(d, d, s2);
        }
      const float rs = __builtin_amdgcn_rsqf(__builtin_fmaf(sum4rows(s2), ih1, LN_EPS));
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x4_v g = *reinterpret_cast<lfloat4*>(p1 + O_B1 + HP + 16 * b);
        const f32x4_v be = *reinterpret_cast<lfloat4*>(p1 + O_B1 + 2 * HP + 16 * b);
#pragma unroll
        for (int r = 0; r < 4; ++r) hv[b][r] = __builtin_fmaf(hv[b][r] * rs, g[r], be[r]);
      }
    }
    // layer 2 on the bf16 matrix cores, six part products per k-step and
    // block, accumulated onto the bias of the lane's column
    f32x4_v acc[NC];
#pragma unroll
    for (int cb = 0; cb < NC; ++cb) {
      const float bn = sm[O_B2 + 16 * cb + ri];
      acc[cb] = (f32x4_v){bn, bn, bn, bn};
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      bf16x8_t ah, am, al;
      float v[8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {            // ReLU; units 32 t + 4 kg + r, then + 16
        v[r] = fmaxf(hv[2 * t][r], 0.0f);
        v[4 + r] = fmaxf(hv[2 * t + 1][r], 0.0f);
      }
      split3x8(v, ah, am, al);
      // the weight rows of column block cb, this lane's 8 units of k-step t, at
      // bytes 2 (32 t + 8 kg) .. + 16 of each row in that order (an
      // opaque pointer per k-step keeps the reads from being hoisted out of the
      // row loop: all of W2's parts would not fit in registers)
      const lchar* w2 = (const lchar*)sm + Y::O_W2 + ri * RS + (32 * t + 8 * kg) * 2;
      asm volatile("" : "+v"(w2));
#pragma unroll
      for (int cb = 0; cb < NC; ++cb) {
        const bf16x8_t bh = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
            w2 + 16 * cb * RS);
        const bf16x8_t bm = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
            w2 + (HP + 16 * cb) * RS);
        const bf16x8_t bl = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
            w2 + (2 * HP + 16 * cb) * RS);
        f32x4_v c = acc[cb];
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bm, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bh, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bm, c, 0, 0, 0);
        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, c, 0, 0, 0);
      }
    }
    // rows 4 kg + i of the block, columns 16 cb + ri (padded columns: weights,
    // bias, gain and shift 0, so exactly 0 but in the variance sum)
    float score[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float z[NC];
      float t1 = 0.0f;
#pragma unroll
      for (int cb = 0; cb < NC; ++cb) {
        z[cb] = acc[cb][i];
        t1 += z[cb];
      }
      float rs = 1.0f;
      if (LN) {
        const float mean = sum16(t1) * ih2;
        float t2 = 0.0f;
#pragma unroll
        for (int cb = 0; cb < NC; ++cb) {
          const float d = z[cb] - mean;
          z[cb] = d;
          if (FULL || (16 * cb + ri) < h2) t2 = __builtin_fmaf(d, d, t2);
        }
        rs = __builtin_amdgcn_rsqf(__builtin_fmaf(sum16(t2), ih2, LN_EPS));
      }
      float o = 0.0f;
#pragma unroll
      for (int cb = 0; cb < NC; ++cb) {
        const int n = 16 * cb + ri;
        float y = LN ? __builtin_fmaf(z[cb] * rs, sm[O_B2 + HP + n], sm[O_B2 + 2 * HP + n]) : z[cb];
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
  // hidden widths up to 64 pad to 64: a quarter of the layer-2 work of 128
  const bool narrow = a.h1 <= 64 && a.h2 <= 64;
  const int mw = narrow ? Cfg<64>::MW : Cfg<128>::MW;
  const int nblk = (a.L + mw * 16 - 1) / (mw * 16);
  // workgroups per unit: enough for about 2048 in all, each staging the weight
  // parts once for as many rows as possible
  int gx = (2048 + a.units - 1) / a.units;
  gx = gx < nblk ? gx : nblk;
  gx = gx > 0 ? gx : 1;
  const bool ln = a.ln != 0;
  const bool full = narrow ? (a.h1 == 64 && a.h2 == 64) : (a.h1 == 128 && a.h2 == 128);
  const size_t lds = (size_t)(narrow ? Lay<64>::BYTES : Lay<128>::BYTES);
  const int variant = (narrow ? 4 : 0) + (ln ? 2 : 0) + (full ? 1 : 0);
  auto launch = [&](auto kern, int mt) {
    hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    for_grid_y(a.units, [&](int y0, int ny) {
      EvictArgs b = a;
      b.y0 = y0;
      hipLaunchKernelGGL(kern, dim3(gx, ny), dim3(mt), lds, (hipStream_t)stream, b, keys, kstride);
    });
  };
  switch (variant) {
    case 0: launch(score_mlp2_kernel<128, false, false>, Cfg<128>::MT); break;
    case 1: launch(score_mlp2_kernel<128, false, true>, Cfg<128>::MT); break;
    case 2: launch(score_mlp2_kernel<128, true, false>, Cfg<128>::MT); break;
    case 3: launch(score_mlp2_kernel<128, true, true>, Cfg<128>::MT); break;
    case 4: launch(score_mlp2_kernel<64, false, false>, Cfg<64>::MT); break;
    case 5: launch(score_mlp2_kernel<64, false, true>, Cfg<64>::MT); break;
    case 6: launch(score_mlp2_kernel<64, true, false>, Cfg<64>::MT); break;
    default: launch(score_mlp2_kernel<64, true, true>, Cfg<64>::MT); break;
  }
  return (int)hipGetLastError();
}

}  // namespace dc
