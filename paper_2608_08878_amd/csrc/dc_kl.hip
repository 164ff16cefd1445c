// Per-step KL reward, KL(P || Q) with P = softmax(h_full W^T), Q = softmax(h_comp W^T)
// (reward R_t = -KL of Sec. 3.1.4), on gfx950 matrix cores.
//
// Numerics.  With delta_v = l_v - l^_v (full minus compressed logit) and
// mu = E_P[delta],
//     KL = E_P[delta] + ln E_P[exp(-delta)] = ln E_P[exp(mu - delta)]
//        = log1p( E_P[ g(mu - delta) ] ),   g(y) = e^y - 1 - y >= 0,
// since E_P[mu - delta] = 0.  Every term is non-negative, so nothing cancels
// even when KL is tiny (a direct "sum P (log P - log Q)" in float32 loses the
// answer to the rounding of the two log-sum-exps), and identical rows give
// exactly 0.  Q's normaliser never appears.
//
// Kernel 1 (up to 64 rows: kl_tile_kernel, one workgroup per 64 vocabulary
// columns and 8, 16, 32 or 64 rows; more rows: the blocked GEMMs below, same
// arithmetic): MFMA
// 16x16x32 bf16 over the hidden dimension for a 16-row A = [8 full rows; the 8
// matching compressed rows], then per (row, 64-column tile) the local statistics
//     m_t = max l,  s_t = sum e^{l - m_t},  mu_t = E_{P_t}[delta],
//     A_t = E_{P_t}[g(mu_t - delta)]
// where P_t is P restricted to the tile.  Kernel 2 merges the tiles exactly:
//     w_t = s_t e^{m_t - M} / S,  mu = sum w_t mu_t,  x_t = mu - mu_t,
//     KL = log1p( sum_t w_t (g(x_t) + e^{x_t} A_t) ).
#include <mutex>

#include "dc_device.hpp"
#include "dc_kernels.hpp"
#include "distillcache.h"

#pragma clang fp contract(off)

namespace dc {

constexpr int KL_WAVES = 4;
constexpr int KL_TILE = 16 * KL_WAVES;   // vocabulary columns per workgroup
constexpr int KL_BK = 64;                // hidden elements per stage (128 bytes of a row)
constexpr int KL_NS = 5;                 // stage buffers (50 KB: two workgroups per CU)

typedef __attribute__((address_space(3))) char lds_char_t;

__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// 16 bytes per lane from global memory to LDS byte lds + 16 lane (lds uniform).
// Issued from inline assembly, out of the compiler's sight: the caller waits
// for it explicitly (vmcnt; loads complete in issue order).  A load into LDS
// needs one wait state after a scalar write of M0 (the s_nop).
__device__ __forceinline__ void load_to_lds16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               : : "v"(g), "s"(lds) : "memory", "m0");
}
// The same with the non-temporal hint: for data read once per call (the
// per-step kernel's lm head), which then does not displace cached lines --
// dirty lines of earlier kernels among them, whose write-back would otherwise
// share the HBM with the stream.
__device__ __forceinline__ void load_to_lds16_nt(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
               : : "v"(g), "s"(lds) : "memory", "m0");
}

// Byte offset of vocabulary row v's first hidden element in the lm head: the
// row-major weight and the packed tile layout differ only in where a 64-row
// tile's rows and 64-element stages sit (KLArgs::w_row, w_stage).
static_assert(KL_TILE == 64, "lm-head tiles of 64 vocabulary rows");
__device__ __forceinline__ size_t w_row_off(const KLArgs& a, int v) {
  return (size_t)(v >> 6) * 128 * (size_t)a.hidden + (size_t)(v & 63) * (size_t)a.w_row;
}

// g(y) = e^y - 1 - y without cancellation.
__device__ __forceinline__ float gfun(float y) {
  const float ay = fabsf(y);
  if (ay < 0.5f) {
    // y^2 (1/2! + y (1/3! + ... + y / 9!)), Horner with fused multiply-adds
    float t = fmaf(y, 1.0f / 362880.0f, 1.0f / 40320.0f);
    t = fmaf(y, t, 1.0f / 5040.0f);
    t = fmaf(y, t, 1.0f / 720.0f);
    t = fmaf(y, t, 1.0f / 120.0f);
    t = fmaf(y, t, 1.0f / 24.0f);
    t = fmaf(y, t, 1.0f / 6.0f);
    t = fmaf(y, t, 0.5f);
    return (y * y) * t;
  }
  return expm1f(y) - y;
}

__device__ __forceinline__ float sum16(float x) {   // over the 16 lanes of a DPP row
  x += dpp<DPP_XOR1>(x);
  x += dpp<DPP_XOR2>(x);
  x += dpp<DPP_HALF_MIRROR>(x);
  x += dpp<DPP_MIRROR>(x);
  return x;
}
__device__ __forceinline__ float max16(float x) {
  x = fmaxf(x, dpp<DPP_XOR1>(x));
  x = fmaxf(x, dpp<DPP_XOR2>(x));
  x = fmaxf(x, dpp<DPP_HALF_MIRROR>(x));
  x = fmaxf(x, dpp<DPP_MIRROR>(x));
  return x;
}

// A workgroup serves RB blocks of 8 kl rows (1, 2, 4 or 8): each block is
// its own 16-row A operand (8 full, then the 8 compressed hidden states), and
// every lm-head stage in LDS feeds the matrix cores for all of them, so a
// call of up to 8 RB rows streams the lm head once.  The stage ring is five
// deep, four for RB = 4 and three for RB = 8 (two workgroups per CU).
template <int RB>
struct KLT {
  static constexpr int NS = RB == 8 ? 3 : RB == 4 ? 4 : KL_NS;    // stage buffers
  static constexpr int AB = 16 * RB * KL_BK * 2;                 // A bytes of a stage
  static constexpr int STG = AB + KL_TILE * KL_BK * 2;           // bytes of a stage
};

// grid: 8 ceil(tiles / 8) ceil(rows / (8 RB)) workgroups of 256 threads (4
// waves).  Workgroups are dealt to the 8 XCDs round-robin by index, so index
// g runs on XCD g mod 8; every row group of one 64-column vocabulary tile is
// given to the same XCD back to back.
template <int RB>
__global__ void __launch_bounds__(64 * KL_WAVES) kl_tile_kernel(KLArgs a) {
  constexpr int NS = KLT<RB>::NS, AB = KLT<RB>::AB, STG = KLT<RB>::STG;
  __shared__ float red[KL_WAVES][8];        // per-wave row maxima
  __shared__ __attribute__((aligned(1024))) char ring[NS * STG];
  __shared__ float4 xp[KL_WAVES][32], xd[KL_WAVES][32], xg[KL_WAVES][32];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nrb = (a.rows + 8 * RB - 1) / (8 * RB);
  const int slot = blockIdx.x >> 3;
  const int tile = (blockIdx.x & 7) + 8 * (slot / nrb), rb = slot % nrb;
  if (tile >= a.ntiles) return;      // whole workgroup: no barrier is skipped
  const int i = lane & 15, kg = lane >> 4;        // MFMA row/col index, k group
  // The hidden dimension goes in stages of 64 elements, every row read as one
  // 128-byte line: a stage holds the 16 RB A rows (block b: rows 16 b .. 16 b
  // + 7 the full, 16 b + 8 .. 16 b + 15 the compressed hidden states of kl
  // rows (rb RB + b) 8 + 0..7) and the workgroup's 64 lm-head rows, loaded
  // straight into LDS (global_load_lds_dwordx4) through a ring of NS stage
  // buffers, NS - 2 stages in flight while one feeds the matrix cores.  A
  // load instruction covers 8 rows x 128 bytes (the A rows: 4 rows, half a
  // wave); row r's 16-byte chunk c sits at position c ^ (r mod 8) of its 128
  // LDS bytes (lane j loads the chunk that lands at byte 16 j), so the
  // operand reads hit eight bank groups per eight lanes.  MFMA t of a stage
  // takes chunk 4t + kg of both operands: the blocks feed the matrix cores in
  // hidden order, as in the GEMM kernels.  The lm-head loads are non-temporal
  // (each slab is read by a tile's row groups back to back on one XCD); the
  // hidden-state rows, which every tile reads, are not.  Where a row's stage
  // sits in the lm head (row-major or packed tiles) is KLArgs::w_row /
  // w_stage.  Every load is unconditional (past the end a stage re-reads the
  // last one), so each wave issues RB + 2 loads per stage and a wait counts
  // stages exactly.
  const int lrow = lane >> 3;
  const char* asrc[RB];
#pragma unroll
  for (int q = 0; q < RB; ++q) {
    const int ar = 4 * (wave + 4 * q) + lrow;      // A row of this lane's load q (lanes 0..31)
    int kr = (rb * RB + (ar >> 4)) * 8 + (ar & 7);
    kr = kr < a.rows ? kr : a.rows - 1;            // past the end: re-read, unused
    asrc[q] = (const char*)((ar & 15) < 8 ? a.h_full : a.h_comp) +
              ((size_t)kr * a.hidden + 8 * ((lane & 7) ^ (ar & 7))) * 2;
  }
  const char* wsrc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    wsrc[j] = (const char*)a.w + w_row_off(a, tile * KL_TILE + 8 * (2 * wave + j) + lrow) +
              16 * ((lane & 7) ^ lrow);
  const int S = a.hidden / KL_BK;
  const uint32_t ring_lds = (uint32_t)(size_t)(lds_char_t*)ring;
  auto issue = [&](int st) {
    const int sc = st < S ? st : S - 1;
    // (uniform: the LDS address goes to M0 through a scalar register)
    const uint32_t base = __builtin_amdgcn_readfirstlane(ring_lds + (st % NS) * STG);
    const size_t offw = (size_t)a.w_stage * sc;
#pragma unroll
    for (int q = 0; q < RB; ++q)
      if (lane < 32) load_to_lds16(asrc[q] + 2 * KL_BK * sc, base + (wave + 4 * q) * 512);
    load_to_lds16_nt(wsrc[0] + offw, base + AB + (2 * wave) * 1024);
    load_to_lds16_nt(wsrc[1] + offw, base + AB + (2 * wave + 1) * 1024);
  };
  f32x4_t acc[RB];
#pragma unroll
  for (int b = 0; b < RB; ++b) acc[b] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
  auto mma = [&](const char* X) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int pos = ((4 * t + kg) ^ (i & 7)) << 4;
      const uint4 bv = *reinterpret_cast<const uint4*>(X + AB + (16 * wave + i) * 128 + pos);
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        const uint4 av = *reinterpret_cast<const uint4*>(X + (16 * b + i) * 128 + pos);
        acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                         __builtin_bit_cast(bf16x8_t, bv), acc[b],
                                                         0, 0, 0);
      }
    }
  };
  for (int st = 0; st < NS - 1; ++st) issue(st);
  for (int st = 0; st < S; ++st) {
    // this wave's loads of stage st have landed (NS - 2 later stages may be
    // in flight); after the barrier every wave's have, and every wave is done
    // with stage st - 1, whose buffer the next issue refills
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"((RB + 2) * (NS - 2)) : "memory");
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(st + NS - 1);
    mma(ring + (st % NS) * STG);
  }
  asm volatile("s_waitcnt vmcnt(0)" : : : "memory");   // no load into LDS outlives the loop
  compiler_fence();
  // block b's statistics: lane holds C[4*kg + r][i] for r < 4: kg 0,1 full
  // rows 0..7, kg 2,3 compressed rows 0..7
  auto epilogue = [&](const f32x4_t& c, int blk) {
    float lf[4], lc[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float x = c[r];
      const float y = __shfl_xor(x, 32);
      lf[r] = x;   // meaningful in lanes 0..31
      lc[r] = y;
    }
    // per kl row rho = 4*kg + r (lanes 0..31): statistics over this workgroup's
    // 64 columns, wave w holding columns 16 w .. 16 w + 15.  The maximum goes
    // through red; every sum adds the four waves' terms of a column lane by
    // lane in column order, then the 16 lanes (the blocked GEMMs' order, where
    // one lane holds all four blocks).
    float m[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) m[r] = max16(lf[r]);
    if (lane < 32 && i == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][4 * kg + r] = m[r];
    __syncthreads();
    float p[4], d[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rho = 4 * (kg & 1) + r;
      float M = red[0][rho];
      for (int w = 1; w < KL_WAVES; ++w) M = fmaxf(M, red[w][rho]);
      m[r] = M;
      p[r] = __expf(lf[r] - M);
      d[r] = lf[r] - lc[r];
    }
    if (lane < 32) {
      xp[wave][lane] = make_float4(p[0], p[1], p[2], p[3]);
      xd[wave][lane] = make_float4(p[0] * d[0], p[1] * d[1], p[2] * d[2], p[3] * d[3]);
    }
    __syncthreads();
    float s[4], mu[4];
    {
      const int l = lane & 31;
      const float4 p0 = xp[0][l], p1 = xp[1][l], p2 = xp[2][l], p3 = xp[3][l];
      const float4 d0 = xd[0][l], d1 = xd[1][l], d2 = xd[2][l], d3 = xd[3][l];
      s[0] = sum16(((p0.x + p1.x) + p2.x) + p3.x);
      s[1] = sum16(((p0.y + p1.y) + p2.y) + p3.y);
      s[2] = sum16(((p0.z + p1.z) + p2.z) + p3.z);
      s[3] = sum16(((p0.w + p1.w) + p2.w) + p3.w);
      mu[0] = sum16(((d0.x + d1.x) + d2.x) + d3.x) / s[0];
      mu[1] = sum16(((d0.y + d1.y) + d2.y) + d3.y) / s[1];
      mu[2] = sum16(((d0.z + d1.z) + d2.z) + d3.z) / s[2];
      mu[3] = sum16(((d0.w + d1.w) + d2.w) + d3.w) / s[3];
    }
    if (lane < 32)
      xg[wave][lane] = make_float4(p[0] * gfun(mu[0] - d[0]), p[1] * gfun(mu[1] - d[1]),
                                   p[2] * gfun(mu[2] - d[2]), p[3] * gfun(mu[3] - d[3]));
    __syncthreads();
    if (wave == 0 && lane < 32) {
      const float4 g0 = xg[0][lane], g1 = xg[1][lane], g2 = xg[2][lane], g3 = xg[3][lane];
      const float At[4] = {sum16(((g0.x + g1.x) + g2.x) + g3.x), sum16(((g0.y + g1.y) + g2.y) + g3.y),
                           sum16(((g0.z + g1.z) + g2.z) + g3.z), sum16(((g0.w + g1.w) + g2.w) + g3.w)};
      if (i == 0)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = blk * 8 + 4 * kg + r;
          if (row < a.rows) {
            float* q = a.part + ((size_t)row * a.ntiles + tile) * 4;
            q[0] = m[r];
            q[1] = s[r];
            q[2] = mu[r];
            q[3] = At[r] / s[r];
          }
        }
    }
    __syncthreads();      // red and the exchange arrays are free for the next block
  };
#pragma unroll
  for (int b = 0; b < RB; ++b) epilogue(acc[b], rb * RB + b);
}

// Many rows (a rollout's deferred rewards): a blocked GEMM.  A workgroup of 4
// waves computes a 128 x NT block of logits -- 64 kl rows, full and compressed
// interleaved per 16 (rows 8 b .. 8 b + 7 full, then the same rows compressed)
// -- against NT = 2 TW vocabulary columns, over the hidden dimension in stages
// of 64 elements staged in LDS (row stride 144 bytes: the 16 rows one fragment
// read touches start 16 bytes apart in the banks).  The global loads of the
// next PF stages are in flight in registers while the current stage feeds the
// matrix cores.  Wave (wm, wn) owns rows 64 wm.. x columns TW wn.. (4 x TW/16
// MFMA 16x16x32 bf16 blocks).  Every logit sees the same MFMA sequence over the
// hidden dimension as in kl_tile_kernel (same k split, same order), and the
// epilogue forms the same per (row, 64-column tile) statistics in the same
// reduction order, for kl_merge_kernel: the KL of a row is bit-identical
// whichever kernel and row count served it.  Workgroup g runs on
// XCD g mod 8; the row blocks of one vocabulary block are consecutive on one
// XCD, so its lm-head slab comes from HBM once and then from that XCD's L2.
// Used from 65 to 128 rows with TW = 64 and two stages in flight; from 129
// rows on kl_mm_kernel below serves the call.
constexpr int KG_M = 128;                       // logit rows per workgroup (64 kl rows)
constexpr int KG_BK = 64;                       // hidden elements per stage
constexpr int KG_RS = KG_BK * 2 + 16;           // LDS row stride (bytes)
// Fewer rows take kl_tile_kernel, whose workgroups stream the lm head once
// for up to 64 rows: measured per call (hidden 4096, vocab 32768, packed lm
// head) 50-53 us up to 16 rows, 60-66 us for 17-32, 92-96 us for 33-64,
// against 107-113 us here for up to 64 rows.
constexpr int KG_MIN_ROWS = 65;

template <int TW>
constexpr int kg_lds() { return (KG_M + 2 * TW) * KG_RS; }

template <int TW, int PF, bool PK>
__global__ void __launch_bounds__(256, 2) kl_gemm_kernel(KLArgs a) {
  constexpr int NT = 2 * TW;            // vocabulary columns per workgroup
  constexpr int CB = TW / 16;           // 16-column MFMA blocks per wave
  constexpr int BJ = NT / 32;           // lm-head chunks per thread per stage
  extern __shared__ __attribute__((aligned(16))) char kls[];
  char* As = kls;
  char* Bs = kls + KG_M * KG_RS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nM = (a.rows + 63) / 64, nN = (a.vocab + NT - 1) / NT;
  const int slot = blockIdx.x >> 3;
  const int nt = (blockIdx.x & 7) + 8 * (slot / nM), mt = slot % nM;
  if (nt >= nN) return;                 // whole workgroup: no barrier is skipped
  // global -> LDS: thread t copies 16-byte chunk t % 8 of rows t / 8 + 32 j
  const int lr = tid >> 3, lc = tid & 7;
  const char* hsrc = (const char*)((lr & 15) < 8 ? a.h_full : a.h_comp);
  int arow[4], vrow[BJ];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = mt * 64 + 8 * ((lr >> 4) + 2 * j) + (lr & 7);     // kl row of logit row lr + 32 j
    arow[j] = r < a.rows ? r : a.rows - 1;                            // past the end: re-read, unused
  }
#pragma unroll
  for (int j = 0; j < BJ; ++j) {
    const int v = nt * NT + lr + 32 * j;
    vrow[j] = v < a.vocab ? v : a.vocab - 1;
  }
  static_assert(NT % 64 == 0, "whole lm-head tiles per workgroup");
  const int wlane = lr * a.w_row + 16 * lc;       // packed layout: this lane's bytes of a block
  uint4 ra[PF][4], rb[PF][BJ];
  auto gload = [&](int k0, uint4 (&xa)[4], uint4 (&xb)[BJ]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) xa[j] = ldg16(hsrc + ((size_t)arow[j] * a.hidden + k0 + 8 * lc) * 2);
#pragma unroll
    for (int j = 0; j < BJ; ++j)
      if constexpr (PK) {
        // packed: chunk j is row lr + 32 (j mod 2) of tile nt NT / 64 + j / 2 (a tile
        // past the vocabulary re-reads the last one; its columns are dropped)
        int t = nt * (NT / 64) + j / 2;
        t = t < a.ntiles ? t : a.ntiles - 1;
        xb[j] = ldg16((const char*)a.w + ((size_t)t * (a.hidden / KG_BK) + k0 / KG_BK) * a.w_stage +
                      (size_t)(32 * (j & 1)) * a.w_row + wlane);
      } else {
        xb[j] = ldg16((const char*)a.w + ((size_t)vrow[j] * a.hidden + k0 + 8 * lc) * 2);
      }
  };
  auto sstore = [&](const uint4 (&xa)[4], const uint4 (&xb)[BJ]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4*>(As + (lr + 32 * j) * KG_RS + 16 * lc) = xa[j];
#pragma unroll
    for (int j = 0; j < BJ; ++j) *reinterpret_cast<uint4*>(Bs + (lr + 32 * j) * KG_RS + 16 * lc) = xb[j];
  };
  const int wm = wave >> 1, wn = wave & 1;
  const int i = lane & 15, kg = lane >> 4;
  f32x4_t acc[4][CB];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int c = 0; c < CB; ++c) acc[b][c] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
  auto compute = [&]() {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      // lane (i, kg) holds elements 32 t + 8 kg .. + 8 of its row in both operands
      uint4 af[4];
#pragma unroll
      for (int b = 0; b < 4; ++b)
        af[b] = *reinterpret_cast<const uint4*>(As + (64 * wm + 16 * b + i) * KG_RS + 16 * (kg + 4 * t));
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        const uint4 bf =
            *reinterpret_cast<const uint4*>(Bs + (TW * wn + 16 * c + i) * KG_RS + 16 * (kg + 4 * t));
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af[b]),
                                                              __builtin_bit_cast(bf16x8_t, bf),
                                                              acc[b][c], 0, 0, 0);
      }
    }
  };
  // every load is unconditional: past the last stage a load re-reads the last one
  const int last = a.hidden - KG_BK;
  {
    static_assert(PF == 2, "two stages in flight");
    // (the stage count hidden / 64 is even: hidden is a multiple of 128)
    gload(0, ra[0], rb[0]);
    gload(KG_BK, ra[1], rb[1]);
    for (int k0 = 0; k0 < a.hidden; k0 += 2 * KG_BK) {
      __syncthreads();
      sstore(ra[0], rb[0]);
      __syncthreads();
      gload(k0 + 2 * KG_BK <= last ? k0 + 2 * KG_BK : last, ra[0], rb[0]);
      compute();
      __syncthreads();
      sstore(ra[1], rb[1]);
      __syncthreads();
      gload(k0 + 3 * KG_BK <= last ? k0 + 3 * KG_BK : last, ra[1], rb[1]);
      compute();
    }
  }
  // acc[b][c][r] = logit of row 16 b + 4 kg + r (of the wave's 64), column 16 c + i:
  // lanes kg = 0, 1 the full rows 4 kg + r of block b, lanes kg = 2, 3 the same
  // rows compressed.  Lanes 0..31 form the statistics of kl row 8 b + 4 kg + r
  // over each 64-column tile g (blocks c = 4 g .. 4 g + 3), in the per-step
  // kernel's reduction order (the four 16-column blocks' terms added lane by
  // lane in column order, then the 16 lanes), so a row's statistics, and its KL, do not depend on how
  // many rows share the call.  One call per row block b, so that every index
  // into the accumulators is a constant.
  auto epilogue = [&](const f32x4_t (&ab)[CB], int b) {
#pragma unroll
    for (int g = 0; g < TW / 64; ++g) {
      float lf[4][4], dl[4][4];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = ab[4 * g + c][r];
          lf[c][r] = x;
          dl[c][r] = x - __shfl_xor(x, 32);     // delta = full - compressed logit
        }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float m = fmaxf(fmaxf(lf[0][r], lf[1][r]), fmaxf(lf[2][r], lf[3][r]));
        m = max16(m);
        float p[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) p[c] = __expf(lf[c][r] - m);
        const float S = sum16(((p[0] + p[1]) + p[2]) + p[3]);
        const float T = sum16(((p[0] * dl[0][r] + p[1] * dl[1][r]) + p[2] * dl[2][r]) + p[3] * dl[3][r]);
        const float mu = T / S;
        float pg[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) pg[c] = p[c] * gfun(mu - dl[c][r]);
        const float A = sum16(((pg[0] + pg[1]) + pg[2]) + pg[3]);
        const int row = mt * 64 + 32 * wm + 8 * b + 4 * kg + r;
        const int tile = (nt * NT + TW * wn) / 64 + g;
        if (lane < 32 && i == 0 && row < a.rows && tile < a.ntiles)
          *reinterpret_cast<float4*>(a.part + ((size_t)row * a.ntiles + tile) * 4) =
              make_float4(m, S, mu, A / S);
      }
    }
  };
  epilogue(acc[0], 0);
  epilogue(acc[1], 1);
  epilogue(acc[2], 2);
  epilogue(acc[3], 3);
}

template <int TW, int PF, bool PK>
static void launch_kl_gemm(const KLArgs& a, hipStream_t s) {
  const int nM = (a.rows + 63) / 64, nN = (a.vocab + 2 * TW - 1) / (2 * TW);
  hipFuncSetAttribute((const void*)kl_gemm_kernel<TW, PF, PK>,
                      hipFuncAttributeMaxDynamicSharedMemorySize, kg_lds<TW>());
  hipLaunchKernelGGL((kl_gemm_kernel<TW, PF, PK>), dim3(8 * nM * ((nN + 7) / 8)), dim3(256),
                     kg_lds<TW>(), s, a);
}

// Many rows, the larger shape: a 256 x 256 block of logits per workgroup (128
// kl rows, full and compressed interleaved per 8 as above, against 256
// vocabulary columns), eight waves of 128 x 64 (32 MFMA 16x16x32 bf16
// accumulators each, two waves per SIMD).  The hidden dimension goes in
// windows of 64 elements, so every row is read 128 bytes (one cache line) at a
// time.  A window is two stages of 32 KB, its 256 hidden-state rows and its
// 256 lm-head rows, loaded straight into LDS (global_load_lds_dwordx4: no
// registers, no LDS stores) through a ring of five stage buffers (160 KB):
// while a window's two stages feed the matrix cores, the next three stages
// are in flight.  Each load instruction covers 8 rows x 128 bytes; a row's
// 16-byte chunk c sits at position c ^ (row mod 8) of its 128 LDS bytes (lane
// j of the instruction loads the chunk that lands at byte 16 j), so the MFMA
// operand reads (lane (i, kg): row i, chunk 4 t + kg) hit eight different
// bank groups per eight lanes.  Each logit sees the per-step kernel's MFMA
// sequence (32-element blocks of the hidden dimension in ascending order) and
// the epilogue keeps kl_gemm_kernel's arithmetic, so the statistics, and the
// KL, are bit-identical to the other kernels'.  The loads into LDS are issued
// from inline assembly, out of the compiler's sight, and their waits are
// explicit: they complete in issue order, so at window w each wave waits until
// only its loads of the stage after the window may be in flight, and then the
// workgroup meets at a barrier.  A stage buffer is refilled only after the
// barrier that follows every wave's last read of it (the MFMAs of the
// previous window have consumed their operands).
constexpr int KM_M = 256;                       // logit rows per workgroup (128 kl rows)
constexpr int KM_N = 256;                       // vocabulary columns per workgroup
constexpr int KM_BK = 64;                       // hidden elements per window
constexpr int KM_STG = 256 * KM_BK * 2;         // LDS bytes of one stage (one operand, one window)
constexpr int KM_SLOTS = 5;                     // stage buffers
constexpr int KM_WAVES = 8;
constexpr int KM_LPW = 256 / 8 / KM_WAVES;      // 8-row load instructions per wave and stage
// From here on this kernel: its 128-row blocks against the blocked GEMM's 64,
// measured 144 rows 142 us against 159 us, 128 rows 141 us against 133 us.
constexpr int KM_MIN_ROWS = 129;

__global__ void __launch_bounds__(64 * KM_WAVES) kl_mm_kernel(KLArgs a) {
  __shared__ __attribute__((aligned(1024))) char ring[KM_SLOTS * KM_STG];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nM = (a.rows + 127) / 128, nN = (a.vocab + KM_N - 1) / KM_N;
  const int slot = blockIdx.x >> 3;
  const int nt = (blockIdx.x & 7) + 8 * (slot / nM), mt = slot % nM;
  if (nt >= nN) return;                 // whole workgroup: no barrier is skipped
  const int i = lane & 15, kg = lane >> 4;
  // load instruction q of this wave: rows 8 (KM_LPW wave + q) + lane / 8 of
  // the stage's operand, source chunk (lane mod 8) ^ (lane / 8), LDS byte
  // 16 lane of the instruction's 1 KB
  const int lrow = lane >> 3, lchunk = (lane & 7) ^ lrow;
  const char* hsrc[KM_LPW];
  const char* wsrc[KM_LPW];
#pragma unroll
  for (int q = 0; q < KM_LPW; ++q) {
    const int R = 8 * (KM_LPW * wave + q) + lrow;     // row of the 256 in the tile
    int r = mt * 128 + 8 * (R >> 4) + (R & 7);        // kl row of logit row R
    r = r < a.rows ? r : a.rows - 1;                   // past the end: re-read, unused
    hsrc[q] = (const char*)((R & 15) < 8 ? a.h_full : a.h_comp) + ((size_t)r * a.hidden + 8 * lchunk) * 2;
    int v = nt * KM_N + R;
    v = v < a.vocab ? v : a.vocab - 1;
    wsrc[q] = (const char*)a.w + w_row_off(a, v) + 16 * lchunk;
  }
  const int NW = a.hidden / KM_BK;
  const uint32_t ring_lds = (uint32_t)(size_t)(lds_char_t*)ring;
  // stage t: window t / 2 (past the last window: the last one again), its
  // hidden-state rows for even t and its lm-head rows for odd t, into buffer t mod 5
  auto issue = [&](int t) {
    const int w = (t >> 1) < NW ? (t >> 1) : NW - 1;
    const uint32_t dst = ring_lds + (t % KM_SLOTS) * KM_STG + KM_LPW * wave * 1024;
    if (t & 1) {
#pragma unroll
      for (int q = 0; q < KM_LPW; ++q) load_to_lds16(wsrc[q] + (size_t)a.w_stage * w, dst + q * 1024);
    } else {
#pragma unroll
      for (int q = 0; q < KM_LPW; ++q) load_to_lds16(hsrc[q] + 2 * KM_BK * w, dst + q * 1024);
    }
  };
  const int wm = wave >> 2, wn = wave & 3;       // rows 128 wm .., columns 64 wn ..
  f32x4_t acc[8][4];
#pragma unroll
  for (int b = 0; b < 8; ++b)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[b][c] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
  // operand of lane (i, kg) for the 16-row block starting at row R0, k-step t
  auto frag = [&](const char* X, int R0, int t) {
    const int r = R0 + i;
    return *reinterpret_cast<const uint4*>(X + r * 128 + (((4 * t + kg) ^ (r & 7)) << 4));
  };
  // k-step 0's operands are read first, then k-step 1's lm-head operands;
  // k-step 1's hidden-state operands are read one block at a time as k-step 0
  // releases the registers of that block (blocks in row order)
  auto compute = [&](const char* A, const char* B) {
    uint4 af[8], bf0[4], bf1[4];
#pragma unroll
    for (int b = 0; b < 8; ++b) af[b] = frag(A, 128 * wm + 16 * b, 0);
#pragma unroll
    for (int c = 0; c < 4; ++c) bf0[c] = frag(B, 64 * wn + 16 * c, 0);
#pragma unroll
    for (int c = 0; c < 4; ++c) bf1[c] = frag(B, 64 * wn + 16 * c, 1);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af[b]),
                                                            __builtin_bit_cast(bf16x8_t, bf0[c]),
                                                            acc[b][c], 0, 0, 0);
      af[b] = frag(A, 128 * wm + 16 * b, 1);
    }
#pragma unroll
    for (int b = 0; b < 8; ++b)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af[b]),
                                                            __builtin_bit_cast(bf16x8_t, bf1[c]),
                                                            acc[b][c], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);
  };
  issue(0);
  issue(1);
  issue(2);
  for (int w = 0; w < NW; ++w) {
    // this wave's loads of window w have landed (those of stage 2 w + 2 may
    // still be in flight); after the barrier every wave's have
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(KM_LPW) : "memory");
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(2 * w + 3);
    issue(2 * w + 4);
    compute(ring + ((2 * w) % KM_SLOTS) * KM_STG, ring + ((2 * w + 1) % KM_SLOTS) * KM_STG);
  }
  asm volatile("s_waitcnt vmcnt(0)" : : : "memory");   // no load into LDS outlives the loop
  compiler_fence();
  // acc[b][c][r]: logit row 16 b + 4 kg + r of the wave's 128, column 16 c + i;
  // lanes kg = 0, 1 hold full rows, kg = 2, 3 the same rows compressed.  One
  // lane swap per pair of row blocks (b, b + 1) gives lanes 0..31 block b and
  // lanes 32..63 block b + 1, full logit in one register and compressed in the
  // other, so all 64 lanes form statistics (same arithmetic per row as above).
  auto epilogue2 = [&](const f32x4_t (&x0)[4], const f32x4_t (&x1)[4], int b) {
    float lf[4][4], dl[4][4];
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x0[c][r]),
                                                         __float_as_uint(x1[c][r]), false, false);
        const float full = __uint_as_float(sw[0]), comp = __uint_as_float(sw[1]);
        lf[c][r] = full;
        dl[c][r] = full - comp;                 // delta = full - compressed logit
      }
    const int bb = b + (kg >> 1);               // row block of this half-wave
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float m = fmaxf(fmaxf(lf[0][r], lf[1][r]), fmaxf(lf[2][r], lf[3][r]));
      m = max16(m);
      float p[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) p[c] = __expf(lf[c][r] - m);
      const float S = sum16(((p[0] + p[1]) + p[2]) + p[3]);
      const float T = sum16(((p[0] * dl[0][r] + p[1] * dl[1][r]) + p[2] * dl[2][r]) + p[3] * dl[3][r]);
      const float mu = T / S;
      float pg[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) pg[c] = p[c] * gfun(mu - dl[c][r]);
      const float A = sum16(((pg[0] + pg[1]) + pg[2]) + pg[3]);
      const int row = mt * 128 + 64 * wm + 8 * bb + 4 * (kg & 1) + r;
      const int tile = (nt * KM_N + 64 * wn) / 64;
      if (i == 0 && row < a.rows && tile < a.ntiles)
        *reinterpret_cast<float4*>(a.part + ((size_t)row * a.ntiles + tile) * 4) =
            make_float4(m, S, mu, A / S);
    }
  };
  epilogue2(acc[0], acc[1], 0);
  epilogue2(acc[2], acc[3], 2);
  epilogue2(acc[4], acc[5], 4);
  epilogue2(acc[6], acc[7], 6);
}

static void launch_kl_mm(const KLArgs& a, hipStream_t s) {
  const int nM = (a.rows + 127) / 128, nN = (a.vocab + KM_N - 1) / KM_N;
  hipLaunchKernelGGL(kl_mm_kernel, dim3(8 * nM * ((nN + 7) / 8)), dim3(64 * KM_WAVES), 0, s, a);
}

// One workgroup per row: merge the tile statistics (fixed reduction order).
__global__ void __launch_bounds__(256) kl_merge_kernel(KLArgs a) {
  __shared__ float red[256];
  __shared__ float bc[2];
  const int row = blockIdx.x, t = threadIdx.x;
  const float* P = a.part + (size_t)row * a.ntiles * 4;
  float M = NEG_BIG;
  for (int j = t; j < a.ntiles; j += 256) M = fmaxf(M, P[4 * j]);
  red[t] = M;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = fmaxf(red[t], red[t + w]);
    __syncthreads();
  }
  M = red[0];
  __syncthreads();
  float S = 0.0f, U = 0.0f;
  for (int j = t; j < a.ntiles; j += 256) {
    const float w = P[4 * j + 1] * __expf(P[4 * j] - M);
    S = S + w;
    U = U + w * P[4 * j + 2];
  }
  red[t] = S;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = red[t] + red[t + w];
    __syncthreads();
  }
  S = red[0];
  __syncthreads();
  red[t] = U;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = red[t] + red[t + w];
    __syncthreads();
  }
  if (t == 0) {
    bc[0] = S;
    bc[1] = red[0] / S;
  }
  __syncthreads();
  S = bc[0];
  const float mu = bc[1];
  float acc = 0.0f;
  for (int j = t; j < a.ntiles; j += 256) {
    const float w = P[4 * j + 1] * __expf(P[4 * j] - M) / S;
    const float x = mu - P[4 * j + 2];
    acc = acc + w * (gfun(x) + __expf(x) * P[4 * j + 3]);
  }
  __syncthreads();
  red[t] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = red[t] + red[t + w];
    __syncthreads();
  }
  if (t == 0) a.out[row] = log1pf(red[0]);
}

// The packed lm-head layout: the 64 x 64 block of tile t (vocabulary rows
// 64 t .. 64 t + 63) and stage k (hidden elements 64 k .. 64 k + 63) is one
// contiguous 8 KB run, its 64 rows of 128 bytes in order; a tile's blocks
// follow each other in k, and the tiles in t.  A workgroup of kl_tile_kernel
// then reads one contiguous slab (512 KB at hidden 4096) instead of 64 rows
// 2 hidden bytes apart.  One thread per 16-byte chunk of the output (stores
// coalesced; each load instruction reads whole 128-byte row pieces).
__global__ void __launch_bounds__(256) kl_pack_kernel(const uint4* __restrict__ w,
                                                      uint4* __restrict__ out, int hidden,
                                                      size_t n16) {
  const size_t S = (size_t)hidden / KL_BK, cpr = (size_t)hidden / 8;
  for (size_t d = (size_t)blockIdx.x * 256 + threadIdx.x; d < n16; d += (size_t)gridDim.x * 256) {
    const size_t c = d & 7, r = (d >> 3) & 63, blk = d >> 9;
    const size_t t = blk / S, k = blk - t * S;
    out[d] = w[(t * KL_TILE + r) * cpr + 8 * k + c];
  }
}

int launch_kl_pack(const void* w, void* packed, int hidden, int vocab, void* stream) {
  const size_t n16 = (size_t)vocab * (size_t)hidden / 8;
  const size_t want = (n16 + 255) / 256;
  const unsigned blocks = (unsigned)(want < 16384 ? want : 16384);
  hipLaunchKernelGGL(kl_pack_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     (const uint4*)w, (uint4*)packed, hidden, n16);
  return (int)hipGetLastError();
}

int kl_tile_cols() { return KL_TILE; }

int launch_kl(const KLArgs& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (a.rows >= KM_MIN_ROWS) {
    launch_kl_mm(a, s);
  } else if (a.rows >= KG_MIN_ROWS) {
    // (the packed layout's stages are 64 rows apart; the row-major weight keeps
    // the plain row addressing, which needs two registers fewer)
    if (a.w_stage != 128) launch_kl_gemm<64, 2, true>(a, s);
    else launch_kl_gemm<64, 2, false>(a, s);
  } else {
    // 8-row blocks per workgroup: one, two, four or eight (the lm head streams
    // once per row group)
    const int rb = a.rows <= 8 ? 1 : a.rows <= 16 ? 2 : a.rows <= 32 ? 4 : 8;
    const int nrb = (a.rows + 8 * rb - 1) / (8 * rb);
    const dim3 g1(8 * ((a.ntiles + 7) / 8) * nrb), blk(64 * KL_WAVES);
    if (rb == 1) hipLaunchKernelGGL(kl_tile_kernel<1>, g1, blk, 0, s, a);
    else if (rb == 2) hipLaunchKernelGGL(kl_tile_kernel<2>, g1, blk, 0, s, a);
    else if (rb == 4) hipLaunchKernelGGL(kl_tile_kernel<4>, g1, blk, 0, s, a);
    else hipLaunchKernelGGL(kl_tile_kernel<8>, g1, blk, 0, s, a);
  }
  hipLaunchKernelGGL(kl_merge_kernel, dim3(a.rows), dim3(256), 0, s, a);
  return (int)hipGetLastError();
}

}  // namespace dc

// Scratch of dc_kl_reward_static: the per-(row, tile) statistics (4 floats per
// pair) in a fixed device array instead of a caller workspace.  Each device
// holds its own copy at its own address.  Host code never passes the array's
// name to a kernel (on the host it is only a stand-in for the symbol): the
// device address is looked up once per device with that device current and
// kept, and the kernels receive it as their `part` argument.
static __device__ __align__(256) float scratch[(size_t)DC_KL_STATIC_MAX_PAIRS * 4];

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_addr[SCRATCH_MAX_DEVICES] = {};
}  // namespace

namespace dc {

int kl_static_scratch(float** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_MAX_DEVICES) return -1;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return -1;
    scratch_addr[dev] = p;
  }
  *out = static_cast<float*>(scratch_addr[dev]);
  return 0;
}

}  // namespace dc
