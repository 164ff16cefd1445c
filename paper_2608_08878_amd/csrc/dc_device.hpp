// Device-side building blocks shared by the decode-step kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dc {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float LOG2E = 1.44269504088896340736f;
constexpr float NEG_BIG = -1.0e30f;   // "minus infinity" that keeps 0 * x finite

// Row layout: one lane owns 16 contiguous bytes of a key/value row.
template <int DTYPE, int D>
struct RowT {
  static constexpr int ELT = DTYPE == 0 ? 4 : 2;    // bytes per element
  static constexpr int EPL = 16 / ELT;              // elements per lane
  static constexpr int LPR = D / EPL;               // lanes per row: 8, 16 or 32
  static_assert(LPR == 8 || LPR == 16 || LPR == 32, "row layout");
};

__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (b >> 16) | 0x40u;  // NaN stays NaN
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// Partial dot product of the lane's 16-byte slices (fixed evaluation order).
template <int DTYPE>
__device__ __forceinline__ float dot_slice(const uint4& q, const uint4& k) {
  if constexpr (DTYPE == 1) {
    float acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.x),
                                                __builtin_bit_cast(bf16x2_t, k.x), 0.0f, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.y),
                                          __builtin_bit_cast(bf16x2_t, k.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.z),
                                          __builtin_bit_cast(bf16x2_t, k.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.w),
                                          __builtin_bit_cast(bf16x2_t, k.w), acc, false);
    return acc;
  } else {
    float acc = __uint_as_float(q.x) * __uint_as_float(k.x);
    acc = __builtin_fmaf(__uint_as_float(q.y), __uint_as_float(k.y), acc);
    acc = __builtin_fmaf(__uint_as_float(q.z), __uint_as_float(k.z), acc);
    acc = __builtin_fmaf(__uint_as_float(q.w), __uint_as_float(k.w), acc);
    return acc;
  }
}

// Unpack a lane slice to float.
template <int DTYPE>
__device__ __forceinline__ void unpack_slice(const uint4& v, float* f) {
  if constexpr (DTYPE == 1) {
    f[0] = bf16lo(v.x); f[1] = bf16hi(v.x); f[2] = bf16lo(v.y); f[3] = bf16hi(v.y);
    f[4] = bf16lo(v.z); f[5] = bf16hi(v.z); f[6] = bf16lo(v.w); f[7] = bf16hi(v.w);
  } else {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
}

// DPP lane exchanges inside a 16-lane row.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int DPP_XOR1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <- lane 7-i within 8
constexpr int DPP_MIRROR = 0x140;      // lane i <- lane 15-i within 16

// Sum over the LPR lanes of a row group; every lane receives the same bits
// (each step adds two values in either order, and + is commutative).
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
  x += dpp<DPP_XOR1>(x);
  x += dpp<DPP_XOR2>(x);
  x += dpp<DPP_HALF_MIRROR>(x);
  if constexpr (LPR >= 16) x += dpp<DPP_MIRROR>(x);
  if constexpr (LPR >= 32) x += __shfl_xor(x, 16);
  return x;
}

// One unit of attention weight, exp(s - m) / l, evaluated identically wherever
// it is needed (the retire step recomputes exactly what was added w steps ago).
__device__ __forceinline__ float attn_weight(float s, float m, float invl) {
  return __builtin_amdgcn_exp2f((s - m) * LOG2E) * invl;
}

// Feature contributions of one row for one step from its weights a_j:
//   cz = sum_j a_j,  cn = sum_j a_j H_j,
// summed in order within blocks of four heads, blocks added in order.
template <int G>
__device__ __forceinline__ void contrib_from_weights(const float* a, const float* H, float& cz,
                                                     float& cn) {
  cz = 0.0f;
  cn = 0.0f;
#pragma unroll
  for (int b = 0; b < G; b += 4) {
    float z = 0.0f, n = 0.0f;
#pragma unroll
    for (int j = b; j < (b + 4 < G ? b + 4 : G); ++j) {
      z = z + a[j];
      n = n + a[j] * H[j];
    }
    cz = cz + z;
    cn = cn + n;
  }
}

template <int G>
__device__ __forceinline__ void row_contrib(const float* s, const float* m, const float* invl,
                                            const float* H, float& cz, float& cn) {
  float a[G];
#pragma unroll
  for (int j = 0; j < G; ++j) a[j] = attn_weight(s[j], m[j], invl[j]);
  contrib_from_weights<G>(a, H, cz, cn);
}

// sigma_i: variance over the G heads of the weights a row received this step,
// (1/G) sum_j (a_j - mean)^2 (two passes: no cancellation; 0 for G = 1).
template <int G>
__device__ __forceinline__ float head_variance(const float* a) {
  float m = a[0];
#pragma unroll
  for (int j = 1; j < G; ++j) m = m + a[j];
  m = m * (1.0f / G);
  float v = 0.0f;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const float d = a[j] - m;
    v = __builtin_fmaf(d, d, v);
  }
  return v * (1.0f / G);
}

__device__ __forceinline__ uint4 ldg16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

}  // namespace dc
