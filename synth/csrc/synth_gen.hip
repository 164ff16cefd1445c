// GPU twin of synth/philox.py and synth/workloads.py: fills device buffers with
// the very same seeded synthetic inputs, bit for bit, so that full-size
// workloads (tens of GB of key/value rows) need not be generated on the host.
//
// Every arithmetic step mirrors the host definition: Philox4x32-10 bits,
// (x + 0.5) * 2^-32 uniforms, Box-Muller with the fixed-polynomial ln/sin/cos,
// and exp for the log-normal key factor, all in binary64 using only correctly
// rounded operations in the same order.  Contraction into fused multiply-add is
// disabled for this file (the build passes -ffp-contract=off as well).
//
// This library holds no part of the decode-step method; it only produces inputs.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <thread>
#include <vector>

#pragma clang fp contract(off)

namespace {

constexpr double LOG_COEF[] = {0x1.0000000000000p+0, 0x1.5555555555555p-2, 0x1.999999999999ap-3,
    0x1.2492492492492p-3, 0x1.c71c71c71c71cp-4, 0x1.745d1745d1746p-4, 0x1.3b13b13b13b14p-4,
    0x1.1111111111111p-4, 0x1.e1e1e1e1e1e1ep-5, 0x1.af286bca1af28p-5, 0x1.8618618618618p-5,
    0x1.642c8590b2164p-5, 0x1.47ae147ae147bp-5, 0x1.2f684bda12f68p-5};
constexpr double SIN_COEF[] = {0x1.0000000000000p+0, -0x1.5555555555555p-3, 0x1.1111111111111p-7,
    -0x1.a01a01a01a01ap-13, 0x1.71de3a556c734p-19, -0x1.ae64567f544e4p-26, 0x1.6124613a86d09p-33,
    -0x1.ae7f3e733b81fp-41, 0x1.952c77030ad4ap-49, -0x1.2f49b46814157p-57, 0x1.71b8ef6dcf572p-66,
    -0x1.761b41316381ap-75, 0x1.3f3ccdd165fa9p-84};
constexpr double COS_COEF[] = {0x1.0000000000000p+0, -0x1.0000000000000p-1, 0x1.5555555555555p-5,
    -0x1.6c16c16c16c17p-10, 0x1.a01a01a01a01ap-16, -0x1.27e4fb7789f5cp-22, 0x1.1eed8eff8d898p-29,
    -0x1.93974a8c07c9dp-37, 0x1.ae7f3e733b81fp-45, -0x1.6827863b97d97p-53, 0x1.e542ba4020225p-62,
    -0x1.0ce396db7f853p-70, 0x1.f2cf01972f578p-80};
constexpr double EXP_COEF[] = {0x1.0000000000000p+0, 0x1.0000000000000p+0, 0x1.0000000000000p-1,
    0x1.5555555555555p-3, 0x1.5555555555555p-5, 0x1.1111111111111p-7, 0x1.6c16c16c16c17p-10,
    0x1.a01a01a01a01ap-13, 0x1.a01a01a01a01ap-16, 0x1.71de3a556c734p-19, 0x1.27e4fb7789f5cp-22,
    0x1.ae64567f544e4p-26, 0x1.1eed8eff8d898p-29, 0x1.6124613a86d09p-33, 0x1.93974a8c07c9dp-37,
    0x1.ae7f3e733b81fp-41, 0x1.ae7f3e733b81fp-45, 0x1.952c77030ad4ap-49};
constexpr int N_LOG = 14, N_SIN = 13, N_COS = 13, N_EXP = 18;
constexpr double LN2 = 0x1.62e42fefa39efp-1;
constexpr double INV_LN2 = 0x1.71547652b82fep+0;
constexpr double PI_2 = 0x1.921fb54442d18p+0;
constexpr double SQRT_HALF = 0x1.6a09e667f3bcdp-1;
constexpr double TWO_M32 = 0x1.0000000000000p-32;
constexpr uint64_t ROWSPAN = 1ull << 20;

struct U4 { uint32_t x0, x1, x2, x3; };

__host__ __device__ inline U4 philox(uint64_t call, uint32_t stream, uint32_t step, uint64_t seed) {
  uint32_t c0 = (uint32_t)call, c1 = (uint32_t)(call >> 32), c2 = stream, c3 = step;
  uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
  }
  return {c0, c1, c2, c3};
}

__host__ __device__ inline double to_unit(uint32_t x) { return ((double)x + 0.5) * TWO_M32; }

__host__ __device__ inline double horner(const double* c, int n, double x) {
  double p = c[n - 1];
  for (int i = n - 2; i >= 0; --i) { p = p * x; p = p + c[i]; }
  return p;
}

__host__ __device__ inline double det_log(double u) {
  int e;
  double m = frexp(u, &e);
  if (m < SQRT_HALF) { m = m * 2.0; e -= 1; }
  double z = (m - 1.0) / (m + 1.0);
  double z2 = z * z;
  double s = horner(LOG_COEF, N_LOG, z2);
  s = s * z;
  s = s * 2.0;
  return (double)e * LN2 + s;
}

__host__ __device__ inline void det_sincos(double u, double* cos_t, double* sin_t) {
  double v = u * 4.0;
  double q = floor(v);
  double f = v - q;
  double x = f * PI_2;
  double x2 = x * x;
  double s = horner(SIN_COEF, N_SIN, x2);
  s = s * x;
  double c = horner(COS_COEF, N_COS, x2);
  int qi = ((int)q) & 3;
  if (qi == 0) { *cos_t = c; *sin_t = s; }
  else if (qi == 1) { *cos_t = -s; *sin_t = c; }
  else if (qi == 2) { *cos_t = -c; *sin_t = -s; }
  else { *cos_t = s; *sin_t = -c; }
}

__host__ __device__ inline double det_exp(double x) {
  double k = rint(x * INV_LN2);
  double r = x - k * LN2;
  double p = horner(EXP_COEF, N_EXP, r);
  return ldexp(p, (int)k);
}

__host__ __device__ inline double uniform_at(uint64_t seed, uint32_t stream, uint32_t step, uint64_t idx) {
  U4 w = philox(idx >> 2, stream, step, seed);
  uint32_t lane = (uint32_t)(idx & 3);
  uint32_t x = lane == 0 ? w.x0 : lane == 1 ? w.x1 : lane == 2 ? w.x2 : w.x3;
  return to_unit(x);
}

__host__ __device__ inline double normal_at(uint64_t seed, uint32_t stream, uint32_t step, uint64_t idx) {
  U4 w = philox(idx >> 2, stream, step, seed);
  bool pair = (idx >> 1) & 1;
  double ua = to_unit(pair ? w.x2 : w.x0);
  double ub = to_unit(pair ? w.x3 : w.x1);
  double r = sqrt(det_log(ua) * -2.0);   // correctly rounded (IEEE) on host and device
  double c, s;
  det_sincos(ub, &c, &s);
  return (idx & 1) ? r * s : r * c;
}

__host__ __device__ inline uint32_t f32_bits(float f) {
  uint32_t b;
  __builtin_memcpy(&b, &f, 4);
  return b;
}

__host__ __device__ inline float bits_f32(uint32_t b) {
  float f;
  __builtin_memcpy(&f, &b, 4);
  return f;
}

__host__ __device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t b = f32_bits(f);
  b = (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
  return (uint16_t)b;
}

__host__ __device__ inline void store(void* out, int dtype, uint64_t i, double v) {
  float f = (float)v;                      // round to nearest even
  if (dtype == 0) ((float*)out)[i] = f;
  else ((uint16_t*)out)[i] = f32_to_bf16(f);
}

// key_structure: -1 value rows (no factor), 0 none, 1 heavy (x8 w.p. 0.01),
// 2 log-normal exp(0.5 n), 3 sink (positions < 64 scaled x4)
__host__ __device__ inline double row_factor(uint64_t seed, int ks, uint64_t rid, int64_t pos) {
  switch (ks) {
    case 1: return uniform_at(seed, 4, 0, rid) < 0.01 ? 8.0 : 1.0;
    case 2: return det_exp(normal_at(seed, 5, 0, rid) * 0.5);
    case 3: return pos < 64 ? 4.0 : 1.0;
    default: return 1.0;
  }
}

// One element of a key/value row block (see synth_fill_rows).
__host__ __device__ inline void row_elem(void* out, int dtype, uint64_t seed, int stream, int ks,
                                         int64_t unit0, int d, int64_t unit_stride_rows,
                                         int64_t pos0, int nrows, int64_t dst_row0, uint64_t t) {
  uint64_t e = t % d;
  uint64_t r = (t / d) % nrows;
  uint64_t u = t / ((uint64_t)d * nrows);
  int64_t pos = pos0 + (int64_t)r;
  uint64_t rid = (unit0 + u) * ROWSPAN + (uint64_t)pos;
  double z = normal_at(seed, (uint32_t)stream, 0, rid * d + e);
  double v = z * row_factor(seed, ks, rid, pos);
  store(out, dtype, (u * unit_stride_rows + dst_row0 + r) * d + e, v);
}

__host__ __device__ inline void noisy_elem(uint16_t* out, const uint16_t* base, uint64_t seed,
                                           int stream, int step, double eps, uint64_t i) {
  double b = (double)bits_f32((uint32_t)base[i] << 16);
  double z = normal_at(seed, (uint32_t)stream, (uint32_t)step, i);
  out[i] = f32_to_bf16((float)(b + z * eps));
}

__global__ void fill_rows_kernel(void* out, int dtype, uint64_t seed, int stream, int ks,
                                 int64_t unit0, int units, int d, int64_t unit_stride_rows,
                                 int64_t pos0, int nrows, int64_t dst_row0) {
  uint64_t total = (uint64_t)units * nrows * d;
  for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (uint64_t)gridDim.x * blockDim.x)
    row_elem(out, dtype, seed, stream, ks, unit0, d, unit_stride_rows, pos0, nrows, dst_row0, t);
}

__global__ void fill_normal_kernel(void* out, int dtype, uint64_t seed, int stream, int step,
                                   uint64_t n, double stdev) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    store(out, dtype, i, normal_at(seed, (uint32_t)stream, (uint32_t)step, i) * stdev);
}

// bf16 h_comp = round(h_full + eps * N(0,1)), h_full given as bf16 bits
__global__ void fill_noisy_kernel(uint16_t* out, const uint16_t* base, uint64_t seed, int stream,
                                  int step, uint64_t n, double eps) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    noisy_elem(out, base, seed, stream, step, eps, i);
}

template <typename F>
void host_parallel(uint64_t n, int threads, F f) {
  if (threads < 1) threads = 1;
  if ((uint64_t)threads > n / 4096 + 1) threads = (int)(n / 4096 + 1);
  std::vector<std::thread> pool;
  for (int w = 0; w < threads; ++w)
    pool.emplace_back([=]() {
      for (uint64_t i = (uint64_t)w; i < n; i += (uint64_t)threads) f(i);
    });
  for (auto& th : pool) th.join();
}

inline int grid_for(uint64_t n) {
  uint64_t g = (n + 255) / 256;
  return (int)(g > 65536 ? 65536 : (g == 0 ? 1 : g));
}

}  // namespace

extern "C" {

// Rows of units unit0 .. unit0+units-1 at positions pos0 .. pos0+nrows-1, written to
// out[(u - unit0) * unit_stride_rows + dst_row0 + r][0..d).  Returns a hipError_t.
int synth_fill_rows(void* out, int dtype, uint64_t seed, int stream, int key_structure,
                    int64_t unit0, int units, int d, int64_t unit_stride_rows, int64_t pos0,
                    int nrows, int64_t dst_row0, void* hip_stream) {
  uint64_t n = (uint64_t)units * nrows * d;
  hipLaunchKernelGGL(fill_rows_kernel, dim3(grid_for(n)), dim3(256), 0, (hipStream_t)hip_stream,
                     out, dtype, seed, stream, key_structure, unit0, units, d, unit_stride_rows,
                     pos0, nrows, dst_row0);
  return (int)hipGetLastError();
}

// out[i] = round(stdev * N(0,1)) for i < n, stream/step as in synth.philox.normal.
int synth_fill_normal(void* out, int dtype, uint64_t seed, int stream, int step, uint64_t n,
                      double stdev, void* hip_stream) {
  hipLaunchKernelGGL(fill_normal_kernel, dim3(grid_for(n)), dim3(256), 0, (hipStream_t)hip_stream,
                     out, dtype, seed, stream, step, n, stdev);
  return (int)hipGetLastError();
}

int synth_fill_noisy(void* out, const void* base, uint64_t seed, int stream, int step, uint64_t n,
                     double eps, void* hip_stream) {
  hipLaunchKernelGGL(fill_noisy_kernel, dim3(grid_for(n)), dim3(256), 0, (hipStream_t)hip_stream,
                     (uint16_t*)out, (const uint16_t*)base, seed, stream, step, n, eps);
  return (int)hipGetLastError();
}

// Host versions of the three fills (same arithmetic, host memory, `threads` workers).
void synth_cpu_fill_rows(void* out, int dtype, uint64_t seed, int stream, int key_structure,
                         int64_t unit0, int units, int d, int64_t unit_stride_rows, int64_t pos0,
                         int nrows, int64_t dst_row0, int threads) {
  uint64_t n = (uint64_t)units * nrows * d;
  host_parallel(n, threads, [=](uint64_t t) {
    row_elem(out, dtype, seed, stream, key_structure, unit0, d, unit_stride_rows, pos0, nrows,
             dst_row0, t);
  });
}

void synth_cpu_fill_normal(void* out, int dtype, uint64_t seed, int stream, int step, uint64_t n,
                           double stdev, int threads) {
  host_parallel(n, threads, [=](uint64_t i) {
    store(out, dtype, i, normal_at(seed, (uint32_t)stream, (uint32_t)step, i) * stdev);
  });
}

void synth_cpu_fill_noisy(void* out, const void* base, uint64_t seed, int stream, int step,
                          uint64_t n, double eps, int threads) {
  host_parallel(n, threads, [=](uint64_t i) {
    noisy_elem((uint16_t*)out, (const uint16_t*)base, seed, stream, step, eps, i);
  });
}

// Raw generator values for cross-checks: normals (kind 0) or uniforms (kind 1)
// in binary64 for the given element indices.
void synth_cpu_values(double* out, const uint64_t* idx, uint64_t n, uint64_t seed, int stream,
                      int step, int kind, int threads) {
  host_parallel(n, threads, [=](uint64_t i) {
    out[i] = kind == 0 ? normal_at(seed, (uint32_t)stream, (uint32_t)step, idx[i])
                       : uniform_at(seed, (uint32_t)stream, (uint32_t)step, idx[i]);
  });
}

}  // extern "C"
