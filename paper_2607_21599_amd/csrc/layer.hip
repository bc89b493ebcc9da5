// Row-wise pieces of the decoder layer around the DAF attention, on the rows
// the layer recomputes (the important and question rows: Sec. 2 item 2, the
// QKV computation phase; Sec. 2 item 3, the compact fused state feeds the next
// layer): RMSNorm before the projections, the rotary position embedding of
// q and k at each row's original position, and the MLP gate SiLU(g) * u.
// All HBM-bound; bf16 in and out, fp32 arithmetic (the rotation angle in
// fp64, since positions reach 10^5).
#include "daf_internal.h"

namespace daf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRowThreads = 256;  // 4 waves, one row each

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// y = x / sqrt(mean(x^2) + eps) * w, one wave per row, 16-byte pieces.
__global__ __launch_bounds__(kRowThreads) void rmsnorm_kernel(int64_t rows, int width, const __bf16 *x,
                                                              const __bf16 *w, float eps, __bf16 *y) {
  const int64_t row = (int64_t)blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const int pieces = width / 8;
  const bf16x8 *xr = reinterpret_cast<const bf16x8 *>(x + row * width);
  float ss = 0.f;
  for (int j = lane; j < pieces; j += 64) {
    const bf16x8 v = xr[j];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float f = (float)v[e];
      ss = __builtin_fmaf(f, f, ss);
    }
  }
  const float inv = 1.0f / sqrtf(wave_sum(ss) / (float)width + eps);
  const bf16x8 *wr = reinterpret_cast<const bf16x8 *>(w);
  bf16x8 *yr = reinterpret_cast<bf16x8 *>(y + row * width);
  for (int j = lane; j < pieces; j += 64) {
    const bf16x8 v = xr[j], g = wr[j];
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (__bf16)((float)v[e] * inv * (float)g[e]);
    yr[j] = o;
  }
}

// In place: features (i, i + D/2) of every head rotate by pos * theta^(-2i/D).
// One thread per (row, i): the angle depends on neither the head nor the
// tensor, so each thread computes it once and rotates pair i of every head;
// the D/2 threads of a row are consecutive (128-byte runs per head).
__global__ __launch_bounds__(kRowThreads) void rope_kernel(int64_t rows, int heads, int d, int64_t row_stride,
                                                           __bf16 *x, const int32_t *pos, double log2_theta) {
  const int half = d / 2;
  const int64_t t = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  if (t >= rows * half) return;
  const int64_t row = t / half;
  const int i = (int)(t - row * half);
  const double inv = exp2(-(2.0 * i / d) * log2_theta);
  double sd, cd;
  sincos((double)pos[row] * inv, &sd, &cd);
  const float s = (float)sd, c = (float)cd;
  __bf16 *p = x + row * row_stride + i;
  for (int h = 0; h < heads; ++h, p += d) {
    const float a = (float)p[0], b = (float)p[half];
    p[0] = (__bf16)(a * c - b * s);
    p[half] = (__bf16)(b * c + a * s);
  }
}

// out[r][j] = SiLU(gu[r][j]) * gu[r][width + j] (gate then up in one row).
__global__ __launch_bounds__(kRowThreads) void silu_mul_kernel(int64_t rows, int width, const __bf16 *gu,
                                                               __bf16 *out) {
  const int pieces = width / 8;
  const int64_t t = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  if (t >= rows * pieces) return;
  const int64_t row = t / pieces;
  const int j = (int)(t - row * pieces);
  const bf16x8 g = reinterpret_cast<const bf16x8 *>(gu + row * 2 * width)[j];
  const bf16x8 u = reinterpret_cast<const bf16x8 *>(gu + row * 2 * width + width)[j];
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float gf = (float)g[e];
    o[e] = (__bf16)(gf / (1.0f + __expf(-gf)) * (float)u[e]);
  }
  reinterpret_cast<bf16x8 *>(out + row * width)[j] = o;
}

}  // namespace

hipError_t launch_rmsnorm(int64_t rows, int width, const void *x, const void *w, float eps, void *y,
                          hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int64_t blocks = (rows + kRowThreads / 64 - 1) / (kRowThreads / 64);
  rmsnorm_kernel<<<dim3((unsigned)blocks), dim3(kRowThreads), 0, st>>>(
      rows, width, static_cast<const __bf16 *>(x), static_cast<const __bf16 *>(w), eps, static_cast<__bf16 *>(y));
  return hipGetLastError();
}

hipError_t launch_rope(int64_t rows, int heads, int d, int64_t row_stride, void *x, const int32_t *pos,
                       double theta, hipStream_t st) {
  const int64_t n = rows * (d / 2);
  if (n <= 0 || heads <= 0) return hipSuccess;
  rope_kernel<<<dim3((unsigned)((n + kRowThreads - 1) / kRowThreads)), dim3(kRowThreads), 0, st>>>(
      rows, heads, d, row_stride, static_cast<__bf16 *>(x), pos, log2(theta));
  return hipGetLastError();
}

hipError_t launch_silu_mul(int64_t rows, int width, const void *gu, void *out, hipStream_t st) {
  const int64_t n = rows * (width / 8);
  if (n <= 0) return hipSuccess;
  silu_mul_kernel<<<dim3((unsigned)((n + kRowThreads - 1) / kRowThreads)), dim3(kRowThreads), 0, st>>>(
      rows, width, static_cast<const __bf16 *>(gu), static_cast<__bf16 *>(out));
  return hipGetLastError();
}

}  // namespace daf
