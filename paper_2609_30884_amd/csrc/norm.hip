// RMSNorm (normalised attention / MLP input) and the rotary angle table.
#include "kernels.hpp"

namespace crf {
namespace {

template <typename T>
CRF_DEV float ldf(const T *p, int64_t i);
template <>
CRF_DEV float ldf<float>(const float *p, int64_t i) { return p[i]; }
template <>
CRF_DEV float ldf<bf16>(const bf16 *p, int64_t i) { return bf2f(p[i]); }

template <typename T>
CRF_DEV void load8(const T *p, float (&v)[8]);
template <>
CRF_DEV void load8<float>(const float *p, float (&v)[8]) {
  f32x4 a = *reinterpret_cast<const f32x4 *>(p), b = *reinterpret_cast<const f32x4 *>(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[i] = a[i]; v[i + 4] = b[i]; }
}
template <>
CRF_DEV void load8<bf16>(const bf16 *p, float (&v)[8]) {
  bf16x8 a = as_bf16x8(ld16(p));
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = bf2f(a[i]);
}

template <typename T>
CRF_DEV void store8(T *p, const float (&v)[8]);
template <>
CRF_DEV void store8<float>(float *p, const float (&v)[8]) {
  *reinterpret_cast<f32x4 *>(p) = f32x4{v[0], v[1], v[2], v[3]};
  *reinterpret_cast<f32x4 *>(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
}
template <>
CRF_DEV void store8<bf16>(bf16 *p, const float (&v)[8]) {
  bf16x8 o;
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = f2bf(v[i]);
  st16(p, as_u32x4(o));
}

// One wave per row; 4 rows per workgroup.  d must be a multiple of 8.
template <typename TX, typename TG, typename TY>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const TX *__restrict__ x, const TG *__restrict__ g,
                                                      TY *__restrict__ y, float *__restrict__ copy_out, int M,
                                                      int d, float eps) {
  const int row = blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (row >= M) return;
  const TX *xr = x + (int64_t)row * d;
  float ss = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    float v[8];
    load8(xr + c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(v[i], v[i], ss);
    if (copy_out) store8(copy_out + (int64_t)row * d + c, v);
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = lane * 8; c < d; c += 512) {
    float v[8], gv[8];
    load8(xr + c, v);
    load8(g + c, gv);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = v[i] * r * gv[i];
    store8(y + (int64_t)row * d + c, v);
  }
}

// The same with the row held in registers (one pass over HBM): lane l holds
// elements [512 c + 8 l, 512 c + 8 l + 8) of chunk c < NCH, d <= 512 NCH.  All
// of a wave's loads are issued before the first use, so a row's bytes are in
// flight at once.
template <typename TX, typename TG, typename TY, int NCH>
__global__ __launch_bounds__(256) void rmsnorm_reg_kernel(const TX *__restrict__ x, const TG *__restrict__ g,
                                                          TY *__restrict__ y, float *__restrict__ copy_out, int M,
                                                          int d, float eps) {
  const int row = blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (row >= M) return;
  const TX *xr = x + (int64_t)row * d;
  float v[NCH][8];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int k = 512 * c + lane * 8;
    if (k < d) {
      load8(xr + k, v[c]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[c][i] = 0.f;
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(v[c][i], v[c][i], ss);
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int k = 512 * c + lane * 8;
    if (k >= d) continue;
    if (copy_out) store8(copy_out + (int64_t)row * d + k, v[c]);
    float gv[8];
    load8(g + k, gv);
#pragma unroll
    for (int i = 0; i < 8; ++i) gv[i] = v[c][i] * r * gv[i];
    store8(y + (int64_t)row * d + k, gv);
  }
}

__global__ void rope_table_kernel(float2 *cs, int T, int hd, double log_theta) {
  const int half = hd / 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)T * half) return;
  const int p = (int)(idx / half), i = (int)(idx % half);
  const double inv_freq = exp(-(2.0 * i / hd) * log_theta);
  const double phi = (double)p * inv_freq;
  cs[idx] = make_float2((float)cos(phi), (float)sin(phi));
}

template <typename TX, typename TG, typename TY>
hipError_t go(hipStream_t s, const void *x, const void *g, void *y, float *copy_out, int M, int d, float eps) {
  if (M <= 0) return hipSuccess;
  const dim3 grid((M + 3) / 4), block(256);
  const TX *xp = (const TX *)x;
  const TG *gp = (const TG *)g;
  TY *yp = (TY *)y;
  switch ((d + 511) / 512) {
#define CRF_NORM_CASE(n)                                                                                   \
  case n:                                                                                                  \
    hipLaunchKernelGGL((rmsnorm_reg_kernel<TX, TG, TY, n>), grid, block, 0, s, xp, gp, yp, copy_out, M, d, eps); \
    break;
    CRF_NORM_CASE(1) CRF_NORM_CASE(2) CRF_NORM_CASE(3) CRF_NORM_CASE(4) CRF_NORM_CASE(5) CRF_NORM_CASE(6)
    CRF_NORM_CASE(7) CRF_NORM_CASE(8) CRF_NORM_CASE(9) CRF_NORM_CASE(10) CRF_NORM_CASE(11) CRF_NORM_CASE(12)
    CRF_NORM_CASE(13) CRF_NORM_CASE(14) CRF_NORM_CASE(15) CRF_NORM_CASE(16)
#undef CRF_NORM_CASE
    default:  // wider rows: two passes over the row
      hipLaunchKernelGGL((rmsnorm_kernel<TX, TG, TY>), grid, block, 0, s, xp, gp, yp, copy_out, M, d, eps);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rmsnorm(hipStream_t s, const void *x, bool x_f32, const void *g, bool g_f32, void *y, bool y_f32,
                          float *copy_out, int M, int d, float eps) {
  if (x_f32 && g_f32 && y_f32) return go<float, float, float>(s, x, g, y, copy_out, M, d, eps);
  if (x_f32 && !g_f32 && !y_f32) return go<float, bf16, bf16>(s, x, g, y, copy_out, M, d, eps);
  if (!x_f32 && !g_f32 && !y_f32) return go<bf16, bf16, bf16>(s, x, g, y, copy_out, M, d, eps);
  if (!x_f32 && g_f32 && y_f32) return go<bf16, float, float>(s, x, g, y, copy_out, M, d, eps);
  return hipErrorInvalidValue;
}

hipError_t launch_rope_table(hipStream_t s, float2 *cs, int T, int hd, float theta) {
  const int64_t n = (int64_t)T * (hd / 2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, cs, T, hd,
                     log((double)theta));
  return hipGetLastError();
}

}  // namespace crf
