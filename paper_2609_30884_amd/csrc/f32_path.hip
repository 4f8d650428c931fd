// fp32 storage path: plain LDS-tiled FMA GEMM plus elementwise rotation /
// paged write, SwiGLU and a one-query-per-workgroup causal attention.  Used
// when the model's storage type is fp32 (small decoders); every step is
// computed in fp32.
#include <math.h>

#include "kernels.hpp"

namespace crf {
namespace {

constexpr int TM = 64, TN = 64, TK = 16;

__global__ __launch_bounds__(256) void gemm_f32_kernel(int M, int N, int K, const float *__restrict__ A, int lda,
                                                       const float *__restrict__ B, int ldb, float *C, int ldc,
                                                       float alpha, float beta) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tm = blockIdx.y * TM, tn = blockIdx.x * TN;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += TK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + 256 * i;
      const int r = idx / TK, c = idx % TK;
      const int gk = k0 + c;
      As[c][r] = (tm + r < M && gk < K) ? A[(int64_t)(tm + r) * lda + gk] : 0.f;
      Bs[c][r] = (tn + r < N && gk < K) ? B[(int64_t)(tn + r) * ldb + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        b[i] = Bs[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = tm + ty * 4 + i, c = tn + tx * 4 + j;
      if (r < M && c < N) {
        float v = alpha * acc[i][j];
        float *cp = C + (int64_t)r * ldc + c;
        if (beta != 0.f) v = fmaf(beta, *cp, v);
        *cp = v;
      }
    }
}

// One thread per (token, head, pair index i < hd/2) over the nq + 2*nkv heads.
__global__ void qkv_post_f32_kernel(const float *__restrict__ P, const float *bq, const float *bk,
                                    const float *bv, float *__restrict__ Q, PagedKV kv,
                                    const float2 *__restrict__ cs, int M, int nq, int nkv, int hd) {
  const int half = hd / 2;
  const int heads = nq + 2 * nkv;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)M * heads * half) return;
  const int i = (int)(idx % half);
  const int h = (int)((idx / half) % heads);
  const int m = (int)(idx / ((int64_t)half * heads));
  const int width = (nq + 2 * nkv) * hd;
  const float *row = P + (int64_t)m * width + (int64_t)h * hd;
  float x1 = row[i], x2 = row[i + half];
  const float *bias = h < nq ? bq : (h < nq + nkv ? bk : bv);
  const int hl = h < nq ? h : (h < nq + nkv ? h - nq : h - nq - nkv);
  if (bias) {
    x1 += bias[hl * hd + i];
    x2 += bias[hl * hd + i + half];
  }
  if (h < nq + nkv) {  // rotate Q and K
    const float2 c = cs[(int64_t)m * half + i];
    const float y1 = x1 * c.x - x2 * c.y, y2 = x2 * c.x + x1 * c.y;
    x1 = y1;
    x2 = y2;
  }
  if (h < nq) {
    float *q = Q + (int64_t)m * nq * hd + (int64_t)h * hd;
    q[i] = x1;
    q[i + half] = x2;
    return;
  }
  const int64_t r = paged_row(kv, m, hl, hd);
  if (r < 0) return;
  float *dst = (h < nq + nkv ? (float *)kv.k : (float *)kv.v) + r;
  dst[i] = x1;
  dst[i + half] = x2;
}

__global__ void silu_mul_f32_kernel(const float *__restrict__ GU, float *__restrict__ act, int M, int f) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)M * f) return;
  const int m = (int)(idx / f), j = (int)(idx % f);
  const float g = GU[(int64_t)m * 2 * f + j], u = GU[(int64_t)m * 2 * f + f + j];
  act[idx] = g / (1.0f + expf(-g)) * u;
}

// One 64-lane workgroup per (query, head); keys in chunks of 64 with an online
// softmax.  Lane e owns output elements e, e+64, ...
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float *__restrict__ Q, PagedKV kv, float *__restrict__ O,
                                                      int nq, int nkv) {
  constexpr int R = (HD + 63) / 64;
  const int qi = blockIdx.x, h = blockIdx.y, g = h / (nq / nkv);
  const int lane = threadIdx.x;
  __shared__ float qs[HD];
  __shared__ float ps[64];
  __shared__ int64_t rows[64];
  for (int e = lane; e < HD; e += 64) qs[e] = Q[((int64_t)qi * nq + h) * HD + e];
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)HD);
  const float *K = (const float *)kv.k, *V = (const float *)kv.v;
  float m = -INFINITY, l = 0.f, o[R];
#pragma unroll
  for (int r = 0; r < R; ++r) o[r] = 0.f;
  for (int k0 = 0; k0 <= qi; k0 += 64) {
    const int key = k0 + lane;
    float s = -INFINITY;
    int64_t row = -1;
    if (key <= qi) {
      row = paged_row(kv, key, g, HD);
      float dot = 0.f;
      if (row >= 0)
        for (int e = 0; e < HD; ++e) dot = fmaf(qs[e], K[row + e], dot);
      s = dot * scale;
    }
    rows[lane] = row;
    const float mt = wave_max(s);
    const float mn = fmaxf(m, mt);
    const float alpha = expf(m - mn);
    const float p = key <= qi ? expf(s - mn) : 0.f;
    l = l * alpha + wave_sum(p);
    ps[lane] = p;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) o[r] *= alpha;
    const int nk = min(64, qi - k0 + 1);
    for (int j = 0; j < nk; ++j) {
      const int64_t rj = rows[j];
      if (rj < 0) continue;
      const float pj = ps[j];
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (lane + 64 * r < HD) o[r] = fmaf(pj, V[rj + lane + 64 * r], o[r]);
    }
    __syncthreads();
    m = mn;
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (lane + 64 * r < HD) O[((int64_t)qi * nq + h) * HD + lane + 64 * r] = o[r] / l;
}

}  // namespace

hipError_t launch_gemm_f32(hipStream_t s, int M, int N, int K, const float *A, int lda, const float *B, int ldb,
                           float *C, int ldc, float alpha, float beta) {
  if (M <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + TN - 1) / TN, (M + TM - 1) / TM);
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, M, N, K, A, lda, B, ldb, C, ldc, alpha, beta);
  return hipGetLastError();
}

hipError_t launch_qkv_post_f32(hipStream_t s, const float *P, const float *bq, const float *bk, const float *bv,
                               float *Q, const PagedKV &kv, const float2 *cs, int M, int nq, int nkv, int hd) {
  const int64_t n = (int64_t)M * (nq + 2 * nkv) * (hd / 2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(qkv_post_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, P, bq, bk, bv, Q, kv,
                     cs, M, nq, nkv, hd);
  return hipGetLastError();
}

hipError_t launch_silu_mul_f32(hipStream_t s, const float *GU, float *act, int M, int f) {
  const int64_t n = (int64_t)M * f;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(silu_mul_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, GU, act, M, f);
  return hipGetLastError();
}

hipError_t launch_attn_f32(hipStream_t s, const float *Q, const PagedKV &kv, float *O, int M, int nq, int nkv,
                           int hd) {
  if (M <= 0) return hipSuccess;
  dim3 grid(M, nq);
  if (hd == 64)
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, Q, kv, O, nq, nkv);
  else if (hd == 128)
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, Q, kv, O, nq, nkv);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace crf
