// Skinny LoRA down-projection U = scale * X A^T for up to three adapter targets
// that read the same input (q/k/v, gate/up, o or down).  The input is read
// once; the r x K factors stay in L2.  HBM-bound.
#include "kernels.hpp"

namespace crf {
namespace {

constexpr int MAXT = 3;
constexpr int MAXB = 12;  // 16-row blocks over all targets (3 targets x rank 64)
// block counts n_targets * rank_pad / 16 that occur: {1,2,3} targets x rank_pad {16,32,48,64}

struct LdArgs {
  const bf16 *X;
  int64_t ldx;
  int M, K;
  const bf16 *A[MAXT];
  int rank[MAXT];
  float scale[MAXT];
  int ucol[MAXT];
  int n_targets, rank_pad;
  bf16 *U;
  int ldu;
};

// Workgroup: 16 tokens, 4 waves splitting K (wave w takes k-steps w, w+4, ...).
// Per k-step of 32: D[j, token] += A_t[j, k..k+32] . X[token, k..k+32] on the
// 16x16x32 MFMA, one MFMA per 16-row block of the concatenated factors.  The
// loads of UNROLL k-steps are issued before their MFMAs so enough bytes are in
// flight to keep HBM busy; the factors (a few hundred KB) stay in L2.
template <int NB, int UNROLL>
__global__ __launch_bounds__(256) void lora_down_kernel(LdArgs a) {
  __shared__ f32x4 red[4][NB][64];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int m0 = blockIdx.x * 16;
  const int tok = min(m0 + lane % 16, a.M - 1);
  const int kq = (lane / 16) * 8;
  const bf16 *xrow = a.X + (int64_t)tok * a.ldx + kq;
  // per block: factor row pointer (or null -> zeros)
  const bf16 *arow[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int t = (b * 16) / a.rank_pad;
    const int j = b * 16 - t * a.rank_pad + lane % 16;
    arow[b] = (a.A[t] && j < a.rank[t]) ? a.A[t] + (int64_t)j * a.K + kq : nullptr;
  }
  f32x4 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nsteps = a.K / 32;
  int st = wave;
  for (; st + 4 * (UNROLL - 1) < nsteps; st += 4 * UNROLL) {
    bf16x8 xb[UNROLL], ab[UNROLL][NB];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int k = (st + 4 * u) * 32;
      xb[u] = as_bf16x8(ld16(xrow + k));
#pragma unroll
      for (int b = 0; b < NB; ++b) ab[u][b] = arow[b] ? as_bf16x8(ld16(arow[b] + k)) : as_bf16x8(u32x4{0u, 0u, 0u, 0u});
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[b] = mfma16(ab[u][b], xb[u], acc[b]);
  }
  for (; st < nsteps; st += 4) {
    const int k = st * 32;
    const bf16x8 xb = as_bf16x8(ld16(xrow + k));
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bf16x8 av = arow[b] ? as_bf16x8(ld16(arow[b] + k)) : as_bf16x8(u32x4{0u, 0u, 0u, 0u});
      acc[b] = mfma16(av, xb, acc[b]);
    }
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) red[wave][b][lane] = acc[b];
  __syncthreads();
  if (wave != 0) return;
  const int m = m0 + lane % 16;
  if (m >= a.M) return;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    f32x4 v = red[0][b][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) v += red[w][b][lane];
    const int t = (b * 16) / a.rank_pad;
    const int jb = b * 16 - t * a.rank_pad + (lane / 16) * 4;  // first of 4 rows held by this lane
    const float sc = a.scale[t];
    st8(a.U + (int64_t)m * a.ldu + a.ucol[t] + jb, pack_bf16x4(v[0] * sc, v[1] * sc, v[2] * sc, v[3] * sc));
  }
}

template <int NB>
void go(hipStream_t s, const LdArgs &a) {
  hipLaunchKernelGGL((lora_down_kernel<NB, (NB <= 4 ? 8 : 2)>), dim3((a.M + 15) / 16), dim3(256), 0, s, a);
}

}  // namespace

hipError_t launch_lora_down_bf16(hipStream_t s, const bf16 *X, int64_t ldx, int M, int K, const LoraDownTarget *t,
                                 int n_targets, int rank_pad, bf16 *U, int ldu) {
  if (M <= 0 || n_targets <= 0) return hipSuccess;
  if (n_targets > MAXT || n_targets * rank_pad > MAXB * 16 || rank_pad % 16 || K % 32) return hipErrorInvalidValue;
  LdArgs a{};
  a.X = X;
  a.ldx = ldx;
  a.M = M;
  a.K = K;
  for (int i = 0; i < n_targets; ++i) {
    a.A[i] = t[i].A;
    a.rank[i] = t[i].A ? t[i].rank : 0;
    a.scale[i] = t[i].scale;
    a.ucol[i] = t[i].ucol;
  }
  a.n_targets = n_targets;
  a.rank_pad = rank_pad;
  a.U = U;
  a.ldu = ldu;
  switch (n_targets * rank_pad / 16) {
    case 1: go<1>(s, a); break;
    case 2: go<2>(s, a); break;
    case 3: go<3>(s, a); break;
    case 4: go<4>(s, a); break;
    case 6: go<6>(s, a); break;
    case 8: go<8>(s, a); break;
    case 9: go<9>(s, a); break;
    case 12: go<12>(s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace crf
