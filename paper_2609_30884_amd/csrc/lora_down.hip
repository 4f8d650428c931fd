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
  int spw;      // k-steps of 32 per workgroup along grid.y
  float *part;  // non-null: fp32 partial sums [grid.y][16][n_targets * rank_pad], unscaled
};

// Workgroup: TB blocks of 16 tokens, NW waves splitting K (wave w takes k-steps
// w, w+NW, ...).  Per k-step of 32: D[j, token] += A_t[j, k..k+32] .
// X[token, k..k+32] on the 16x16x32 MFMA, one MFMA per (16-row block of the
// concatenated factors, token block): the factors are read once per TB*16
// tokens.  The loads of UNROLL k-steps are issued before their MFMAs so enough
// bytes are in flight to keep HBM busy; the factors (a few hundred KB) stay in
// L2.
template <int NB, int UNROLL, int TB, int NW = 4>
__global__ __launch_bounds__(64 * NW) void lora_down_kernel(LdArgs a) {
  __shared__ f32x4 red[NW][NB * TB][64];
  // wave-uniform in a scalar register: the k-step guards below are then scalar
  // branches.  Derived per lane, they become EXEC-masked blocks, and an MFMA in
  // such a block still updates its accumulators when the mask is empty, adding
  // the previous batch's fragments once more.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64), lane = threadIdx.x % 64;
  const int m0 = blockIdx.x * 16 * TB;
  const int kq = (lane / 16) * 8;
  const bf16 *xrow[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) xrow[tb] = a.X + (int64_t)min(m0 + 16 * tb + lane % 16, a.M - 1) * a.ldx + kq;
  // per block: the target's factor as a buffer resource and this lane's row
  // offset; rows past the rank (and absent targets) lie out of range and read
  // as zero, so the loads need no branch
  __amdgpu_buffer_rsrc_t ares[NB];
  uint32_t aoff[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int t = (b * 16) / a.rank_pad;
    const int j = b * 16 - t * a.rank_pad + lane % 16;
    const bool on = a.A[t] != nullptr;
    ares[b] = make_rsrc(on ? (const void *)a.A[t] : (const void *)a.X, on ? (uint32_t)(a.rank[t] * a.K * 2) : 0u);
    aoff[b] = on && j < a.rank[t] ? (uint32_t)((j * a.K + kq) * 2) : CRF_OOB;
  }
  f32x4 acc[NB][TB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) acc[b][tb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int s0 = blockIdx.y * a.spw, s1 = min(a.K / 32, s0 + a.spw);
  for (int st = s0 + wave; st < s1; st += NW * UNROLL) {
    bf16x8 xb[UNROLL][TB], ab[UNROLL][NB];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      if (st + NW * u < s1) {  // wave-uniform
        const int k = (st + NW * u) * 32;
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) xb[u][tb] = as_bf16x8(ld16(xrow[tb] + k));
#pragma unroll
        for (int b = 0; b < NB; ++b)
          ab[u][b] = as_bf16x8(bld16(ares[b], aoff[b], (uint32_t)k * 2));
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the batch in flight before the first MFMA
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      if (st + NW * u < s1)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int tb = 0; tb < TB; ++tb) acc[b][tb] = mfma16(ab[u][b], xb[u][tb], acc[b][tb]);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) red[wave][b * TB + tb][lane] = acc[b][tb];
  __syncthreads();
  // wave w finishes token block w (TB <= 4)
  if (wave >= TB) return;
  const int m = m0 + 16 * wave + lane % 16;
  if (m >= a.M) return;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    f32x4 v = red[0][b * TB + wave][lane];
#pragma unroll
    for (int w = 1; w < NW; ++w) v += red[w][b * TB + wave][lane];
    if (a.part) {  // K split over workgroups: unscaled partial, summed by lora_down_sum_kernel
      const int ncols = a.n_targets * a.rank_pad;
      *reinterpret_cast<f32x4 *>(a.part + ((int64_t)blockIdx.y * 16 + m) * ncols + b * 16 + (lane / 16) * 4) = v;
      continue;
    }
    const int t = (b * 16) / a.rank_pad;
    const int jb = b * 16 - t * a.rank_pad + (lane / 16) * 4;  // first of 4 rows held by this lane
    const float sc = a.scale[t];
    st8(a.U + (int64_t)m * a.ldu + a.ucol[t] + jb, pack_bf16x4(v[0] * sc, v[1] * sc, v[2] * sc, v[3] * sc));
  }
}

// U[m, ucol_t + j] = scale_t * sum over the K split of the partials (M <= 16).
// 16 lanes per output, lane l adding the parts l, l + 16, ...; the 16 sums are
// then combined in a fixed order.
__global__ __launch_bounds__(256) void lora_down_sum_kernel(LdArgs a, int n_split) {
  const int ncols = a.n_targets * a.rank_pad;
  const int o = blockIdx.x * 16 + threadIdx.x / 16, l = threadIdx.x % 16;
  float v = 0.f;
  if (o < a.M * ncols) {
    const int m = o / ncols, c = o % ncols;
    for (int y = l; y < n_split; y += 16) v += a.part[((int64_t)y * 16 + m) * ncols + c];
  }
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) v += __shfl_xor(v, off, 16);
  if (l != 0 || o >= a.M * ncols) return;
  const int m = o / ncols, c = o % ncols;
  const int t = c / a.rank_pad, j = c % a.rank_pad;
  a.U[(int64_t)m * a.ldu + a.ucol[t] + j] = f2bf(v * a.scale[t]);
}

template <int NB>
void go(hipStream_t s, LdArgs a, float *ws, int64_t ws_floats, LoraSplit *split) {
  constexpr int UNROLL = NB <= 4 ? 8 : 2;
  const int nsteps = a.K / 32;
  // a few token rows: split K over workgroups (one batch of loads per wave)
  // and sum the partials in a second, tiny kernel
  const int spw = 4 * UNROLL, n_split = (nsteps + spw - 1) / spw;
  if (a.M <= 16 && n_split > 1 && ws && (int64_t)n_split * 16 * a.n_targets * a.rank_pad <= ws_floats) {
    a.spw = spw;
    a.part = ws;
    hipLaunchKernelGGL((lora_down_kernel<NB, UNROLL, 1>), dim3(1, n_split), dim3(256), 0, s, a);
    if (split && n_split <= 4) {  // the consumer sums the partials
      split->n_parts = n_split;
      split->cols = a.n_targets * a.rank_pad;
      return;
    }
    hipLaunchKernelGGL(lora_down_sum_kernel, dim3((a.M * a.n_targets * a.rank_pad + 15) / 16), dim3(256), 0, s, a,
                       n_split);
    return;
  }
  a.spw = nsteps;
  a.part = nullptr;
  if constexpr (NB <= 4) {
    if (a.M >= 8192) {
      // 64 tokens per workgroup (the factors are read once per 64 tokens) and
      // 8 waves splitting K, so that enough loads are in flight per CU
      hipLaunchKernelGGL((lora_down_kernel<NB, 4, 4, 8>), dim3((a.M + 63) / 64), dim3(512), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((lora_down_kernel<NB, UNROLL, 1>), dim3((a.M + 15) / 16), dim3(256), 0, s, a);
}

}  // namespace

hipError_t launch_lora_down_bf16(hipStream_t s, const bf16 *X, int64_t ldx, int M, int K, const LoraDownTarget *t,
                                 int n_targets, int rank_pad, bf16 *U, int ldu, float *ws, int64_t ws_floats,
                                 LoraSplit *split) {
  if (split) *split = LoraSplit{};
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
    case 1: go<1>(s, a, ws, ws_floats, split); break;
    case 2: go<2>(s, a, ws, ws_floats, split); break;
    case 3: go<3>(s, a, ws, ws_floats, split); break;
    case 4: go<4>(s, a, ws, ws_floats, split); break;
    case 6: go<6>(s, a, ws, ws_floats, split); break;
    case 8: go<8>(s, a, ws, ws_floats, split); break;
    case 9: go<9>(s, a, ws, ws_floats, split); break;
    case 12: go<12>(s, a, ws, ws_floats, split); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace crf
