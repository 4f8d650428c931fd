// Projections of a few token rows (M <= 16: the new tokens of a decoding step,
// or a very short window).  There the weights are streamed once and used M
// times, so the work is HBM-bound and the 256-row tiles of gemm_bf16 would sit
// mostly empty.  Instead, one workgroup owns 16 output features (32 for
// gate/up: the same 16 features of both) for all M tokens: its 4-16 waves split K,
// each issuing v_mfma_f32_16x16x32_bf16 with the weight rows as operand A and
// the token rows as operand B, several k-steps of loads in flight; the partial
// sums meet in LDS, wave 0 adds the adapter delta (U B^T, one more MFMA step
// per 32 of rank) and runs the epilogue.  A lane ends up with 4 consecutive
// features of one token, as in gemm_bf16:
//   EPI_RESID  resid[m, f] (+)= acc, optional bf16 copy;
//   EPI_SWIGLU act[m, f] = silu(gate) * up;
//   EPI_QKV    fp32 projections to `proj`; qkv_post_bf16 then adds the bias,
//              rotates Q and K and writes Q and the paged K/V.
#include "kernels.hpp"

namespace crf {
namespace {

constexpr int UNROLL = 8;  // k-steps of loads issued before their MFMAs

// Row `r` (tile space, as in gemm_bf16) of the weight matrix and its segment.
CRF_DEV const bf16 *skinny_weight_row(const GemmParams &p, GemmEpi epi, int r, int block, int &seg, int &local) {
  if (epi == EPI_SWIGLU) {  // block 0: gate rows, block 1: up rows of the same features
    seg = block;
    local = r;
    return p.w[block] + (int64_t)r * p.K;
  }
  if (epi == EPI_QKV) {
    seg = r < p.seg1 ? 0 : (r < p.seg2 ? 1 : 2);
    local = r - (seg == 0 ? 0 : (seg == 1 ? p.seg1 : p.seg2));
    return p.w[seg] + (int64_t)local * p.K;
  }
  seg = 0;
  local = r;
  return p.w[0] + (int64_t)r * p.K;
}

template <int EPI, int NB, int W>
__global__ __launch_bounds__(64 * W) void gemm_skinny_kernel(const GemmParams p) {
  __shared__ f32x4 red[W][NB][64];
  // wave-uniform in a scalar register, so that the k-step guards are scalar
  // branches: an MFMA in an EXEC-masked block still updates its accumulators
  // when the mask is empty
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64), lane = threadIdx.x % 64;
  const int f0 = blockIdx.x * 16;  // first output feature of the workgroup
  const int nrows = EPI == EPI_SWIGLU ? p.d_ffn : p.N;
  const int tok = min(lane % 16, p.M - 1);  // rows past M repeat the last token; never stored
  const int kq = (lane / 16) * 8;
  const bf16 *xrow = p.X + (int64_t)tok * p.ldx + kq;
  const bf16 *wrow[NB];
  int seg[NB], local[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    wrow[b] = skinny_weight_row(p, (GemmEpi)EPI, min(f0 + lane % 16, nrows - 1), b, seg[b], local[b]) + kq;

  f32x4 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  // wave w takes the k-step pairs w, w + W, ... (a pair covers 128 bytes of
  // each weight row: whole cache lines per wave); UNROLL steps are loaded
  // before their MFMAs (the scheduling barrier keeps every load of a batch in
  // flight at once)
  const int nsteps = p.K / 32;
  for (int sp = wave; 2 * sp < nsteps; sp += W * UNROLL / 2) {
    bf16x8 xb[UNROLL], wb[UNROLL][NB];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int st = 2 * (sp + W * (u / 2)) + u % 2;
      if (st < nsteps) {  // wave-uniform
        const int k = st * 32;
        xb[u] = as_bf16x8(ld16(xrow + k));
#pragma unroll
        for (int b = 0; b < NB; ++b) wb[u][b] = as_bf16x8(ld16(wrow[b] + k));
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      if (2 * (sp + W * (u / 2)) + u % 2 < nsteps)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[b] = mfma16(wb[u][b], xb[u], acc[b]);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) red[wave][b][lane] = acc[b];
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    acc[b] = red[0][b][lane];
#pragma unroll
    for (int w = 1; w < W; ++w) acc[b] += red[w][b][lane];
  }
  // adapter delta: acc += U[token, ucol + j] * lb[row, j], j < rank (zero-padded to 32)
  if (p.U) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bf16 *lb = p.lb[seg[b]];
      if (!lb) continue;
      for (int kk = 0; kk < p.kpad; kk += 32) {
        const int j = kk + kq;
        u32x4 av = {0u, 0u, 0u, 0u}, uv = {0u, 0u, 0u, 0u};
        if (j < p.rank) av = ld16(lb + (int64_t)local[b] * p.rank + j);
        if (j < p.rank && p.upart_n > 0) {  // sum the K-split partials in part order
          const float *pp = p.upart + (int64_t)tok * p.upart_cols + p.ucol[seg[b]] + j;
          f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
          for (int y = 0; y < p.upart_n; ++y) {
            lo += *reinterpret_cast<const f32x4 *>(pp + (int64_t)y * 16 * p.upart_cols);
            hi += *reinterpret_cast<const f32x4 *>(pp + (int64_t)y * 16 * p.upart_cols + 4);
          }
          lo *= p.uscale;
          hi *= p.uscale;
          const bf16x8 u8 = {f2bf(lo[0]), f2bf(lo[1]), f2bf(lo[2]), f2bf(lo[3]),
                             f2bf(hi[0]), f2bf(hi[1]), f2bf(hi[2]), f2bf(hi[3])};
          uv = as_u32x4(u8);
        } else if (j < p.rank) {  // (past the rank: unread)
          uv = ld16(p.U + (int64_t)tok * p.ldu + p.ucol[seg[b]] + j);
        }
        acc[b] = mfma16(as_bf16x8(av), as_bf16x8(uv), acc[b]);
      }
    }
  }
  const int m = lane % 16;
  const int f = f0 + 4 * (lane / 16);  // first of this lane's 4 features
  if (m >= p.M || f >= nrows) return;
  if (EPI == EPI_RESID) {
    float *rp = p.resid + (int64_t)m * p.ldr + f;
    f32x4 r = p.resid_overwrite ? f32x4{0.f, 0.f, 0.f, 0.f} : *reinterpret_cast<f32x4 *>(rp);
    r += acc[0];
    *reinterpret_cast<f32x4 *>(rp) = r;
    if (p.resid_out) st8(p.resid_out + (int64_t)m * p.ldr + f, pack_bf16x4(r[0], r[1], r[2], r[3]));
  } else if (EPI == EPI_SWIGLU) {
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float g = acc[0][i], u = acc[NB - 1][i];
      o[i] = g / (1.0f + __expf(-g)) * u;
    }
    st8(p.act + (int64_t)m * p.d_ffn + f, pack_bf16x4(o[0], o[1], o[2], o[3]));
  } else {
    *reinterpret_cast<f32x4 *>(p.proj + (int64_t)m * p.N + f) = acc[0];
  }
}

// Bias, rotation (token row m at position pos0 + m) and stores of the fp32
// projections [M, N] (segments [0, seg1) Q, [seg1, seg2) K, [seg2, N) V; each a
// whole number of heads).  One thread per (row, head, rotary pair).
__global__ void qkv_post_bf16_kernel(const GemmParams p, int hd) {
  const int half = hd / 2;
  const int heads = p.N / hd;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)p.M * heads * half) return;
  const int i = (int)(idx % half);
  const int h = (int)((idx / half) % heads);
  const int m = (int)(idx / ((int64_t)half * heads));
  const int r0 = h * hd;
  const int seg = r0 < p.seg1 ? 0 : (r0 < p.seg2 ? 1 : 2);
  const int hl = (r0 - (seg == 0 ? 0 : (seg == 1 ? p.seg1 : p.seg2))) / hd;
  const float *row = p.proj + (int64_t)m * p.N + r0;
  float x1 = row[i], x2 = row[i + half];
  if (p.bias[seg]) {
    x1 += bf2f(p.bias[seg][hl * hd + i]);
    x2 += bf2f(p.bias[seg][hl * hd + i + half]);
  }
  if (seg < 2) {
    const float2 c = p.rope_cs[(int64_t)(p.pos0 + m) * half + i];
    const float y1 = x1 * c.x - x2 * c.y, y2 = x2 * c.x + x1 * c.y;
    x1 = y1;
    x2 = y2;
  }
  bf16 *dst;
  if (seg == 0) {
    dst = p.q_out + (int64_t)m * p.dq + (int64_t)hl * hd;
    x1 *= p.q_scale;
    x2 *= p.q_scale;
  } else {
    const int64_t r = paged_row(p.kv, p.pos0 + m, hl, hd);
    if (r < 0) return;
    dst = (bf16 *)(seg == 1 ? p.kv.k : p.kv.v) + r;
  }
  dst[i] = f2bf(x1);
  dst[i + half] = f2bf(x2);
}

// Waves per workgroup (the K split inside one workgroup): enough waves in the
// whole grid to keep HBM busy when there are few 16-feature workgroups.
template <int EPI, int NB>
void launch_skinny(hipStream_t s, int n_wg, const GemmParams &p) {
  const int CUS = p.n_cu > 0 ? p.n_cu : 256;  // compute units of the device
  // about 16 resident waves per CU: one round of 16-wave workgroups up to one
  // per CU, of 8-wave ones up to two per CU, else 4 waves (2 were no faster)
  if (n_wg > 2 * CUS)
    hipLaunchKernelGGL((gemm_skinny_kernel<EPI, NB, 4>), dim3(n_wg), dim3(256), 0, s, p);
  else if (n_wg > CUS)
    hipLaunchKernelGGL((gemm_skinny_kernel<EPI, NB, 8>), dim3(n_wg), dim3(512), 0, s, p);
  else
    hipLaunchKernelGGL((gemm_skinny_kernel<EPI, NB, 16>), dim3(n_wg), dim3(1024), 0, s, p);
}

}  // namespace

hipError_t launch_gemm_skinny_bf16(hipStream_t s, GemmEpi epi, int hd, const GemmParams &p) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (p.M > 16 || p.K % 32 || (p.U && p.kpad % 16)) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_RESID:
      if (p.N % 4) return hipErrorInvalidValue;
      launch_skinny<EPI_RESID, 1>(s, (p.N + 15) / 16, p);
      break;
    case EPI_SWIGLU:
      if (p.d_ffn % 16) return hipErrorInvalidValue;
      launch_skinny<EPI_SWIGLU, 2>(s, p.d_ffn / 16, p);
      break;
    case EPI_QKV: {
      if (!p.proj || p.N % hd || p.seg1 % hd || p.seg2 % hd) return hipErrorInvalidValue;
      launch_skinny<EPI_QKV, 1>(s, (p.N + 15) / 16, p);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const int64_t n = (int64_t)p.M * (p.N / hd) * (hd / 2);
      hipLaunchKernelGGL(qkv_post_bf16_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, hd);
      break;
    }
  }
  return hipGetLastError();
}

}  // namespace crf
