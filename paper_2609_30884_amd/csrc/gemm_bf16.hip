// bf16 MFMA GEMM  D[feature, token] = W[feature, :] . X[token, :]  for the four
// projections of a decoder layer, with the low-rank adapter delta applied as a
// second, skinny contraction (K = padded rank) on the same accumulators and a
// fused epilogue:
//   EPI_QKV    bias + rotary rotation of Q and K, Q to a [M, dq] buffer, K and V
//              straight into the layer's pages of the paged cache;
//   EPI_RESID  fp32 residual update (attention output / down projection);
//   EPI_SWIGLU silu(gate) * up with gate and up rows interleaved per 64 features.
//
// Tiling for CDNA4: 256x256 output tile per 256-thread workgroup, 2x2 waves of
// 128x128, v_mfma_f32_32x32x16_bf16, K staged through LDS in 64-wide slices,
// double-buffered (2 x 64 KB), with the next slice prefetched into registers
// while the current one is consumed.  The weight operand takes the MFMA "A"
// role so each lane ends up holding 4 consecutive output features of one
// token, which makes every epilogue lane-local (a rotary pair (f, f+hd/2) and a
// gate/up pair live in the same lane).  16-byte LDS chunks are XOR-swizzled by
// (row/2) mod 8 so the fragment reads are bank-conflict free.
#include "kernels.hpp"

namespace crf {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;
constexpr int GROUP_M = 8;

CRF_DEV int swz(int row, int chunk) { return row * BK + ((chunk ^ ((row >> 1) & 7)) << 3); }

template <int EPI>
CRF_DEV const bf16 *weight_row(const GemmParams &p, int r) {
  if (EPI == EPI_RESID) return p.w[0] + (int64_t)r * p.K;
  if (EPI == EPI_QKV) {
    if (r < p.seg1) return p.w[0] + (int64_t)r * p.K;
    if (r < p.seg2) return p.w[1] + (int64_t)(r - p.seg1) * p.K;
    return p.w[2] + (int64_t)(r - p.seg2) * p.K;
  }
  // EPI_SWIGLU: 128 tile rows per 64 output features: [gate f..f+64, up f..f+64]
  const int f = (r >> 7) * 64 + (r & 63);
  return p.w[(r >> 6) & 1] + (int64_t)f * p.K;
}

// Segment and in-segment row of tile-space row r (used for LoRA factors and biases).
template <int EPI>
CRF_DEV int segment_of(const GemmParams &p, int r, int &local) {
  if (EPI == EPI_RESID) { local = r; return 0; }
  if (EPI == EPI_QKV) {
    if (r < p.seg1) { local = r; return 0; }
    if (r < p.seg2) { local = r - p.seg1; return 1; }
    local = r - p.seg2;
    return 2;
  }
  local = (r >> 7) * 64 + (r & 63);
  return (r >> 6) & 1;
}

template <int EPI, int HD>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(const GemmParams p) {
  extern __shared__ __align__(16) bf16 smem[];
  bf16 *const lds_x = smem;                  // [2][BM*BK]
  bf16 *const lds_w = smem + 2 * BM * BK;    // [2][BN*BK]

  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = (p.N + BN - 1) / BN;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int group = GROUP_M * tiles_n;
  const int first_m = (t / group) * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int tm = first_m + (t % group) % gm;
  const int tn = (t % group) / gm;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int wm = wave & 1, wn = wave >> 1;
  const int g = lane / 32, l32 = lane % 32;

  // ---- global -> register loader: 8 chunks of X and 8 of W per thread per slice.
  // Thread rows are lr + 32*i; W rows come in four 64-row groups (i = 2q, 2q+1),
  // each contiguous inside one weight segment.  Buffer loads: the per-lane byte
  // offsets are fixed, the slice offset k0 goes in the scalar operand, and X rows
  // past M fall outside the X resource and read as zero.
  const int lc = tid % 8, lr = tid / 8;  // chunk, first row
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(p.X, (uint32_t)((int64_t)p.M * p.ldx * 2));
  uint32_t xoff[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = m0 + lr + 32 * i;
    xoff[i] = r < p.M ? (uint32_t)(((int64_t)r * p.ldx + lc * 8) * 2) : CRF_OOB;
  }
  const bf16 *wsrc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = n0 + 64 * q + lr;
    wsrc[q] = (r < p.N ? weight_row<EPI>(p, r) : p.w[0]) + lc * 8;
  }
  const int64_t wstep = (int64_t)32 * p.K;
  u32x4 px[8], pw[8];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      px[i] = bld16(xres, xoff[i], (uint32_t)k0 * 2);
      pw[i] = ld16(wsrc[i / 2] + (i % 2) * wstep + k0);
    }
  };
  auto lstore = [&](int buf) {
    bf16 *dx = lds_x + buf * BM * BK;
    bf16 *dw = lds_w + buf * BN * BK;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = lr + 32 * i;
      st16(dx + swz(r, lc), px[i]);
      st16(dw + swz(r, lc), pw[i]);
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // ---- low-rank delta: acc += U[token, ucol_s + k] * lb_s[feature, k]
  if (p.U) {
    int seg[4], frow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = min(n0 + wn * 128 + 32 * i + l32, p.N - 1);
      seg[i] = segment_of<EPI>(p, r, frow[i]);
    }
    for (int kk = 0; kk < p.kpad; kk += 16) {
      const int k = kk + 8 * g;
      bf16x8 lbf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u32x4 v = {0u, 0u, 0u, 0u};
        const bf16 *lb = p.lb[seg[i]];
        if (lb && k < p.rank) v = ld16(lb + (int64_t)frow[i] * p.rank + k);
        lbf[i] = as_bf16x8(v);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = min(m0 + wm * 128 + 32 * j + l32, p.M - 1);
        const bf16 *urow = p.U + (int64_t)m * p.ldu + k;
        // segments used by this wave: blocks 0,1 and 2,3 may differ (EPI_SWIGLU)
        const bf16x8 u01 = as_bf16x8(ld16(urow + p.ucol[seg[0]]));
        const bf16x8 u23 = as_bf16x8(ld16(urow + p.ucol[seg[2]]));
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i][j] = mfma32(lbf[i], i < 2 ? u01 : u23, acc[i][j]);
      }
    }
  }

  const int nk = p.K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const bf16 *sx = lds_x + buf * BM * BK;
    const bf16 *sw = lds_w + buf * BN * BK;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rw = wn * 128 + 32 * i + l32;
        a[i] = as_bf16x8(ld16(sw + swz(rw, 2 * s + g)));
        const int rx = wm * 128 + 32 * i + l32;
        b[i] = as_bf16x8(ld16(sx + swz(rx, 2 * s + g)));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogues
  if (EPI == EPI_RESID) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + wm * 128 + 32 * j + l32;
      if (m >= p.M) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int n = n0 + wn * 128 + 32 * i + 8 * ii + 4 * g;
          if (n >= p.N) continue;
          float *rp = p.resid + (int64_t)m * p.ldr + n;
          f32x4 r = *reinterpret_cast<f32x4 *>(rp);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) r[jj] += acc[i][j][ii * 4 + jj];
          *reinterpret_cast<f32x4 *>(rp) = r;
          if (p.resid_out) st8(p.resid_out + (int64_t)m * p.ldr + n, pack_bf16x4(r[0], r[1], r[2], r[3]));
        }
    }
  } else if (EPI == EPI_SWIGLU) {
    const int fbase = (n0 + wn * 128) / 2;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + wm * 128 + 32 * j + l32;
      if (m >= p.M) continue;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int f = fbase + 32 * i + 8 * ii + 4 * g;
          if (f >= p.d_ffn) continue;
          float o[4];
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const float gt = acc[i][j][ii * 4 + jj], up = acc[i + 2][j][ii * 4 + jj];
            o[jj] = gt / (1.0f + __expf(-gt)) * up;
          }
          st8(p.act + (int64_t)m * p.d_ffn + f, pack_bf16x4(o[0], o[1], o[2], o[3]));
        }
    }
  } else {  // EPI_QKV
    constexpr int BPH = HD / 32;          // 32-row blocks per head
    constexpr int HPW = 128 / HD;         // heads per wave
    const int fb = n0 + wn * 128;         // first tile-space row of this wave (head aligned)
    int local;
    const int sg = segment_of<EPI>(p, fb, local);
    const int head0 = local / HD;
    const bf16 *bias = p.bias[sg];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + wm * 128 + 32 * j + l32;
      if (m >= p.M || fb >= p.N) continue;
      int64_t prow[HPW];
#pragma unroll
      for (int hh = 0; hh < HPW; ++hh) prow[hh] = sg ? paged_row(p.kv, m, head0 + hh, HD) : 0;
      const float2 *cs = p.rope_cs + (int64_t)m * (HD / 2);
#pragma unroll
      for (int hh = 0; hh < HPW; ++hh)
#pragma unroll
        for (int i = 0; i < BPH / 2; ++i)
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) {
            const int f = 32 * i + 8 * ii + 4 * g;  // in-head index of the first of 4 rows (< HD/2)
            const int b1 = hh * BPH + i, b2 = b1 + BPH / 2;
            float x1[4], x2[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              x1[jj] = acc[b1][j][ii * 4 + jj];
              x2[jj] = acc[b2][j][ii * 4 + jj];
            }
            if (bias) {
              const bf16 *bp = bias + (head0 + hh) * HD + f;
#pragma unroll
              for (int jj = 0; jj < 4; ++jj) {
                x1[jj] += bf2f(bp[jj]);
                x2[jj] += bf2f(bp[jj + HD / 2]);
              }
            }
            if (sg < 2) {  // rotate Q and K
#pragma unroll
              for (int jj = 0; jj < 4; ++jj) {
                const float2 c = cs[f + jj];
                const float y1 = x1[jj] * c.x - x2[jj] * c.y;
                const float y2 = x2[jj] * c.x + x1[jj] * c.y;
                x1[jj] = y1;
                x2[jj] = y2;
              }
            }
            bf16 *dst;
            if (sg == 0) {
              dst = p.q_out + (int64_t)m * p.dq + (head0 + hh) * HD;
            } else {
              if (prow[hh] < 0) continue;
              dst = (bf16 *)(sg == 1 ? p.kv.k : p.kv.v) + prow[hh];
            }
            st8(dst + f, pack_bf16x4(x1[0], x1[1], x1[2], x1[3]));
            st8(dst + f + HD / 2, pack_bf16x4(x2[0], x2[1], x2[2], x2[3]));
          }
    }
  }
}

template <int EPI, int HD>
hipError_t go(hipStream_t s, const GemmParams &p) {
  const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  const size_t lds = (size_t)2 * (BM + BN) * BK * sizeof(bf16);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)gemm_bf16_kernel<EPI, HD>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((gemm_bf16_kernel<EPI, HD>), dim3(tiles), dim3(NT), lds, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(hipStream_t s, GemmEpi epi, int hd, const GemmParams &p) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (p.K % BK) return hipErrorInvalidValue;
  if ((int64_t)p.M * p.ldx * 2 >= (int64_t)CRF_OOB) return hipErrorInvalidValue;  // X must fit one buffer resource
  switch (epi) {
    case EPI_RESID: return go<EPI_RESID, 128>(s, p);
    case EPI_SWIGLU: return go<EPI_SWIGLU, 128>(s, p);
    case EPI_QKV: return hd == 64 ? go<EPI_QKV, 64>(s, p) : go<EPI_QKV, 128>(s, p);
  }
  return hipErrorInvalidValue;
}

}  // namespace crf
