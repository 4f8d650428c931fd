// Causal grouped-query softmax attention over the full prefix, reading K/V from
// the paged cache (flash-style: K/V tiles staged in LDS, online softmax).
//
// Workgroup = one query head x 128 queries, 4 waves x 32 queries.  Each wave
// computes S^T = K Q^T (keys on MFMA rows, its 32 queries on columns), so a
// lane owns one query and 16 of the 32 keys of a block: the row max / sum of
// the online softmax are in-lane plus one exchange with lane^32.  The
// probabilities then feed O^T = V^T P^T directly from the S accumulators: the
// 8 consecutive accumulator registers of a key half-block are exactly the 8
// k-slots a lane supplies, provided the V^T operand uses the same key order
// (keys 8*ii + 4*(lane/32) + jj).  V is transposed into LDS ([hd][key]) once
// per tile; K is stored [key][hd] with XOR-swizzled 16-byte chunks.
#include <math.h>

#include "kernels.hpp"

namespace crf {
namespace {

constexpr int BQ = 128;  // queries per workgroup
constexpr int BKV = 64;  // keys per tile
constexpr int VT_LD = BKV + 4;

template <int HD>
CRF_DEV int kswz(int row, int chunk) {
  if (HD == 128) return row * HD + ((chunk ^ (row & 15)) << 3);
  return row * HD + ((chunk ^ ((row >> 1) & 7)) << 3);
}

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const bf16 *__restrict__ Q, PagedKV kv,
                                                           bf16 *__restrict__ O, int M, int nq, int nkv) {
  constexpr int CH = HD / 8;   // 16-byte chunks per K row
  constexpr int KS = HD / 16;  // MFMA k-steps for S
  constexpr int HB = HD / 32;  // 32-row hd blocks of O^T
  __shared__ __align__(16) bf16 ks[2][BKV * HD];
  __shared__ __align__(16) bf16 vt[2][HD * VT_LD];

  const int nqb = (M + BQ - 1) / BQ;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int head = t % nq;
  const int qb = nqb - 1 - t / nq;  // longest causal rows first
  const int g_kv = head / (nq / nkv);
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int g = lane / 32, l32 = lane % 32;
  const int q0 = qb * BQ;
  const int q0w = q0 + wave * 32;
  const int qi = q0w + l32;
  const int dq = nq * HD;

  // Q fragments (B operand): query qi, hd chunk 2s+g
  bf16x8 qf[KS];
  {
    const bf16 *qrow = Q + (int64_t)min(qi, M - 1) * dq + head * HD + 8 * g;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = as_bf16x8(ld16(qrow + 16 * s));
  }

  const bf16 *kpool = (const bf16 *)kv.k;
  const bf16 *vpool = (const bf16 *)kv.v;
  // loaders: K = CH/4 chunks per thread, V = 2 keys x CH/16... chunks per thread
  constexpr int KCH = BKV * CH / 256;  // K chunks per thread
  constexpr int VCH = CH / 8;          // V hd-chunks per thread (each for 2 keys)
  u32x4 pk[KCH], pv[2 * VCH];
  auto gload = [&](int kt0) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int idx = tid + 256 * i;
      const int key = idx / CH, c = idx % CH;
      const int tok = kt0 + key;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (tok < M) {
        const int64_t r = paged_row(kv, tok, g_kv, HD);
        if (r >= 0) v = ld16(kpool + r + c * 8);
      }
      pk[i] = v;
    }
    const int kp = tid % 32;
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = tid / 32 + 8 * i;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int tok = kt0 + 2 * kp + e;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (tok < M) {
          const int64_t r = paged_row(kv, tok, g_kv, HD);
          if (r >= 0) v = ld16(vpool + r + c * 8);
        }
        pv[2 * i + e] = v;
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int idx = tid + 256 * i;
      const int key = idx / CH, c = idx % CH;
      st16(&ks[buf][kswz<HD>(key, c)], pk[i]);
    }
    const int kp = tid % 32;
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = tid / 32 + 8 * i;
      const bf16x8 v0 = as_bf16x8(pv[2 * i]), v1 = as_bf16x8(pv[2 * i + 1]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x2 pr = {v0[e], v1[e]};
        *reinterpret_cast<bf16x2 *>(&vt[buf][(c * 8 + e) * VT_LD + 2 * kp]) = pr;
      }
    }
  };

  f32x16 oacc[HB];
#pragma unroll
  for (int b = 0; b < HB; ++b)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[b][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c2 = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)

  const int last_key = min(q0 + BQ, M) - 1;
  const int ntiles = last_key / BKV + 1;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int it = 0; it < ntiles; ++it) {
    const int buf = it & 1;
    const int kt0 = it * BKV;
    if (it + 1 < ntiles) gload(kt0 + BKV);
    if (kt0 <= q0w + 31) {  // some key of this tile is visible to this wave
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[kb][v] = 0.f;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const bf16x8 kf = as_bf16x8(ld16(&ks[buf][kswz<HD>(kb * 32 + l32, 2 * s + g)]));
          sacc[kb] = mfma32(kf, qf[s], sacc[kb]);
        }
      }
      // causal mask (also hides keys >= M, which are always > qi for valid qi)
      if (kt0 + BKV - 1 > q0w) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = kt0 + kb * 32 + 8 * (v / 4) + 4 * g + (v % 4);
            if (key > qi) sacc[kb][v] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kb][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx * c2);
      const float alpha = exp2f(m_run - m_new);
      float psum = 0.f;
      bf16x8 pf[2][2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pv_ = exp2f(fmaf(sacc[kb][8 * hh + e], c2, -m_new));
            psum += pv_;
            pf[kb][hh][e] = f2bf(pv_);
          }
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int b = 0; b < HB; ++b) oacc[b] *= alpha;
      // O^T[hd, q] += V^T[hd, keys] P^T[keys, q]
#pragma unroll
      for (int b = 0; b < HB; ++b) {
        const bf16 *vrow = &vt[buf][(b * 32 + l32) * VT_LD];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int kbase = kb * 32 + 16 * hh + 4 * g;
            const u32x2 lo = ld8(vrow + kbase), hi = ld8(vrow + kbase + 8);
            const u32x4 vv = {lo[0], lo[1], hi[0], hi[1]};
            oacc[b] = mfma32(as_bf16x8(vv), pf[kb][hh], oacc[b]);
          }
      }
    }
    if (it + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  if (qi >= M) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  bf16 *orow = O + (int64_t)qi * dq + head * HD;
#pragma unroll
  for (int b = 0; b < HB; ++b)
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int e = b * 32 + 8 * ii + 4 * g;
      st8(orow + e, pack_bf16x4(oacc[b][ii * 4] * inv, oacc[b][ii * 4 + 1] * inv, oacc[b][ii * 4 + 2] * inv,
                                oacc[b][ii * 4 + 3] * inv));
    }
}

}  // namespace

hipError_t launch_attn_bf16(hipStream_t s, const bf16 *Q, const PagedKV &kv, bf16 *O, int M, int nq, int nkv,
                            int hd) {
  if (M <= 0) return hipSuccess;
  const int nqb = (M + BQ - 1) / BQ;
  dim3 grid(nqb * nq);
  if (hd == 128)
    hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(256), 0, s, Q, kv, O, M, nq, nkv);
  else if (hd == 64)
    hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(256), 0, s, Q, kv, O, M, nq, nkv);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace crf
