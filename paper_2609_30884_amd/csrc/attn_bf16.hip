// Causal grouped-query softmax attention over the full prefix, reading K/V from
// the paged cache (flash-style: K/V tiles staged in LDS, online softmax).
//
// Workgroup = one query head x 128 queries: 4 waves of 32 queries, two
// workgroups per CU (two waves per SIMD, so one wave's softmax overlaps the
// other's MFMAs).  Each wave computes S^T = K Q^T (keys on MFMA rows, queries
// on columns), so a lane owns one query and 16 of the 32 keys of a block: the
// online-softmax max and sum are in-lane plus one exchange with lane^32.  The
// probabilities feed O^T = V^T P^T straight from the S accumulators: the 8
// consecutive accumulator registers of a key half-block are the 8 k-slots a
// lane supplies, provided the V^T operand uses the same key order (keys
// 8*ii + 4*(lane/32) + jj).  V is transposed into LDS ([hd][key]) once per
// tile; K is stored [key][hd] with XOR-swizzled 16-byte chunks.
//
// K/V come from the pages through buffer loads.  The workgroup's page bases
// are staged in LDS once (validated there) and read per tile from LDS, so no
// vector-memory wait ever sits between a tile's prefetch and its use; the page
// base goes into the scalar offset, and keys past the prefix or on a rejected
// page get an out-of-range offset, which the hardware returns as zero.  The running max is
// only moved (and O rescaled) when a score exceeds it by more than 2^8 in
// probability, so most tiles skip the rescale; probabilities stay below 2^8.
#include <math.h>

#include "kernels.hpp"

namespace crf {
namespace {

constexpr int BQ = 128;   // queries per workgroup
constexpr int BKV = 64;   // keys per tile
constexpr int VT_LD = BKV + 4;
constexpr float RESCALE_THRESHOLD = 8.0f;  // log2 units
constexpr int PGCAP = 2048;  // page bases staged in LDS at a time (32768 keys of 16-token pages)

template <int HD>
CRF_DEV int kswz(int row, int chunk) {
  if (HD == 128) return row * HD + ((chunk ^ (row & 15)) << 3);
  return row * HD + ((chunk ^ ((row >> 1) & 7)) << 3);
}

CRF_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Byte offset of the first key of page `p` for this KV head, or CRF_OOB.
struct PageMap {
  const int32_t *bt;
  int n_pages, page_size, M;
  uint32_t page_bytes, head_bytes;
  int *err;
  CRF_DEV uint32_t base(int tok) const {
    if (tok >= M) return CRF_OOB;
    const int p = bt[tok / page_size];
    if (p < 0 || p >= n_pages) {
      atomicOr(err, (int)CRF_DEVERR_BLOCK_TABLE);
      return CRF_OOB;
    }
    return (uint32_t)p * page_bytes + head_bytes;
  }
};

template <int HD, bool PAGE16>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const bf16 *__restrict__ Q, PagedKV kv,
                                                           bf16 *__restrict__ O, int M, int nq, int nkv,
                                                           uint32_t pool_bytes) {
  constexpr int CH = HD / 8;           // 16-byte chunks per K row
  constexpr int KS = HD / 16;          // MFMA k-steps for S
  constexpr int HB = HD / 32;          // 32-row hd blocks of O^T
  constexpr int KCH = BKV * CH / 256;  // K chunks per thread per tile (one key each)
  constexpr int VCH = CH / 8;          // V hd-chunks per thread (each for 2 keys)
  constexpr int KROWS = 256 / CH;      // keys covered by one K chunk round
  __shared__ __align__(16) bf16 ks[2][BKV * HD];
  __shared__ __align__(16) bf16 vt[2][HD * VT_LD];
  __shared__ uint32_t pgbase[PAGE16 ? PGCAP : 1];

  const int nqb = (M + BQ - 1) / BQ;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int head = t % nq;
  const int qblk = nqb - 1 - t / nq;  // longest causal rows first
  const int g_kv = head / (nq / nkv);
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int g = lane / 32, l32 = lane % 32;
  const int q0 = qblk * BQ;
  const int q0w = q0 + wave * 32;
  const int qi = q0w + l32;
  const int dq = nq * HD;

  bf16x8 qf[KS];
  {
    const bf16 *qrow = Q + (int64_t)min(qi, M - 1) * dq + head * HD + 8 * g;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = as_bf16x8(ld16(qrow + 16 * s));
  }

  const __amdgpu_buffer_rsrc_t kres = make_rsrc(kv.k, pool_bytes);
  const __amdgpu_buffer_rsrc_t vres = make_rsrc(kv.v, pool_bytes);
  const PageMap pm{kv.block_table, kv.n_pages, kv.page_size, M, (uint32_t)(kv.page_stride * 2),
                   (uint32_t)(g_kv * kv.page_size * HD * 2), kv.err};

  // per-thread key/chunk coordinates inside a tile
  const int kkey = tid / CH, kc = tid % CH;          // K: keys kkey + KROWS*i, chunk kc
  const int vkp = tid % 32, vc = tid / 32;           // V: keys 2vkp, 2vkp+1, chunks vc + 8i

  // Page bases (16-token pages) staged in LDS: pgbase[i] = base of page
  // pg_first + i.  A refill happens between barriers, never while read.
  int pg_first = 0;
  auto fill_pages = [&](int first, int n_needed) {
    pg_first = first;
    for (int i = tid; i < min(PGCAP, n_needed - first); i += 256) pgbase[i] = pm.base((first + i) * 16);
  };
  auto tile_pages = [&](int kt0, uint32_t (&pb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      pb[i] = PAGE16 ? (uint32_t)__builtin_amdgcn_readfirstlane((int)pgbase[kt0 / 16 + i - pg_first]) : 0u;
  };

  u32x4 pk[KCH], pv[2 * VCH];
  auto gload = [&](int kt0, const uint32_t (&pb)[4]) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int key = kkey + KROWS * i;
      const int tok = kt0 + key;
      uint32_t soff, voff;
      if (PAGE16) {
        // the page (key / 16) is a per-lane choice among the tile's 4 uniform bases
        const uint32_t b = pb[key / 16];
        soff = 0;
        voff = (tok < M && b != CRF_OOB) ? b + (uint32_t)(((key & 15) * HD + kc * 8) * 2) : CRF_OOB;
      } else {
        soff = 0;
        const uint32_t b = pm.base(tok);
        voff = b == CRF_OOB ? CRF_OOB : b + (uint32_t)(((tok % kv.page_size) * HD + kc * 8) * 2);
      }
      pk[i] = bld16(kres, voff, soff);
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int key = 2 * vkp + e;
      const int tok = kt0 + key;
      uint32_t base;
      if (PAGE16) {
        const uint32_t b = pb[key / 16];
        base = (tok < M && b != CRF_OOB) ? b + (uint32_t)((key & 15) * HD * 2) : CRF_OOB;
      } else {
        const uint32_t b = pm.base(tok);
        base = b == CRF_OOB ? CRF_OOB : b + (uint32_t)((tok % kv.page_size) * HD * 2);
      }
#pragma unroll
      for (int i = 0; i < VCH; ++i) pv[2 * i + e] = bld16(vres, base == CRF_OOB ? CRF_OOB : base + (vc + 8 * i) * 16, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) st16(&ks[buf][kswz<HD>(kkey + KROWS * i, kc)], pk[i]);
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = vc + 8 * i;
      const bf16x8 v0 = as_bf16x8(pv[2 * i]), v1 = as_bf16x8(pv[2 * i + 1]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x2 pr = {v0[e], v1[e]};
        *reinterpret_cast<bf16x2 *>(&vt[buf][(c * 8 + e) * VT_LD + 2 * vkp]) = pr;
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
  const int n_pages_needed = ntiles * (BKV / 16);
  if (PAGE16) {
    fill_pages(0, n_pages_needed);
    __syncthreads();
  }
  {
    uint32_t pb[4];
    tile_pages(0, pb);
    gload(0, pb);
  }
  lstore(0);
  __syncthreads();
  for (int it = 0; it < ntiles; ++it) {
    const int buf = it & 1;
    const int kt0 = it * BKV;
    if (it + 1 < ntiles) {
      if (PAGE16 && (kt0 + BKV) / 16 + 4 > pg_first + PGCAP) {
        // every wave is past the previous barrier, so nobody reads pgbase now
        fill_pages((kt0 + BKV) / 16, n_pages_needed);
        __syncthreads();
      }
      uint32_t pb[4];
      tile_pages(kt0 + BKV, pb);
      gload(kt0 + BKV, pb);
    }
    if (kt0 <= q0w + 31) {  // some key of this tile is visible to this wave
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[kb][v] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
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
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c2;
      // move the reference max only when a probability would exceed 2^8
      const bool grow = mx > m_run + RESCALE_THRESHOLD;
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float m_new = grow ? mx : m_run;
        const float alpha = fast_exp2(m_run - m_new);  // 0 on the first visible tile
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int b = 0; b < HB; ++b) oacc[b] *= alpha;
      }
      float psum = 0.f;
      bf16x8 pf[2][2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float p = fast_exp2(fmaf(sacc[kb][8 * hh + e], c2, -m_run));
            psum += p;
            pf[kb][hh][e] = f2bf(p);
          }
      l_run += psum;
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
            oacc[b] = mfma32(as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]}), pf[kb][hh], oacc[b]);
          }
      }
    }
    if (it + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (qi >= M) return;
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

template <int HD>
void launch(hipStream_t s, const bf16 *Q, const PagedKV &kv, bf16 *O, int M, int nq, int nkv, uint32_t pool_bytes) {
  const int nqb = (M + BQ - 1) / BQ;
  if (kv.page_size == 16)
    hipLaunchKernelGGL((attn_bf16_kernel<HD, true>), dim3(nqb * nq), dim3(256), 0, s, Q, kv, O, M, nq, nkv,
                       pool_bytes);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<HD, false>), dim3(nqb * nq), dim3(256), 0, s, Q, kv, O, M, nq, nkv,
                       pool_bytes);
}

}  // namespace

hipError_t launch_attn_bf16(hipStream_t s, const bf16 *Q, const PagedKV &kv, bf16 *O, int M, int nq, int nkv,
                            int hd) {
  if (M <= 0) return hipSuccess;
  const int64_t bytes = (int64_t)kv.n_pages * kv.page_stride * 2;
  if (bytes >= (int64_t)CRF_OOB) return hipErrorInvalidValue;
  if (hd == 128)
    launch<128>(s, Q, kv, O, M, nq, nkv, (uint32_t)bytes);
  else if (hd == 64)
    launch<64>(s, Q, kv, O, M, nq, nkv, (uint32_t)bytes);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace crf
