// Causal grouped-query softmax attention over the full prefix, reading K/V from
// the paged cache (flash-style: K/V tiles staged in LDS, online softmax).
//
// Workgroup = one query head x 128 queries: 4 waves of 32 queries, two
// workgroups per CU (two waves per SIMD from independent workgroups, so one
// wave's softmax overlaps the other's MFMAs).  Each wave computes S^T = K Q^T
// (keys on MFMA rows, queries on columns), so a lane owns one query and 16 of
// the 32 keys of a block: the online-softmax max and sum are in-lane plus one
// exchange with lane^32.  The probabilities feed O^T = V^T P^T straight from
// the S accumulators: the 8 accumulator registers of a key half-block are the
// 8 k-slots a lane supplies, so the V^T operand takes keys in the same order
// (slots 0-3: keys 4*(lane/32) + 0..3, slots 4-7: the same plus 8).
//
// K and V tiles go from the pages straight into LDS (buffer loads with an LDS
// destination, no register staging), both in their natural [key][hd] layout
// with XOR-swizzled 16-byte chunks.  The V^T operand is read with the gfx950
// LDS transpose read: within each 16-lane group, lane 4r+c points at 4
// consecutive hd values of key row r, and lane j receives hd column j of the 4
// rows.  A two-stage ring lets the loads of tile i+1 run under the MFMAs of
// tile i, with one barrier per tile.
//
// The workgroup's page bases are staged in LDS once (validated there); a key
// past the prefix or on a rejected page gets an out-of-range buffer offset,
// which the hardware returns as zero.
//
// Online softmax without a per-block maximum: the query rows come scaled by
// log2(e)/sqrt(hd) (attn_query_scale, applied where Q is stored) and each S
// accumulator starts at -ref, the lane's current reference, so the MFMAs hand
// back scores in log2 units already shifted and the probabilities are plain
// exp2 of the accumulators.  The reference is the row maximum of the first
// key block and is raised only when a half-block's probabilities sum past
// 2^8, which bounds every probability by 2^8; only then is the block maximum
// formed and O rescaled.  The result is the softmax of the definition (the
// reference cancels between O and the row sum).
//
// Launch order: workgroup b runs on XCD b % 8.  When the KV-head count divides
// 8, each XCD serves one KV head and every R-th query block (R = 8 / n_kv),
// longest causal rows first, with the G query heads of that KV head adjacent:
// the work per XCD is balanced and the heads that share K/V tiles run side by
// side on one L2.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "kernels.hpp"

namespace crf {
namespace {

#ifndef CRF_ATTN_WAVES
#define CRF_ATTN_WAVES 4
#endif
constexpr int NW = CRF_ATTN_WAVES;  // waves per workgroup, 32 queries each
constexpr int BQ = 32 * NW;         // queries per workgroup
constexpr int NT = 64 * NW;         // threads per workgroup
constexpr int BKV = 64;   // keys per tile
constexpr float PSUM_MAX = 256.0f;  // bound on a half-block's probability sum (and each probability)
constexpr int PGCAP = 2048;  // page bases staged in LDS at a time
constexpr int SPLIT_WG = 1024;  // workgroups aimed at when a few query rows are split over the keys

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// 16-byte chunk slot of chunk c in K row r: conflict-free 16-byte fragment reads.
template <int HD>
CRF_DEV int kslot(int r, int c) {
  return c ^ (r & (HD / 8 - 1));
}
// Chunk slot in V row r: every transpose read (4 rows x 32 bytes per 16 lanes,
// 4 rows x 64 bytes per 32 lanes) lands on distinct banks.
template <int HD>
CRF_DEV int vslot(int r, int c) {
  if (HD == 128) return c ^ ((0xCA60 >> (4 * (r & 3))) & 15);
  return c ^ (2 * (r & 3));
}

CRF_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

CRF_DEV s16x4 ld_tr(const bf16 *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(const __attribute__((address_space(3))) void *)p);
}

// Byte offset of the first key of logical page p for this KV head, or CRF_OOB.
struct PageMap {
  const int32_t *bt;
  int n_pages;
  uint32_t page_bytes, head_bytes;
  int *err;
  CRF_DEV uint32_t base(int p) const {
    const int q = bt[p];
    if (q < 0 || q >= n_pages) {
      atomicOr(err, (int)CRF_DEVERR_BLOCK_TABLE);
      return CRF_OOB;
    }
    return (uint32_t)q * page_bytes + head_bytes;
  }
};

// Query head and query block of workgroup `bid` over nqb blocks of BQ rows;
// false for padding at the end of a per-XCD list (uniform per workgroup).
// Packed: one workgroup per KV head carries the group's query heads stacked on
// the rows of one tile.  xcd_r > 0: XCD x (= bid % 8) serves KV head x / xcd_r
// and every xcd_r-th query block from x % xcd_r, longest causal rows first,
// with the group's query heads adjacent.  Otherwise head-major, longest rows
// first.
__host__ __device__ inline bool attn_block(int bid, int nq, int nkv, int nqb, int xcd_r, int packed, int &head,
                                           int &qblk) {
  const int group = nq / nkv;
  if (packed) {
    head = bid * group;
    qblk = 0;
    return true;
  }
  if (xcd_r > 0) {
    const int x = bid % 8, j = bid / 8;
    const int qi = j / group;
    head = (x / xcd_r) * group + j % group;
    qblk = nqb - 1 - (qi * xcd_r + x % xcd_r);
    return qblk >= 0;
  }
  head = bid % nq;
  qblk = nqb - 1 - bid / nq;
  return true;
}

// Workgroups of a window launch (no key split); sets xcd_r for attn_block
// (0 when the KV-head count does not divide the XCD count).
inline int attn_window_grid(int nq, int nkv, int nqb, int &xcd_r) {
  if (nkv <= 8 && 8 % nkv == 0) {
    xcd_r = 8 / nkv;
    return 8 * (nq / nkv) * ((nqb + xcd_r - 1) / xcd_r);
  }
  xcd_r = 0;
  return nqb * nq;
}

// PS: page size when fixed at compile time (16), 0 = runtime kv.page_size.
template <int HD, int PS>
__global__ __launch_bounds__(NT, 8 / NW) void attn_bf16_kernel(const bf16 *__restrict__ Q, PagedKV kv,
                                                           bf16 *__restrict__ O, int Mq, int q_off, int nq,
                                                           int nkv, uint32_t pool_bytes, int xcd_r,
                                                           int split_tiles, int packed, float *__restrict__ part) {
  constexpr int CH = HD / 8;             // 16-byte chunks per row
  constexpr int KS = HD / 16;            // MFMA k-steps for S
  constexpr int HB = HD / 32;            // 32-row hd blocks of O^T
  constexpr int RPI = 64 / CH;           // rows per 64-lane load instruction
  constexpr int RPW = BKV / NW;          // key rows each wave loads per tile
  constexpr int IPW = RPW / RPI;         // load instructions per wave per tile (each of K and V)
  constexpr int TILE = BKV * HD;         // elements per K (or V) tile
  // one array per stage and operand, so the compiler sees that loads into one
  // stage never alias reads of the other
  __shared__ __align__(16) bf16 ks0[TILE], ks1[TILE], vs0[TILE], vs1[TILE];
  __shared__ uint32_t pgbase[PGCAP];

  // Query rows 0..Mq-1 sit at positions q_off..q_off+Mq-1 and attend to keys
  // 0..q_off+row: the cached prefix and the rows before them (q_off = 0 and
  // Mq = the prefix length for a window).
  const int M = q_off + Mq;  // keys
  const int nqb = (Mq + BQ - 1) / BQ;
  const int group = nq / nkv;
  int head, qblk;
  if (!attn_block(blockIdx.x, nq, nkv, nqb, xcd_r, packed, head, qblk)) return;
  const int g_kv = head / group;
  const int ps = PS > 0 ? PS : kv.page_size;
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int g = lane / 32, l32 = lane % 32;
  const int q0 = qblk * BQ;
  const int q0w = q0 + wave * 32;
  const int qi = q0w + l32;
  const int dq = nq * HD;
  // This lane's query: row qrow of head qhead.  Packed, tile row qi holds
  // (query head qi / Mq of the group, query row qi % Mq).
  const int n_rows = packed ? group * Mq : Mq;
  const int qrow = packed ? qi % Mq : qi;
  const int qhead = packed ? head + min(qi / Mq, group - 1) : head;
  // first and last position of the wave's queries
  const int pos_lo = packed ? q_off : q_off + q0w;
  const int pos_hi = packed ? q_off + Mq - 1 : q_off + q0w + 31;

  bf16x8 qf[KS];
  {
    const bf16 *qrow_p = Q + (int64_t)min(qrow, Mq - 1) * dq + qhead * HD + 8 * g;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = as_bf16x8(ld16(qrow_p + 16 * s));
  }

  const __amdgpu_buffer_rsrc_t kres = make_rsrc(kv.k, pool_bytes);
  const __amdgpu_buffer_rsrc_t vres = make_rsrc(kv.v, pool_bytes);
  const PageMap pm{kv.block_table, kv.n_pages, (uint32_t)(kv.page_stride * 2), (uint32_t)(g_kv * ps * HD * 2),
                   kv.err};

  const int last_key = min(q_off + q0 + BQ, M) - 1;
  const int ntiles = last_key / BKV + 1;
  // Split over keys (a few query rows over a long prefix): this workgroup takes
  // tiles [t_begin, t_end) and leaves an unnormalised partial for the merge.
  int t_begin = 0, t_end = ntiles;
  if (split_tiles > 0) {
    t_begin = blockIdx.y * split_tiles;
    t_end = min(ntiles, t_begin + split_tiles);
  }
  const int n_pages_needed = last_key / ps + 1;

  // pgbase[i] = base of logical page pg_first + i; refilled only between barriers.
  int pg_first = 0;
  auto fill_pages = [&](int first) {
    pg_first = first;
    for (int i = tid; i < min(PGCAP, n_pages_needed - first); i += NT) pgbase[i] = pm.base(first + i);
  };

  // This lane's row and chunk in each of the wave's load instructions.  A wave
  // loads RPW consecutive rows (keys) of the tile; the in-page part of each
  // lane's offset (row in the page, swizzled chunk) is fixed for the kernel
  // when the page size is a multiple of 16.
  const int lrow = lane / CH, lslot = lane % CH;
  uint32_t koff[IPW], voff[IPW];
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int row = RPI * i + lrow;    // row within the wave's rows
    const int trow = wave * RPW + row;  // row within the tile (the LDS swizzle's row)
    koff[i] = (uint32_t)(row * HD * 2 + kslot<HD>(trow, lslot) * 16);
    voff[i] = (uint32_t)(row * HD * 2 + vslot<HD>(trow, lslot) * 16);
  }
  auto dma = [&](int kt0, bf16 *kdst, bf16 *vdst) {
    const int wrow0 = kt0 + wave * RPW;  // first key of this wave's rows
    if (PS > 0 && PS % 16 == 0) {
      // the wave's rows share one page: one uniform base (CRF_OOB plus an
      // in-page offset stays out of range, pool sizes being below 2^31)
      const int pidx = min(max(wrow0 / PS - pg_first, 0), PGCAP - 1);
      const uint32_t b =
          (uint32_t)__builtin_amdgcn_readfirstlane((int)pgbase[pidx]) + (uint32_t)((wrow0 % PS) * HD * 2);
      if (wrow0 + RPW <= M) {  // uniform: all the wave's rows inside the prefix
#pragma unroll
        for (int i = 0; i < IPW; ++i) {
          const int ldsoff = (wave * RPW + RPI * i) * HD;  // wave-uniform first row of this instruction
          dma16(kres, (lds_char *)(kdst + ldsoff), b + koff[i], 0);
          dma16(vres, (lds_char *)(vdst + ldsoff), b + voff[i], 0);
        }
      } else {
#pragma unroll
        for (int i = 0; i < IPW; ++i) {
          const int ldsoff = (wave * RPW + RPI * i) * HD;
          const bool in = wrow0 + RPI * i + lrow < M;
          dma16(kres, (lds_char *)(kdst + ldsoff), in ? b + koff[i] : CRF_OOB, 0);
          dma16(vres, (lds_char *)(vdst + ldsoff), in ? b + voff[i] : CRF_OOB, 0);
        }
      }
    } else {
      uint32_t b[IPW];
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int tok = wrow0 + RPI * i + lrow;
        b[i] = pgbase[min(max(tok / ps - pg_first, 0), PGCAP - 1)];  // clamped: used only when tok < M
      }
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int row = wave * RPW + RPI * i + lrow;  // key within the tile
        const int tok = kt0 + row;
        const bool ok = tok < M && b[i] != CRF_OOB;
        const uint32_t rowoff = b[i] + (uint32_t)((tok % ps) * HD * 2);
        const int ldsoff = (wave * RPW + RPI * i) * HD;
        dma16(kres, (lds_char *)(kdst + ldsoff), ok ? rowoff + (uint32_t)(kslot<HD>(row, lslot) * 16) : CRF_OOB, 0);
        dma16(vres, (lds_char *)(vdst + ldsoff), ok ? rowoff + (uint32_t)(vslot<HD>(row, lslot) * 16) : CRF_OOB, 0);
      }
    }
  };

  f32x16 oacc[HB];
#pragma unroll
  for (int b = 0; b < HB; ++b)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[b][v] = 0.f;
  // Scores arrive in log2 units (the query rows are stored pre-multiplied by
  // log2(e)/sqrt(hd)) and relative to the lane's reference `ref`: the S
  // accumulators start at -ref (negm), so exp2 of an accumulator is the
  // probability up to the common factor 2^ref.  The reference is set to the
  // row maximum on the wave's first key block and afterwards only raised,
  // when the probabilities of a 32-key half-block sum past PSUM_MAX (which
  // bounds each of them); most half-blocks therefore need no maximum at all.
  float ref = 0.f, l_run = 0.f;
  f32x16 negm;
#pragma unroll
  for (int v = 0; v < 16; ++v) negm[v] = 0.f;

  // Transpose-read coordinates: 16-lane group gq covers hd 16*(gq&1) .. +15 of a
  // 32-row block and key rows 4*(gq>>1) + r; lane 4r + c reads hd chunk c*4.
  const int tr_r = (lane % 16) / 4, tr_c = lane % 4, tr_g = lane / 16;
  const int tr_key = 4 * (tr_g >> 1) + tr_r;            // + key half-block base (+8 for slots 4-7)
  const int tr_hd = 16 * (tr_g & 1) + 4 * tr_c;         // + 32*b

  // One tile: wait for its loads, publish them, start the next tile's loads
  // into the other stage, then compute.  FIRST: the range's first tile, where
  // the reference is set (a row that sees any key of the range sees that
  // tile's first key, which lies in its first half-block).
  auto tile = [&](int it, const bf16 *kt, const bf16 *vt, bf16 *kn, bf16 *vn, auto first_t) {
    constexpr bool FIRST = decltype(first_t)::value;
    const int kt0 = it * BKV;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (it + 1 < t_end) {
      const int next_last_page = (min(kt0 + 2 * BKV, M) - 1) / ps;
      if (next_last_page >= pg_first + PGCAP) {
        fill_pages((kt0 + BKV) / ps);
        __syncthreads();
      }
      dma(kt0 + BKV, kn, vn);
    }
    // every key of this tile is in this wave's future, or every row of the wave is padding
    if (kt0 > pos_hi || q0w >= n_rows) return;
    f32x16 sacc[2];
    // K fragments are read two k-steps ahead of the MFMAs that use them (the
    // scheduling barriers keep the compiler from regrouping them)
    bf16x8 kf[3][2];
    auto kread = [&](int s, bf16x8 (&f)[2]) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int r = kb * 32 + l32;
        f[kb] = as_bf16x8(ld16(kt + r * HD + kslot<HD>(r, 2 * s + g) * 8));
      }
    };
    kread(0, kf[0]);
    kread(1, kf[1]);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (s + 2 < KS) kread(s + 2, kf[(s + 2) % 3]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sacc[kb] = mfma32(kf[s % 3][kb], qf[s], s == 0 ? negm : sacc[kb]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // causal mask (also hides keys >= M, which are always > q_off + qrow for a valid row)
    if (kt0 + BKV - 1 > pos_lo) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kt0 + kb * 32 + 8 * (v / 4) + 4 * g + (v % 4);
          if (key > q_off + qrow) sacc[kb][v] = -INFINITY;
        }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float pr[16];
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        pr[v] = fast_exp2(sacc[kb][v]);
        psum += pr[v];
      }
      // (the negated test also catches an infinite sum)
      if ((FIRST && kb == 0) || __builtin_amdgcn_ballot_w64(!(psum <= PSUM_MAX))) {
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kb][v]);
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        float shift;
        if (FIRST && kb == 0) {
          // the reference jumps to the row maximum (a row that sees no key
          // here sees none of the range: it keeps l = 0)
          shift = mx > -INFINITY ? mx : 0.f;
        } else {
          shift = fmaxf(mx, 0.f);
          const float alpha = fast_exp2(-shift);
          l_run *= alpha;
#pragma unroll
          for (int b = 0; b < HB; ++b) oacc[b] *= alpha;
        }
        ref += shift;
#pragma unroll
        for (int v = 0; v < 16; ++v) negm[v] = -ref;
#pragma unroll
        for (int k2 = kb; k2 < 2; ++k2)
#pragma unroll
          for (int v = 0; v < 16; ++v) sacc[k2][v] -= shift;
        psum = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          pr[v] = fast_exp2(sacc[kb][v]);
          psum += pr[v];
        }
      }
      l_run += psum;
      bf16x8 pf[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[hh][e] = f2bf(pr[8 * hh + e]);
      // O^T[hd, q] += V^T[hd, keys] P^T[keys, q]
#pragma unroll
      for (int b = 0; b < HB; ++b) {
        const int hd = 32 * b + tr_hd;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int r0 = kb * 32 + 16 * hh + tr_key, r1 = r0 + 8;
          const s16x4 lo = ld_tr(vt + r0 * HD + vslot<HD>(r0, hd / 8) * 8 + hd % 8);
          const s16x4 hi = ld_tr(vt + r1 * HD + vslot<HD>(r1, hd / 8) * 8 + hd % 8);
          const s16x4 lohi[2] = {lo, hi};
          oacc[b] = mfma32(__builtin_bit_cast(bf16x8, lohi), pf[hh], oacc[b]);
        }
      }
    }
  };

  fill_pages(t_begin * BKV / ps);
  __syncthreads();
  dma(t_begin * BKV, ks0, vs0);
  tile(t_begin, ks0, vs0, ks1, vs1, std::true_type());
  for (int it = t_begin + 1; it < t_end; it += 2) {
    tile(it, ks1, vs1, ks0, vs0, std::false_type());
    if (it + 1 < t_end) tile(it + 1, ks0, vs0, ks1, vs1, std::false_type());
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (qi >= n_rows) return;
  if (split_tiles > 0) {  // partial: unnormalised O^T row, then the running max and sum
    float *prow = part + (((int64_t)blockIdx.y * nq + qhead) * Mq + qrow) * (HD + 4);
#pragma unroll
    for (int b = 0; b < HB; ++b)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii)
        *reinterpret_cast<f32x4 *>(prow + b * 32 + 8 * ii + 4 * g) =
            f32x4{oacc[b][ii * 4], oacc[b][ii * 4 + 1], oacc[b][ii * 4 + 2], oacc[b][ii * 4 + 3]};
    if (g == 0) {
      prow[HD] = l_tot > 0.f ? ref : -1e30f;  // a row that saw no key weighs 0 in the merge
      prow[HD + 1] = l_tot;
    }
    return;
  }
  const float inv = 1.0f / l_tot;
  bf16 *orow = O + (int64_t)qrow * dq + qhead * HD;
#pragma unroll
  for (int b = 0; b < HB; ++b)
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int e = b * 32 + 8 * ii + 4 * g;
      st8(orow + e, pack_bf16x4(oacc[b][ii * 4] * inv, oacc[b][ii * 4 + 1] * inv, oacc[b][ii * 4 + 2] * inv,
                                oacc[b][ii * 4 + 3] * inv));
    }
}

// Merge of the key splits of one (query row, head): O = sum_s 2^(m_s - m) O_s /
// sum_s 2^(m_s - m) l_s with m = max_s m_s (scores in log2 units).  Groups of
// HD / 4 threads take every NG-th split, 4 output elements per thread.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float *__restrict__ part, bf16 *__restrict__ O,
                                                         int Mq, int nq, int n_splits) {
  constexpr int TPG = HD / 4, NG = 256 / TPG;
  __shared__ float wmax[4];
  __shared__ f32x4 osum[NG][TPG];
  __shared__ float lsum[NG];
  const int qi = blockIdx.x / nq, head = blockIdx.x % nq;
  const int tid = threadIdx.x;
  const int64_t stride = (int64_t)nq * Mq * (HD + 4);
  const float *p0 = part + ((int64_t)head * Mq + qi) * (HD + 4);
  float m = -INFINITY;
  for (int sp = tid; sp < n_splits; sp += 256) m = fmaxf(m, p0[sp * stride + HD]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if (tid % 64 == 0) wmax[tid / 64] = m;
  __syncthreads();
  m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  const int gi = tid / TPG, e = 4 * (tid % TPG);
  f32x4 o = {0.f, 0.f, 0.f, 0.f};
  float l = 0.f;
#pragma unroll 4
  for (int sp = gi; sp < n_splits; sp += NG) {
    const float *ps = p0 + sp * stride;
    const float w = exp2f(ps[HD] - m);
    l += w * ps[HD + 1];
    o += w * *reinterpret_cast<const f32x4 *>(ps + e);
  }
  osum[gi][tid % TPG] = o;
  if (tid % TPG == 0) lsum[gi] = l;
  __syncthreads();
  if (tid >= TPG) return;
  f32x4 ot = osum[0][tid];
  float lt = lsum[0];
#pragma unroll
  for (int g2 = 1; g2 < NG; ++g2) {
    ot += osum[g2][tid];
    lt += lsum[g2];
  }
  const float inv = 1.0f / lt;
  st8(O + (int64_t)qi * nq * HD + head * HD + e, pack_bf16x4(ot[0] * inv, ot[1] * inv, ot[2] * inv, ot[3] * inv));
}

template <int HD>
void launch(hipStream_t s, const bf16 *Q, const PagedKV &kv, bf16 *O, int Mq, int q_off, int nq, int nkv,
            uint32_t pool_bytes, float *part, int64_t part_floats) {
  const int nqb = (Mq + BQ - 1) / BQ;
  int xcd_r = 0, grid = nqb * nq, n_splits = 1, split_tiles = 0, packed = 0;
  const int64_t keys = (int64_t)q_off + Mq;
  const int ntiles = (int)((keys + BKV - 1) / BKV);
  const int64_t max_splits = part ? part_floats / ((int64_t)nq * Mq * (HD + 4)) : 0;
  if (Mq <= 16 && ntiles >= 8 && max_splits >= 2) {
    // a few query rows over a long prefix: split the keys over workgroups;
    // when the group's heads fit one tile, one workgroup serves all of them
    // (the K/V tiles are read once per KV head)
    packed = (nq / nkv) * Mq <= BQ;
    const int units = packed ? nkv : nq;
    split_tiles = std::max<int>(1, (ntiles * units + SPLIT_WG - 1) / SPLIT_WG);
    split_tiles = std::max<int>(split_tiles, (int)((ntiles + max_splits - 1) / max_splits));
    n_splits = (ntiles + split_tiles - 1) / split_tiles;
    grid = units;
  } else {
    grid = attn_window_grid(nq, nkv, nqb, xcd_r);
  }
  const dim3 g3(grid, n_splits);
  if (kv.page_size == 16)
    hipLaunchKernelGGL((attn_bf16_kernel<HD, 16>), g3, dim3(NT), 0, s, Q, kv, O, Mq, q_off, nq, nkv, pool_bytes,
                       xcd_r, split_tiles, packed, part);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<HD, 0>), g3, dim3(NT), 0, s, Q, kv, O, Mq, q_off, nq, nkv, pool_bytes,
                       xcd_r, split_tiles, packed, part);
  if (split_tiles > 0)
    hipLaunchKernelGGL((attn_merge_kernel<HD>), dim3(Mq * nq), dim3(256), 0, s, part, O, Mq, nq, n_splits);
}

}  // namespace

hipError_t launch_attn_bf16(hipStream_t s, const bf16 *Q, const PagedKV &kv, bf16 *O, int Mq, int q_off, int nq,
                            int nkv, int hd, float *part, int64_t part_floats) {
  if (Mq <= 0) return hipSuccess;
  if (q_off < 0) return hipErrorInvalidValue;
  const int64_t bytes = (int64_t)kv.n_pages * kv.page_stride * 2;
  if (bytes >= (int64_t)CRF_OOB) return hipErrorInvalidValue;
  if (hd == 128)
    launch<128>(s, Q, kv, O, Mq, q_off, nq, nkv, (uint32_t)bytes, part, part_floats);
  else if (hd == 64)
    launch<64>(s, Q, kv, O, Mq, q_off, nq, nkv, (uint32_t)bytes, part, part_floats);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace crf
