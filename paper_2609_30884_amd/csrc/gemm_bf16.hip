// bf16 MFMA GEMM  D[feature, token] = W[feature, :] . X[token, :]  for the four
// projections of a decoder layer, with the low-rank adapter delta applied as a
// second, skinny contraction (K = padded rank) on the same accumulators and a
// fused epilogue:
//   EPI_QKV    bias + rotary rotation of Q and K, Q to a [M, dq] buffer, K and V
//              straight into the layer's pages of the paged cache;
//   EPI_RESID  fp32 residual update (attention output / down projection);
//   EPI_SWIGLU silu(gate) * up with gate and up rows interleaved per 64 features,
//              optionally also the down projection's adapter down-projection
//              act . A_down^T, summed over the features a workgroup produces.
//
// Tiling for CDNA4: a 256x256 output tile per work item, 8 waves of 128x64 (two
// waves per SIMD, so one wave issues MFMAs while the other waits on LDS or
// memory); every wave owns 128 output features.  v_mfma_f32_32x32x16_bf16; K
// staged through LDS in 64-wide slices, double-buffered (2 x 64 KB).  Slices
// move global -> LDS by DMA (buffer_load ... lds): no staging registers and no
// LDS stores in the waves' instruction stream.  Rows past M (or past N) get an
// out-of-range offset and arrive as zeros.  The weight operand takes the MFMA
// "A" role so each lane ends up holding 4 consecutive output features of one
// token, which makes every epilogue lane-local (a rotary pair (f, f+hd/2) and a
// gate/up pair live in the same lane).  16-byte LDS chunks are XOR-swizzled by
// (row/2) mod 8 so the fragment reads are bank-conflict free.
//
// Persistent: one workgroup per CU walks its share of the work items, and the
// DMA cursor runs ahead across item boundaries, so the next item's first slices
// load during this item's epilogue.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "kernels.hpp"

namespace crf {
namespace {

#ifndef CRF_GEMM_BK
#define CRF_GEMM_BK 64
#endif
#ifndef CRF_GEMM_STAGES
#define CRF_GEMM_STAGES 2
#endif

constexpr int BM = 256, BN = 256;
constexpr int BK = CRF_GEMM_BK;          // k-width of one LDS slice
constexpr int STAGES = CRF_GEMM_STAGES;  // slices resident in LDS (STAGES * 32 KB per 32 of BK)
constexpr int GROUP_M = 8;
constexpr int LPR = BK / 8;              // 16-byte chunks (lanes) per row of a slice
constexpr int RPB = 64 / LPR;            // rows per 1 KB DMA block
constexpr int WAVES = 8;
constexpr int STAGE_BYTES = STAGES * (BM + BN) * BK * 2;
// fused down-projection adapter sums: [2 feature halves][256 tokens][16 ranks] fp32
constexpr int DN_RANK = 16;
constexpr int DN_BYTES = 2 * BM * DN_RANK * 4;
static_assert(BK == 32 || BK == 64, "slice width");
static_assert(STAGES >= 2 && STAGE_BYTES <= 160 * 1024, "LDS budget");
static_assert(BM * BK * 2 / 1024 >= 2 * WAVES, "each wave owns two x blocks of a stage");

// Chunk c of slice row r sits at position c ^ s(r), s(r) = (r / 2) % 8 for
// 128-byte rows and (r / 4) % 4 for 64-byte rows: the 16 rows one quarter of a
// ds_read_b128 touches (same chunk) hit 16 distinct 16-byte bank groups.
CRF_DEV int swz(int row, int chunk) {
  if (BK == 64) return row * BK + ((chunk ^ ((row >> 1) & 7)) << 3);
  return row * BK + ((chunk ^ ((row >> 2) & 3)) << 3);
}

template <int N>
CRF_DEV void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Segment and in-segment row of tile-space row r (used for weights, LoRA factors and biases).
template <int EPI>
CRF_DEV int segment_of(const GemmParams &p, int r, int &local) {
  if (EPI == EPI_RESID) { local = r; return 0; }
  if (EPI == EPI_QKV) {
    if (r < p.seg1) { local = r; return 0; }
    if (r < p.seg2) { local = r - p.seg1; return 1; }
    local = r - p.seg2;
    return 2;
  }
  // EPI_SWIGLU: 128 tile rows per 64 output features: [gate f..f+64, up f..f+64]
  local = (r >> 7) * 64 + (r & 63);
  return (r >> 6) & 1;
}

// ---- work items.  Shared by the kernel and the host (fused-sum slot count).
//
// A work item is a whole 256x256 tile (part -1) or K-part `part` of one of the
// split tiles, over K slices [kb, ke).  Whole tiles come first in item order
// and K-parts after them; each range is remapped on its own so that every XCD
// gets an equal, contiguous share of both (workgroup b runs on XCD b % 8).
struct WorkItem {
  int w, t, part, kb, ke, tm, tn;
};

__host__ __device__ inline int xcd_map(int i, int n) {
  return n % 8 ? i : (i % 8) * (n / 8) + i / 8;
}

// Tile t of the grouped order (GROUP_M token tiles share a weight panel).
__host__ __device__ inline void tile_coords(int t, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int group = GROUP_M * tiles_n;
  const int first_m = (t / group) * GROUP_M;
  const int gm = tiles_m - first_m < GROUP_M ? tiles_m - first_m : GROUP_M;
  tm = first_m + (t % group) % gm;
  tn = (t % group) / gm;
}

struct Sched {
  int tiles_m, tiles_n, nk, n_items, split_first, split_s, grid;
  bool stagger;  // odd workgroups take their last item (a K-part) first
};

__host__ __device__ inline int n_mine(const Sched &s, int b) {
  return b < s.n_items ? (s.n_items - 1 - b) / s.grid + 1 : 0;
}

// i-th work item of workgroup b
__host__ __device__ inline WorkItem work_item(const Sched &s, int b, int i) {
  const int mine = n_mine(s, b);
  int k = i;
  if (s.stagger && (b & 1) && mine > 1) k = i == 0 ? mine - 1 : i - 1;
  const int raw = b + k * s.grid;
  WorkItem it;
  it.part = -1;
  it.kb = 0;
  it.ke = s.nk;
  if (s.split_s > 1 && raw >= s.split_first) {
    const int n_parts = s.n_items - s.split_first;
    it.w = s.split_first + xcd_map(raw - s.split_first, n_parts);
    it.t = s.split_first + (it.w - s.split_first) / s.split_s;
    it.part = (it.w - s.split_first) % s.split_s;
    it.kb = it.part * s.nk / s.split_s;
    it.ke = (it.part + 1) * s.nk / s.split_s;
  } else {
    it.w = xcd_map(raw, s.split_s > 1 ? s.split_first : s.n_items);
    it.t = it.w;
  }
  tile_coords(it.t, s.tiles_m, s.tiles_n, it.tm, it.tn);
  return it;
}

// Runs (maximal sequences of consecutive items on one token tile) of workgroup b.
inline int n_runs(const Sched &s, int b) {
  int runs = 0, tm = -1;
  for (int i = 0; i < n_mine(s, b); ++i) {
    const WorkItem it = work_item(s, b, i);
    if (it.tm != tm) ++runs;
    tm = it.tm;
  }
  return runs;
}

template <int EPI, int HD>
__global__ __launch_bounds__(64 * WAVES, 1) void gemm_bf16_kernel(const GemmParams p, const Sched sc) {
  constexpr int WM_COUNT = 4;              // token groups
  constexpr int WTM = BM / WM_COUNT;       // tokens per wave
  constexpr int NJ = WTM / 32;             // 32-token blocks per wave
  constexpr int BLK = (BM / RPB) / WAVES;  // 1 KB DMA blocks per operand per wave per slice
  constexpr int DMA_PER_SLICE = 2 * BLK;
  extern __shared__ __align__(16) bf16 smem[];
  bf16 *const lds_x = smem;                       // [STAGES][BM*BK]
  bf16 *const lds_w = smem + STAGES * BM * BK;    // [STAGES][BN*BK]

  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);  // uniform: keeps DMA targets scalar
  const int wn = wave / WM_COUNT, wm = wave % WM_COUNT;
  const int g = lane / 32, l32 = lane % 32;
  const int mine = n_mine(sc, b);

  // ---- producer: the global -> LDS DMA cursor runs STAGES slices ahead of
  // the MFMAs and carries on into the workgroup's next item.  A slice of one
  // operand is 256 rows x BK k = BK/2 blocks of 1 KB; wave w moves blocks
  // WAVES*j + w.  Inside a block, lane L writes LDS bytes [16 L, 16 L + 16):
  // row RPB*block + L/LPR, swizzled position L%LPR, which holds the logical
  // k-chunk at that position of swz.
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(p.X, (uint32_t)((int64_t)p.M * p.ldx * 2));
  uint32_t xoff[BLK], woff[BLK];
  __amdgpu_buffer_rsrc_t wres[BLK];
  int pi = 0, pk = 0, pke = 0;  // item index and slice of the cursor
  auto producer_setup = [&](int i) {
    const WorkItem it = work_item(sc, b, i);
    const int m0 = it.tm * BM, n0 = it.tn * BN;
    pk = it.kb;
    pke = it.ke;
#pragma unroll
    for (int j = 0; j < BLK; ++j) {
      const int blk = WAVES * j + wave;
      const int row = blk * RPB + lane / LPR;
      const int c = BK == 64 ? (lane % 8) ^ ((row >> 1) & 7) : (lane % 4) ^ ((row >> 2) & 3);
      const int xr = m0 + row;
      xoff[j] = xr < p.M ? (uint32_t)(((int64_t)xr * p.ldx + c * 8) * 2) : CRF_OOB;
      // weight rows: the RPB rows of a block sit in one 64-row group, inside one segment
      const int wr = n0 + row;
      int lr0, local;
      const int sg = segment_of<EPI>(p, min(n0 + blk * RPB, p.N - 1), lr0);
      const int seg_rows = EPI == EPI_QKV ? (sg == 0 ? p.seg1 : sg == 1 ? p.seg2 - p.seg1 : p.N - p.seg2)
                                          : (EPI == EPI_SWIGLU ? p.N / 2 : p.N);
      segment_of<EPI>(p, min(wr, p.N - 1), local);
      wres[j] = make_rsrc(p.w[sg], (uint32_t)((int64_t)seg_rows * p.K * 2));
      woff[j] = wr < p.N ? (uint32_t)(((int64_t)local * p.K + c * 8) * 2) : CRF_OOB;
    }
  };
  // one slice into `stage` (past the last item the cursor stays on the last
  // slice: those copies are never consumed)
  auto produce = [&](int stage) {
    lds_char *dx = (lds_char *)(lds_x + stage * BM * BK);
    lds_char *dw = (lds_char *)(lds_w + stage * BN * BK);
    const uint32_t k0 = (uint32_t)pk * BK * 2;
#pragma unroll
    for (int j = 0; j < BLK; ++j) {
      const int blk = WAVES * j + wave;
      dma16(xres, dx + blk * 1024, xoff[j], k0);
      dma16(wres[j], dw + blk * 1024, woff[j], k0);
    }
  };
  auto advance = [&]() {
    if (++pk == pke) {
      if (pi + 1 < mine) {
        producer_setup(++pi);
      } else {
        pk = pke - 1;
      }
    }
  };

  // ---- fused down-projection adapter sums (EPI_SWIGLU with p.dn_a): wave
  // (wn, wm) owns tokens [64 wm, 64 wm + 64) of half wn of the LDS sums, so the
  // read-add-write below needs no synchronisation.
  float *const dn_lds = (float *)((char *)smem + STAGE_BYTES);
  const bool dn_on = EPI == EPI_SWIGLU && p.dn_a;
  auto dn_zero = [&]() {
    float *d = dn_lds + ((wn * BM + wm * WTM + lane) * DN_RANK);
#pragma unroll
    for (int r = 0; r < DN_RANK; r += 4) *reinterpret_cast<f32x4 *>(d + r) = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  // the sums of a run on token tile tm go to slot `slot`: [slot][wn][256][16]
  auto dn_flush = [&](int tm, int slot) {
    const int ml = wm * WTM + lane, m = tm * BM + ml;
    float *d = dn_lds + ((wn * BM + ml) * DN_RANK);
    float *o = p.dn_part + (((int64_t)slot * 2 + wn) * BM + ml) * DN_RANK;
    float z;  // materialised here: a hoisted zero vector would be spilled
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
#pragma unroll
    for (int r = 0; r < DN_RANK; r += 4) {
      if (m < p.M) *reinterpret_cast<f32x4 *>(o + r) = *reinterpret_cast<f32x4 *>(d + r);
      *reinterpret_cast<f32x4 *>(d + r) = f32x4{z, z, z, z};
    }
  };
  if (dn_on) dn_zero();
  // The factor rows A_down[0..16)[fb, fb + 64) of this wave's 64 features go,
  // right after the last slice's barrier, into x blocks `wave` and
  // `WAVES + wave` of the stage that slice used: nobody reads that stage
  // again, and only this wave refills those blocks (after the epilogue).
  // Instruction t, lane L: rank 8 t + L / 8, features fb + 8 (L % 8) ..+8
  // (ranks at or past dn_rank read as zero).
  int dn_fb = 0;
  auto dn_fetch = [&](int stage) {
    lds_char *dx = (lds_char *)(lds_x + stage * BM * BK);
    const __amdgpu_buffer_rsrc_t dres = make_rsrc(p.dn_a, (uint32_t)((int64_t)p.dn_rank * p.d_ffn * 2));
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int r = 8 * t + lane / 8;
      const uint32_t vo = r < p.dn_rank && dn_fb < p.d_ffn
                              ? (uint32_t)(((int64_t)r * p.d_ffn + dn_fb + 8 * (lane % 8)) * 2)
                              : CRF_OOB;
      dma16(dres, dx + (t * WAVES + wave) * 1024, vo, 0);
    }
  };

  f32x16 acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  constexpr int KSTEPS = BK / 16;
  constexpr int NMM = 4 * NJ, NDS = 4 + NJ;
  auto frag = [&](int stage, int s, bf16x8 (&fa)[4], bf16x8 (&fb)[NJ]) {
    const bf16 *sx = lds_x + stage * BM * BK;
    const bf16 *sw = lds_w + stage * BN * BK;
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = as_bf16x8(ld16(sw + swz(wn * 128 + 32 * i + l32, 2 * s + g)));
#pragma unroll
    for (int j = 0; j < NJ; ++j) fb[j] = as_bf16x8(ld16(sx + swz(wm * WTM + 32 * j + l32, 2 * s + g)));
  };
  auto mm = [&](bf16x8 (&fa)[4], bf16x8 (&fb)[NJ]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32(fa[i], fb[j], acc[i][j]);
  };
  auto interleave = [&](auto n_vmem) {
    constexpr int NV = decltype(n_vmem)::value;
#pragma unroll
    for (int i = 0; i < NMM; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global load
      if (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
  };

  // Ring of STAGES slices.  Each k-step is one scheduling region: its MFMAs
  // with the next step's fragment reads interleaved one by one (the MFMAs use
  // fragments read one region earlier).  The last k-step of a slice follows
  // the slice's single barrier: wait for slice kt+1 (own DMA; later slices
  // may stay in flight), a bare barrier that publishes every wave's part and
  // retires all reads of slice kt, then the refill of that stage with the
  // cursor's slice, interleaved with the MFMAs and with slice kt+1's first
  // reads.  The last slice of an item defers its refill and the next item's
  // first reads until after the epilogue, so the epilogue's own loads do not
  // wait behind that refill.
  bf16x8 a0[4], b0[NJ], a1[4], b1[NJ];
  int st = 0;
  auto slice = [&](auto is_last) {
    constexpr bool LAST = decltype(is_last)::value;
    const int nst = st + 1 == STAGES ? 0 : st + 1;
#pragma unroll
    for (int s = 0; s + 1 < KSTEPS; ++s) {
      __builtin_amdgcn_sched_barrier(0);
      if (s & 1) {
        frag(st, s + 1, a0, b0);
        mm(a1, b1);
      } else {
        frag(st, s + 1, a1, b1);
        mm(a0, b0);
      }
      interleave(std::integral_constant<int, 0>());
      __builtin_amdgcn_sched_barrier(0);
    }
    wait_vm<(STAGES - 2) * DMA_PER_SLICE>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!LAST) {
      produce(st);
      frag(nst, 0, a0, b0);
    } else {
      if (dn_on) dn_fetch(st);
    }
    mm(a1, b1);  // KSTEPS is even: the last k-step of a slice uses (a1, b1)
    interleave(std::integral_constant<int, LAST ? 0 : DMA_PER_SLICE>());
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!LAST) {
      advance();
      st = nst;
    }
  };

  if (mine > 0) {
    producer_setup(0);
#pragma unroll
    for (int s = 0; s < STAGES; ++s) {
      produce(s);
      advance();
    }
    wait_vm<(STAGES - 1) * DMA_PER_SLICE>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    frag(0, 0, a0, b0);
  }

  int run_tm = -1, run_slot = -1, n_run = 0;
  for (int i = 0; i < mine; ++i) {
    const WorkItem it = work_item(sc, b, i);
    const int m0 = it.tm * BM, n0 = it.tn * BN;
    const int part = it.part;

    for (int kt = it.kb; kt + 1 < it.ke; ++kt) slice(std::false_type());
    if (EPI == EPI_SWIGLU) dn_fb = (n0 + wn * 128) / 2;
    slice(std::true_type());

    // ---- low-rank delta: acc += U[token, ucol_s + k] * lb_s[feature, k] (K-part 0 only)
    if (p.U && part <= 0) {
      int seg[4], frow[4];
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int r = min(n0 + wn * 128 + 32 * ii + l32, p.N - 1);
        seg[ii] = segment_of<EPI>(p, r, frow[ii]);
      }
      for (int kk = 0; kk < p.kpad; kk += 16) {
        const int k = kk + 8 * g;
        bf16x8 lbf[4];
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          u32x4 v = {0u, 0u, 0u, 0u};
          const bf16 *lb = p.lb[seg[ii]];
          if (lb && k < p.rank) v = ld16(lb + (int64_t)frow[ii] * p.rank + k);
          lbf[ii] = as_bf16x8(v);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int m = min(m0 + wm * WTM + 32 * j + l32, p.M - 1);
          const bf16 *urow = p.U + (int64_t)m * p.ldu + k;
          // segments used by this wave: blocks 0,1 and 2,3 may differ (EPI_SWIGLU);
          // U columns past the rank stay unread (the factor side is zero there,
          // and they may lie past the row or the buffer)
          const u32x4 zero = {0u, 0u, 0u, 0u};
          const bf16x8 u01 = as_bf16x8(k < p.rank ? ld16(urow + p.ucol[seg[0]]) : zero);
          const bf16x8 u23 = as_bf16x8(k < p.rank ? ld16(urow + p.ucol[seg[2]]) : zero);
#pragma unroll
          for (int ii = 0; ii < 4; ++ii) acc[ii][j] = mfma32(lbf[ii], ii < 2 ? u01 : u23, acc[ii][j]);
        }
      }
    }

    // ---- epilogues
    if ((EPI == EPI_RESID || EPI == EPI_QKV) && part >= 0) {  // fp32 partial of a K-part, [256 tokens][256 features]
      float *pp = p.split_part + (int64_t)(it.w - sc.split_first) * BM * BN;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        float *pr = pp + (wm * WTM + 32 * j + l32) * BN + wn * 128 + 4 * g;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<f32x4 *>(pr + 32 * ii + 8 * q) = f32x4{acc[ii][j][q * 4], acc[ii][j][q * 4 + 1],
                                                                     acc[ii][j][q * 4 + 2], acc[ii][j][q * 4 + 3]};
      }
    } else if (EPI == EPI_RESID) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int m = m0 + wm * WTM + 32 * j + l32;
        if (m >= p.M) continue;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int n = n0 + wn * 128 + 32 * ii + 8 * q + 4 * g;
            if (n >= p.N) continue;
            float *rp = p.resid + (int64_t)m * p.ldr + n;
            f32x4 r = p.resid_overwrite ? f32x4{0.f, 0.f, 0.f, 0.f}
                      : p.resid_in      ? unpack_bf16x4(ld8(p.resid_in + (int64_t)m * p.ldr + n))
                                        : *reinterpret_cast<f32x4 *>(rp);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) r[jj] += acc[ii][j][q * 4 + jj];
            if (!p.resid_final) *reinterpret_cast<f32x4 *>(rp) = r;
            if (p.resid_out) st8(p.resid_out + (int64_t)m * p.ldr + n, pack_bf16x4(r[0], r[1], r[2], r[3]));
          }
      }
    } else if (EPI == EPI_SWIGLU) {
      const int fbase = (n0 + wn * 128) / 2;
      // fused adapter sums: this run's slot (a new run starts on a new token tile)
      if (dn_on) {
        bool head = false;
        if (it.tm != run_tm) {
          if (run_tm >= 0) dn_flush(run_tm, run_slot);
          run_tm = it.tm;
          run_slot = b * p.dn_runs + n_run++;
          head = true;
        }
        // every tile records whether it opens a run (slot + 1) or not (0)
        if (tid == 0) p.dn_head[it.tm * sc.tiles_n + it.tn] = head ? run_slot + 1 : 0;
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int m = m0 + wm * WTM + 32 * j + l32;
        u32x2 packed[2][4];
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float o[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const float gt = acc[ii][j][q * 4 + jj], up = acc[ii + 2][j][q * 4 + jj];
              o[jj] = gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up;
            }
            packed[ii][q] = pack_bf16x4(o[0], o[1], o[2], o[3]);
          }
        // the factor rows' DMA is the only memory operation in flight here
        // (the deferred refill comes after the epilogue): wait for it after
        // the first block's activations (the operands pin the wait there) and
        // before the first act store, so the wait covers nothing else
        if (dn_on && j == 0)
          asm volatile("s_waitcnt vmcnt(0)" ::"v"(packed[0][0]), "v"(packed[0][1]), "v"(packed[0][2]),
                       "v"(packed[0][3]), "v"(packed[1][0]), "v"(packed[1][1]), "v"(packed[1][2]),
                       "v"(packed[1][3])
                       : "memory");
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int f = fbase + 32 * ii + 8 * q + 4 * g;
            if (m < p.M && f < p.d_ffn) st8(p.act + (int64_t)m * p.d_ffn + f, packed[ii][q]);
          }
        if (dn_on && fbase < p.d_ffn) {
          // D[rank, token] += A_down[rank, f] act[token, f] over this wave's 64
          // features, 16 at a time.  The B operand is a lane's own stored act
          // values: k-slot e of k-step (ii, h) is feature
          // fbase + 32 ii + 16 h + 8 (e / 4) + 4 g + e % 4, and the factor rows
          // (rank = l32; rows past the rank are zero) are read in that order.
          f32x16 ud;
#pragma unroll
          for (int v = 0; v < 16; ++v) ud[v] = 0.f;
#pragma unroll
          for (int ii = 0; ii < 2; ++ii)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              // features fbase + 32 ii + 16 h + 4 g ..+4 and 8 further, from
              // 8-feature groups 4 ii + 2 h and 4 ii + 2 h + 1 of row l32
              const int r = l32 & 15;
              const char *ar = (const char *)(lds_x + st * BM * BK) + ((r >> 3) * WAVES + wave) * 1024 +
                               (r & 7) * 128 + (4 * ii + 2 * h) * 16 + 8 * g;
              const u32x2 lo = *reinterpret_cast<const u32x2 *>(ar), hi = *reinterpret_cast<const u32x2 *>(ar + 16);
              const u32x4 av = l32 < DN_RANK ? u32x4{lo[0], lo[1], hi[0], hi[1]} : u32x4{0u, 0u, 0u, 0u};
              const u32x4 bv = {packed[ii][2 * h][0], packed[ii][2 * h][1], packed[ii][2 * h + 1][0],
                                packed[ii][2 * h + 1][1]};
              ud = mfma32(as_bf16x8(av), as_bf16x8(bv), ud);
            }
          // ranks 8 (v / 4) + 4 g + v % 4 for v < 8 (rows 16..31 are padding)
          float *d = dn_lds + (wn * BM + wm * WTM + 32 * j + l32) * DN_RANK + 4 * g;
          f32x4 s0 = *reinterpret_cast<f32x4 *>(d), s1 = *reinterpret_cast<f32x4 *>(d + 8);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            s0[v] += ud[v];
            s1[v] += ud[4 + v];
          }
          *reinterpret_cast<f32x4 *>(d) = s0;
          *reinterpret_cast<f32x4 *>(d + 8) = s1;
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
      for (int j = 0; j < NJ; ++j) {
        const int m = m0 + wm * WTM + 32 * j + l32;
        if (m >= p.M || fb >= p.N) continue;
        int64_t prow[HPW];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) prow[hh] = sg ? paged_row(p.kv, p.pos0 + m, head0 + hh, HD) : 0;
        const float2 *cs = p.rope_cs + (int64_t)(p.pos0 + m) * (HD / 2);
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh)
#pragma unroll
          for (int ii = 0; ii < BPH / 2; ++ii)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int f = 32 * ii + 8 * q + 4 * g;  // in-head index of the first of 4 rows (< HD/2)
              const int b1 = hh * BPH + ii, b2 = b1 + BPH / 2;
              float x1[4], x2[4];
#pragma unroll
              for (int jj = 0; jj < 4; ++jj) {
                x1[jj] = acc[b1][j][q * 4 + jj];
                x2[jj] = acc[b2][j][q * 4 + jj];
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
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                  x1[jj] *= p.q_scale;
                  x2[jj] *= p.q_scale;
                }
              } else {
                if (prow[hh] < 0) continue;
                dst = (bf16 *)(sg == 1 ? p.kv.k : p.kv.v) + prow[hh];
              }
              st8(dst + f, pack_bf16x4(x1[0], x1[1], x1[2], x1[3]));
              st8(dst + f + HD / 2, pack_bf16x4(x2[0], x2[1], x2[2], x2[3]));
            }
      }
    }

    // the deferred refill (the next item's second slice) and the next item's
    // first fragments, then a fresh accumulator
    if (i + 1 < mine) {
      produce(st);
      advance();
      st = st + 1 == STAGES ? 0 : st + 1;
      frag(st, 0, a0, b0);
    }
#pragma unroll
    for (int ii = 0; ii < 4; ++ii)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[ii][j][v] = 0.f;
  }
  if (dn_on && run_tm >= 0) dn_flush(run_tm, run_slot);
  wait_vm<0>();  // refills nobody consumes must land before the workgroup ends
}

// resid[m, n] (+)= sum over the K-parts of a split tile, in part order; one
// thread per 4 features.
__global__ __launch_bounds__(256) void split_reduce_kernel(const GemmParams p, const Sched sc) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // over split tiles x 256 x 64
  const int ti = (int)(idx / (BM * BN / 4));
  const int e = (int)(idx % (BM * BN / 4));
  const int ml = e / (BN / 4), nl = 4 * (e % (BN / 4));
  int tm, tn;
  tile_coords(sc.split_first + ti, sc.tiles_m, sc.tiles_n, tm, tn);
  const int m = tm * BM + ml, n = tn * BN + nl;
  if (m >= p.M || n >= p.N) return;
  const float *pp = p.split_part + (int64_t)ti * sc.split_s * BM * BN + ml * BN + nl;
  f32x4 v = *reinterpret_cast<const f32x4 *>(pp);
  for (int sp = 1; sp < sc.split_s; ++sp) v += *reinterpret_cast<const f32x4 *>(pp + (int64_t)sp * BM * BN);
  float *rp = p.resid + (int64_t)m * p.ldr + n;
  f32x4 r = p.resid_overwrite ? f32x4{0.f, 0.f, 0.f, 0.f}
            : p.resid_in      ? unpack_bf16x4(ld8(p.resid_in + (int64_t)m * p.ldr + n))
                              : *reinterpret_cast<f32x4 *>(rp);
  r += v;
  if (!p.resid_final) *reinterpret_cast<f32x4 *>(rp) = r;
  if (p.resid_out) st8(p.resid_out + (int64_t)m * p.ldr + n, pack_bf16x4(r[0], r[1], r[2], r[3]));
}

// The K-parts of a split QKV tile summed in part order, then the QKV epilogue:
// bias, rotary rotation of Q and K, Q to its buffer and K/V into the pages.
// One thread per 4 in-head features f..f+3 and their rotary partners
// f+HD/2..f+HD/2+3 of one token (32 threads per token and tile).
template <int HD>
__global__ __launch_bounds__(256) void qkv_split_reduce_kernel(const GemmParams p, const Sched sc) {
  constexpr int TPH = HD / 8;  // threads per head
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // over split tiles x 256 tokens x 32
  const int ti = (int)(idx / (BM * 32));
  const int e = (int)(idx % (BM * 32));
  const int ml = e / 32, c = e % 32;
  const int n1 = (c / TPH) * HD + 4 * (c % TPH);  // tile column of the first feature
  int tm, tn;
  tile_coords(sc.split_first + ti, sc.tiles_m, sc.tiles_n, tm, tn);
  const int m = tm * BM + ml, r = tn * BN + n1;
  if (m >= p.M || r >= p.N) return;
  const float *pp = p.split_part + (int64_t)ti * sc.split_s * BM * BN + ml * BN + n1;
  f32x4 x1 = *reinterpret_cast<const f32x4 *>(pp), x2 = *reinterpret_cast<const f32x4 *>(pp + HD / 2);
  for (int sp = 1; sp < sc.split_s; ++sp) {
    x1 += *reinterpret_cast<const f32x4 *>(pp + (int64_t)sp * BM * BN);
    x2 += *reinterpret_cast<const f32x4 *>(pp + (int64_t)sp * BM * BN + HD / 2);
  }
  int local;
  const int sg = segment_of<EPI_QKV>(p, r, local);
  const int head = local / HD, f = local % HD;
  if (const bf16 *bias = p.bias[sg]) {
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      x1[jj] += bf2f(bias[head * HD + f + jj]);
      x2[jj] += bf2f(bias[head * HD + f + HD / 2 + jj]);
    }
  }
  if (sg < 2) {
    const float2 *cs = p.rope_cs + (int64_t)(p.pos0 + m) * (HD / 2) + f;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const float2 cj = cs[jj];
      const float y1 = x1[jj] * cj.x - x2[jj] * cj.y;
      const float y2 = x2[jj] * cj.x + x1[jj] * cj.y;
      x1[jj] = y1;
      x2[jj] = y2;
    }
  }
  bf16 *dst;
  if (sg == 0) {
    dst = p.q_out + (int64_t)m * p.dq + head * HD;
    x1 *= p.q_scale;
    x2 *= p.q_scale;
  } else {
    const int64_t prow = paged_row(p.kv, p.pos0 + m, head, HD);
    if (prow < 0) return;
    dst = (bf16 *)(sg == 1 ? p.kv.k : p.kv.v) + prow;
  }
  st8(dst + f, pack_bf16x4(x1[0], x1[1], x1[2], x1[3]));
  st8(dst + f + HD / 2, pack_bf16x4(x2[0], x2[1], x2[2], x2[3]));
}

// U[m, ucol + r] = bf16(scale * sum of the fused down-projection adapter sums
// of token m): over the runs that cover m's token tile in increasing order of
// their first tile, then over the two feature halves.  One thread per 4 ranks.
constexpr int DN_MAX_TILES_N = 1024;  // feature tiles of a gate/up row the slot list holds (d_ffn <= 131072)

__global__ __launch_bounds__(256) void dn_sum_kernel(const GemmParams p, const Sched sc, bf16 *U, int ldu, int ucol,
                                                     float scale) {
  // the workgroup's 64 tokens share one token tile: its slots, in order of
  // their first feature tile, are listed once in LDS (wave 0 compacts the
  // table with ballots), then every thread walks the short list
  __shared__ int slots[DN_MAX_TILES_N];
  __shared__ int n_slots;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int m = idx / (DN_RANK / 4), r = 4 * (idx % (DN_RANK / 4));
  const int tm = (blockIdx.x * 256 / (DN_RANK / 4)) / BM, ml = m % BM;
  if (threadIdx.x < 64) {
    const int *head = p.dn_head + tm * sc.tiles_n;
    int count = 0;
    for (int t0 = 0; t0 < sc.tiles_n; t0 += 64) {
      const int tn = t0 + (int)threadIdx.x;
      const int h = tn < sc.tiles_n ? head[tn] : 0;
      const uint64_t mask = __ballot(h != 0);
      if (h) slots[count + __popcll(mask & ((1ull << threadIdx.x) - 1))] = h - 1;
      count += __popcll(mask);
    }
    if (threadIdx.x == 0) n_slots = count;
  }
  __syncthreads();
  if (m >= p.M || r >= p.dn_rank) return;
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < n_slots; ++i) {
    const int slot = slots[i];
#pragma unroll
    for (int wn = 0; wn < 2; ++wn)
      v += *reinterpret_cast<const f32x4 *>(p.dn_part + (((int64_t)slot * 2 + wn) * BM + ml) * DN_RANK + r);
  }
  bf16 *u = U + (int64_t)m * ldu + ucol + r;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (r + q < p.dn_rank) u[q] = f2bf(v[q] * scale);
}

Sched schedule(GemmEpi epi, const GemmParams &p) {
  Sched sc{};
  sc.tiles_m = (p.M + BM - 1) / BM;
  sc.tiles_n = (p.N + BN - 1) / BN;
  sc.nk = p.K / BK;
  const int tiles = sc.tiles_m * sc.tiles_n;
  sc.split_first = tiles;
  sc.split_s = 1;
  if ((epi == EPI_RESID || epi == EPI_QKV) && p.split_part && p.n_cu > 0) {
    // a last wave at most half full: split its tiles (or all tiles, when there
    // are fewer than compute units) into K-parts of at least 8 slices
    const int r = tiles % p.n_cu;
    int first = tiles, sp = 1;
    if (tiles < p.n_cu) {
      first = 0;
      sp = p.n_cu / tiles;
    } else if (r > 0 && 2 * r <= p.n_cu) {
      first = tiles - r;
      sp = 2;
    }
    sp = std::min(sp, std::min(8, sc.nk / 8));
    if (sp >= 2 && (int64_t)(tiles - first) * sp * BM * BN <= p.split_cap) {
      sc.split_first = first;
      sc.split_s = sp;
    }
  }
  sc.n_items = sc.split_first + (tiles - sc.split_first) * sc.split_s;
  sc.grid = p.n_cu > 0 ? std::min(sc.n_items, p.n_cu) : sc.n_items;
  // K-parts sit at the end of every workgroup's list when the last round is
  // split; with a short K range (where the residual epilogue is a large share
  // of an item) odd workgroups take theirs first, so that half of the
  // workgroups reach each residual epilogue at another time
  sc.stagger = sc.split_s > 1 && sc.split_first % sc.grid == 0 && (sc.n_items - sc.split_first) == sc.grid &&
               sc.nk <= 128;
  return sc;
}

template <int EPI, int HD>
hipError_t go(hipStream_t s, const GemmParams &p0, bool *dn_done) {
  GemmParams p = p0;
  const Sched sc = schedule((GemmEpi)EPI, p);
  p.split_first = sc.split_first;
  p.split_s = sc.split_s;
  bool dn = false;
  if (EPI == EPI_SWIGLU && p.dn_a && p.dn_part && p.dn_head && p.dn_rank > 0 && p.dn_rank <= DN_RANK &&
      p.dn_runs > 0 && STAGE_BYTES + DN_BYTES <= 160 * 1024 && sc.tiles_n <= DN_MAX_TILES_N) {
    int runs = 0;
    for (int b = 0; b < sc.grid && runs <= p.dn_runs; ++b) runs = std::max(runs, n_runs(sc, b));
    dn = runs <= p.dn_runs;
  }
  if (!dn) p.dn_a = nullptr;
  if (dn_done) *dn_done = dn;
  const size_t lds = (size_t)STAGE_BYTES + (dn ? DN_BYTES : 0);
  // the dynamic-LDS limit is raised once per device (bit d of attr_set)
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
  if (!bit || !(attr_set.load() & bit)) {
    e = hipFuncSetAttribute((const void *)gemm_bf16_kernel<EPI, HD>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            STAGE_BYTES + (EPI == EPI_SWIGLU ? DN_BYTES : 0));
    if (e != hipSuccess) return e;
    attr_set.fetch_or(bit);
  }
  hipLaunchKernelGGL((gemm_bf16_kernel<EPI, HD>), dim3(sc.grid), dim3(64 * WAVES), lds, s, p, sc);
  if (sc.split_s > 1) {
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int split_tiles = sc.tiles_m * sc.tiles_n - sc.split_first;
    if (EPI == EPI_QKV) {
      const int64_t n = (int64_t)split_tiles * BM * 32;
      hipLaunchKernelGGL((qkv_split_reduce_kernel<HD>), dim3((unsigned)(n / 256)), dim3(256), 0, s, p, sc);
    } else {
      const int64_t n = (int64_t)split_tiles * BM * BN / 4;
      hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)(n / 256)), dim3(256), 0, s, p, sc);
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(hipStream_t s, GemmEpi epi, int hd, const GemmParams &p, bool *dn_done) {
  if (dn_done) *dn_done = false;
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (p.K % BK) return hipErrorInvalidValue;
  if ((int64_t)p.M * p.ldx * 2 >= (int64_t)CRF_OOB) return hipErrorInvalidValue;  // X must fit one buffer resource
  switch (epi) {
    case EPI_RESID: return go<EPI_RESID, 128>(s, p, nullptr);
    case EPI_SWIGLU: return go<EPI_SWIGLU, 128>(s, p, dn_done);
    case EPI_QKV: return hd == 64 ? go<EPI_QKV, 64>(s, p, nullptr) : go<EPI_QKV, 128>(s, p, nullptr);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_dn_sum(hipStream_t s, const GemmParams &p, bf16 *U, int ldu, int ucol, float scale) {
  if (p.M <= 0) return hipSuccess;
  const Sched sc = schedule(EPI_SWIGLU, p);
  const int threads = p.M * (DN_RANK / 4);
  if (sc.tiles_n > DN_MAX_TILES_N) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dn_sum_kernel, dim3((threads + 255) / 256), dim3(256), 0, s, p, sc, U, ldu, ucol, scale);
  return hipGetLastError();
}

}  // namespace crf
