// bf16 MFMA GEMM  D[feature, token] = W[feature, :] . X[token, :]  for the four
// projections of a decoder layer, with the low-rank adapter delta applied as a
// second, skinny contraction (K = padded rank) on the same accumulators and a
// fused epilogue:
//   EPI_QKV    bias + rotary rotation of Q and K, Q to a [M, dq] buffer, K and V
//              straight into the layer's pages of the paged cache;
//   EPI_RESID  fp32 residual update (attention output / down projection);
//   EPI_SWIGLU silu(gate) * up with gate and up rows interleaved per 64 features.
//
// Tiling for CDNA4: a 256x256 output tile per workgroup, either 4 waves of
// 128x128 (one wave per SIMD) or 8 waves of 128x64 (two waves per SIMD, so one
// wave issues MFMAs while the other waits on LDS or memory); every wave owns
// 128 output features.  v_mfma_f32_32x32x16_bf16; K staged through LDS in
// 64-wide slices, double-buffered (2 x 64 KB).  Slices move global -> LDS by
// DMA (buffer_load ... lds): no staging registers and no LDS stores in the
// waves' instruction stream; slice kt+2's DMA is issued right after the single
// per-slice barrier and overlaps slice kt+1's MFMAs, and fragment reads run one
// MFMA group ahead.  Rows past M (or past N) get an out-of-range offset and
// arrive as zeros.  The weight operand takes the MFMA "A"
// role so each lane ends up holding 4 consecutive output features of one
// token, which makes every epilogue lane-local (a rotary pair (f, f+hd/2) and a
// gate/up pair live in the same lane).  16-byte LDS chunks are XOR-swizzled by
// (row/2) mod 8 so the fragment reads are bank-conflict free.
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
#ifndef CRF_GEMM_WAVES
#define CRF_GEMM_WAVES 8
#endif

constexpr int BM = 256, BN = 256;
constexpr int BK = CRF_GEMM_BK;          // k-width of one LDS slice
constexpr int STAGES = CRF_GEMM_STAGES;  // slices resident in LDS (STAGES * 32 KB per 32 of BK)
constexpr int GROUP_M = 8;
constexpr int LPR = BK / 8;              // 16-byte chunks (lanes) per row of a slice
constexpr int RPB = 64 / LPR;            // rows per 1 KB DMA block
static_assert(BK == 32 || BK == 64, "slice width");
static_assert(STAGES >= 2 && STAGES * (BM + BN) * BK * 2 <= 160 * 1024, "LDS budget");

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

// Tile t of the grouped order (GROUP_M token tiles share a weight panel).
CRF_DEV void tile_coords(int t, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int group = GROUP_M * tiles_n;
  const int first_m = (t / group) * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  tm = first_m + (t % group) % gm;
  tn = (t % group) / gm;
}

// WAVES = 4: 2 (features) x 2 (tokens) waves of 128 x 128.
// WAVES = 8: 2 (features) x 4 (tokens) waves of 128 x 64.
template <int EPI, int HD, int WAVES>
__global__ __launch_bounds__(64 * WAVES, 1) void gemm_bf16_kernel(const GemmParams p) {
  constexpr int NT = 64 * WAVES;
  constexpr int WM_COUNT = WAVES / 2;      // token groups
  constexpr int WTM = BM / WM_COUNT;       // tokens per wave: 128 or 64
  constexpr int NJ = WTM / 32;             // 32-token blocks per wave
  constexpr int BLK = (BM / RPB) / WAVES;  // 1 KB DMA blocks per operand per wave per slice
  constexpr int DMA_PER_SLICE = 2 * BLK;
  extern __shared__ __align__(16) bf16 smem[];
  bf16 *const lds_x = smem;                       // [STAGES][BM*BK]
  bf16 *const lds_w = smem + STAGES * BM * BK;    // [STAGES][BN*BK]

  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = (p.N + BN - 1) / BN;
  const int nk = p.K / BK;
  // work item: a whole tile, or K-part `part` of one of the last tiles.  The
  // whole tiles come first in dispatch order and the K-parts after them, each
  // range remapped on its own so that every XCD gets an equal, contiguous
  // share of both.
  int w, t, part = -1, kb = 0, ke = nk;
  if (EPI == EPI_RESID && p.split_s > 1 && (int)blockIdx.x >= p.split_first) {
    const int n_parts = (int)gridDim.x - p.split_first;
    w = p.split_first + xcd_remap((int)blockIdx.x - p.split_first, n_parts);
    t = p.split_first + (w - p.split_first) / p.split_s;
    part = (w - p.split_first) % p.split_s;
    kb = part * nk / p.split_s;
    ke = (part + 1) * nk / p.split_s;
  } else {
    w = xcd_remap(blockIdx.x, EPI == EPI_RESID && p.split_s > 1 ? p.split_first : gridDim.x);
    t = w;
  }
  int tm, tn;
  tile_coords(t, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);  // uniform: keeps DMA targets scalar
  const int wn = wave / WM_COUNT, wm = wave % WM_COUNT;
  const int g = lane / 32, l32 = lane % 32;

  // ---- global -> LDS DMA.  A slice of one operand is 256 rows x BK k = BK/2
  // blocks of 1 KB; wave w moves blocks WAVES*j + w.  Inside a block, lane L
  // writes LDS bytes [16 L, 16 L + 16): row RPB*block + L/LPR, swizzled
  // position L%LPR, which holds the logical k-chunk at that position of swz.
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(p.X, (uint32_t)((int64_t)p.M * p.ldx * 2));
  uint32_t xoff[BLK], woff[BLK];
  __amdgpu_buffer_rsrc_t wres[BLK];
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
  auto dma = [&](int k0, int stage) {
    lds_char *dx = (lds_char *)(lds_x + stage * BM * BK);
    lds_char *dw = (lds_char *)(lds_w + stage * BN * BK);
#pragma unroll
    for (int j = 0; j < BLK; ++j) {
      const int blk = WAVES * j + wave;
      dma16(xres, dx + blk * 1024, xoff[j], (uint32_t)k0 * 2);
      dma16(wres[j], dw + blk * 1024, woff[j], (uint32_t)k0 * 2);
    }
  };
  // blocks [J0, J1) of both operands
  auto dma_part = [&](int k0, int stage, auto j0, auto j1) {
    constexpr int J0 = decltype(j0)::value, J1 = decltype(j1)::value;
    lds_char *dx = (lds_char *)(lds_x + stage * BM * BK);
    lds_char *dw = (lds_char *)(lds_w + stage * BN * BK);
#pragma unroll
    for (int j = J0; j < J1; ++j) {
      const int blk = WAVES * j + wave;
      dma16(xres, dx + blk * 1024, xoff[j], (uint32_t)k0 * 2);
      dma16(wres[j], dw + blk * 1024, woff[j], (uint32_t)k0 * 2);
    }
  };

  f32x16 acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // ---- low-rank delta: acc += U[token, ucol_s + k] * lb_s[feature, k] (K-part 0 only)
  if (p.U && part <= 0) {
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
        for (int i = 0; i < 4; ++i) acc[i][j] = mfma32(lbf[i], i < 2 ? u01 : u23, acc[i][j]);
      }
    }
  }

  constexpr int KSTEPS = BK / 16;
  constexpr int NMM = 4 * NJ, NDS = 4 + NJ;
  constexpr int NMM4 = NMM;
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
  if constexpr (WAVES == 4) {
    // One wave per SIMD: no second wave covers a stall, so fragments are read
    // two k-steps ahead of their MFMAs (one register set per k-step of a
    // slice).  The slice barrier sits after k-step 1: by then this wave has
    // read all of slice kt (its k-steps 2 and 3 were read during k-steps 0
    // and 1), so the stage can take slice kt+2, and slice kt+1 (issued one
    // slice earlier) has landed for the reads made during k-steps 2 and 3.
    static_assert(BK == 64 && STAGES == 2, "two stages of 64-wide slices");
    bf16x8 fa[4][4], fb[4][NJ];
    // per k-step region: 16 MFMAs; the first 8 each followed by one LDS read
    // and, when refilling, one global->LDS load
    auto sched = [&](auto n_vmem) {
      constexpr int NV = decltype(n_vmem)::value;
#pragma unroll
      for (int i = 0; i < NMM4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (i < 4 + NJ) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    };
    dma(kb * BK, 0);
    dma(min(kb + 1, ke - 1) * BK, 1);
    wait_vm<DMA_PER_SLICE>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    frag(0, 0, fa[0], fb[0]);
    frag(0, 1, fa[1], fb[1]);
    for (int kt = kb; kt < ke; ++kt) {
      const int st = (kt - kb) & 1;
      __builtin_amdgcn_sched_barrier(0);
      frag(st, 2, fa[2], fb[2]);
      mm(fa[0], fb[0]);
      sched(std::integral_constant<int, 0>());
      __builtin_amdgcn_sched_barrier(0);
      frag(st, 3, fa[3], fb[3]);
      mm(fa[1], fb[1]);
      sched(std::integral_constant<int, 0>());
      __builtin_amdgcn_sched_barrier(0);
      wait_vm<0>();
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      __builtin_amdgcn_sched_barrier(0);
      const int kn = min(kt + 2, ke - 1) * BK;  // clamped: every slice issues the same loads
      dma_part(kn, st, std::integral_constant<int, 0>(), std::integral_constant<int, BLK / 2>());
      frag(st ^ 1, 0, fa[0], fb[0]);
      mm(fa[2], fb[2]);
      sched(std::integral_constant<int, BLK>());
      __builtin_amdgcn_sched_barrier(0);
      dma_part(kn, st, std::integral_constant<int, BLK / 2>(), std::integral_constant<int, BLK>());
      frag(st ^ 1, 1, fa[1], fb[1]);
      mm(fa[3], fb[3]);
      sched(std::integral_constant<int, BLK>());
      __builtin_amdgcn_sched_barrier(0);
    }
    wait_vm<0>();
  } else {
  // Ring of STAGES slices.  The prologue puts slices 0..STAGES-1 in flight.
  // Each k-step is one scheduling region: its MFMAs with the next step's
  // fragment reads interleaved one by one (the MFMAs use fragments read one
  // region earlier).  The last k-step of a slice follows the slice's single
  // barrier: wait for slice kt+1 (own DMA; later slices may stay in flight),
  // a bare barrier that publishes every wave's part and retires all reads of
  // slice kt, then the refill of that stage with slice kt+STAGES (clamped to
  // the last slice near the end, so every slice issues the same number of
  // loads), interleaved with the MFMAs and with slice kt+1's first reads.

  auto interleave = [&](auto n_vmem) {
    constexpr int NV = decltype(n_vmem)::value;
#pragma unroll
    for (int i = 0; i < NMM; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global load
      if (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
  };
#pragma unroll
  for (int s = 0; s < STAGES; ++s) dma(min(kb + s, ke - 1) * BK, s);
  wait_vm<(STAGES - 1) * DMA_PER_SLICE>();
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  bf16x8 a0[4], b0[NJ], a1[4], b1[NJ];
  frag(0, 0, a0, b0);
  int st = 0;
  for (int kt = kb; kt < ke; ++kt) {
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
    // also after the last slice (stage nst then holds a clamped copy): the loop
    // body stays one basic block per region
    wait_vm<(STAGES - 2) * DMA_PER_SLICE>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    dma(min(kt + STAGES, ke - 1) * BK, st);
    frag(nst, 0, a0, b0);
    mm(a1, b1);  // KSTEPS is even: the last k-step of a slice uses (a1, b1)
    interleave(std::integral_constant<int, DMA_PER_SLICE>());
    __builtin_amdgcn_sched_barrier(0);
    st = nst;
  }
  wait_vm<0>();  // the clamped refills of the last slices
  }

  // ---- epilogues
  if (EPI == EPI_RESID && part >= 0) {  // fp32 partial of a K-part, [256 tokens][256 features]
    float *pp = p.split_part + (int64_t)(w - p.split_first) * BM * BN;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int ml = wm * WTM + 32 * j + l32;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int nl = wn * 128 + 32 * i + 8 * ii + 4 * g;
          *reinterpret_cast<f32x4 *>(pp + ml * BN + nl) =
              f32x4{acc[i][j][ii * 4], acc[i][j][ii * 4 + 1], acc[i][j][ii * 4 + 2], acc[i][j][ii * 4 + 3]};
        }
    }
  } else if (EPI == EPI_RESID) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int m = m0 + wm * WTM + 32 * j + l32;
      if (m >= p.M) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int n = n0 + wn * 128 + 32 * i + 8 * ii + 4 * g;
          if (n >= p.N) continue;
          float *rp = p.resid + (int64_t)m * p.ldr + n;
          f32x4 r = p.resid_overwrite ? f32x4{0.f, 0.f, 0.f, 0.f} : *reinterpret_cast<f32x4 *>(rp);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) r[jj] += acc[i][j][ii * 4 + jj];
          *reinterpret_cast<f32x4 *>(rp) = r;
          if (p.resid_out) st8(p.resid_out + (int64_t)m * p.ldr + n, pack_bf16x4(r[0], r[1], r[2], r[3]));
        }
    }
  } else if (EPI == EPI_SWIGLU) {
    const int fbase = (n0 + wn * 128) / 2;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int m = m0 + wm * WTM + 32 * j + l32;
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

// resid[m, n] (+)= sum over the K-parts of a split tile, in part order; one
// thread per 4 features.
__global__ __launch_bounds__(256) void split_reduce_kernel(const GemmParams p) {
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // over split tiles x 256 x 64
  const int ti = (int)(idx / (BM * BN / 4));
  const int e = (int)(idx % (BM * BN / 4));
  const int ml = e / (BN / 4), nl = 4 * (e % (BN / 4));
  int tm, tn;
  tile_coords(p.split_first + ti, tiles_m, tiles_n, tm, tn);
  const int m = tm * BM + ml, n = tn * BN + nl;
  if (m >= p.M || n >= p.N) return;
  const float *pp = p.split_part + (int64_t)ti * p.split_s * BM * BN + ml * BN + nl;
  f32x4 v = *reinterpret_cast<const f32x4 *>(pp);
  for (int sp = 1; sp < p.split_s; ++sp) v += *reinterpret_cast<const f32x4 *>(pp + (int64_t)sp * BM * BN);
  float *rp = p.resid + (int64_t)m * p.ldr + n;
  f32x4 r = p.resid_overwrite ? f32x4{0.f, 0.f, 0.f, 0.f} : *reinterpret_cast<f32x4 *>(rp);
  r += v;
  *reinterpret_cast<f32x4 *>(rp) = r;
  if (p.resid_out) st8(p.resid_out + (int64_t)m * p.ldr + n, pack_bf16x4(r[0], r[1], r[2], r[3]));
}

template <int EPI, int HD, int WAVES>
hipError_t go(hipStream_t s, const GemmParams &p0) {
  const int tiles = ((p0.M + BM - 1) / BM) * ((p0.N + BN - 1) / BN);
  GemmParams p = p0;
  p.split_first = tiles;
  p.split_s = 1;
  if (EPI == EPI_RESID && p.split_part && p.n_cu > 0) {
    // a last wave at most half full: split its tiles (or all tiles, when there
    // are fewer than compute units) into K-parts of at least 8 slices
    const int nk = p.K / BK, r = tiles % p.n_cu;
    int first = tiles, sp = 1;
    if (tiles < p.n_cu) {
      first = 0;
      sp = p.n_cu / tiles;
    } else if (r > 0 && 2 * r <= p.n_cu) {
      first = tiles - r;
      sp = 2;
    }
    sp = std::min(sp, std::min(8, nk / 8));
    if (sp >= 2 && (int64_t)(tiles - first) * sp * BM * BN <= p.split_cap) {
      p.split_first = first;
      p.split_s = sp;
    }
  }
  const int grid = p.split_first + (tiles - p.split_first) * p.split_s;
  const size_t lds = (size_t)STAGES * (BM + BN) * BK * sizeof(bf16);
  // the dynamic-LDS limit is raised once per device (bit d of attr_set)
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
  if (!bit || !(attr_set.load() & bit)) {
    e = hipFuncSetAttribute((const void *)gemm_bf16_kernel<EPI, HD, WAVES>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
    if (e != hipSuccess) return e;
    attr_set.fetch_or(bit);
  }
  hipLaunchKernelGGL((gemm_bf16_kernel<EPI, HD, WAVES>), dim3(grid), dim3(64 * WAVES), lds, s, p);
  if (p.split_s > 1) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)(tiles - p.split_first) * BM * BN / 4;
    hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)(n / 256)), dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(hipStream_t s, GemmEpi epi, int hd, const GemmParams &p) {
  constexpr int W = CRF_GEMM_WAVES;
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (p.K % BK) return hipErrorInvalidValue;
  if ((int64_t)p.M * p.ldx * 2 >= (int64_t)CRF_OOB) return hipErrorInvalidValue;  // X must fit one buffer resource
  switch (epi) {
    case EPI_RESID: return go<EPI_RESID, 128, W>(s, p);
    case EPI_SWIGLU: return go<EPI_SWIGLU, 128, W>(s, p);
    case EPI_QKV: return hd == 64 ? go<EPI_QKV, 64, W>(s, p) : go<EPI_QKV, 128, W>(s, p);
  }
  return hipErrorInvalidValue;
}

}  // namespace crf
