// Launchers of the device kernels (internal to libcrf.so).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace crf {

// ---------------------------------------------------------------- shared
// y = g * x / sqrt(mean(x^2) + eps) row-wise over d; x fp32 or bf16, y fp32 or
// bf16, g in the model dtype.  copy_out (nullable) receives x as fp32.
hipError_t launch_rmsnorm(hipStream_t s, const void *x, bool x_f32, const void *g, bool g_f32, void *y,
                          bool y_f32, float *copy_out, int M, int d, float eps);
// cos/sin table cs[p*hd/2 + i] = (cos, sin)(p * theta^(-2i/hd)), angles in fp64.
hipError_t launch_rope_table(hipStream_t s, float2 *cs, int T, int hd, float theta);

// ---------------------------------------------------------------- fp32 path
// C = alpha * A B^T + beta * C with A [M,K] (lda), B [N,K] (ldb), C [M,N] (ldc).
hipError_t launch_gemm_f32(hipStream_t s, int M, int N, int K, const float *A, int lda, const float *B, int ldb,
                           float *C, int ldc, float alpha, float beta);
// P [M, dq+2dkv] -> Q (rotated) [M, dq], K (rotated) and V written to pages.
hipError_t launch_qkv_post_f32(hipStream_t s, const float *P, const float *bq, const float *bk, const float *bv,
                               float *Q, const PagedKV &kv, const float2 *cs, int M, int nq, int nkv, int hd);
// act[m, f] = silu(G[m, f]) * U[m, f] with G = GU[:, :f], U = GU[:, f:2f].
hipError_t launch_silu_mul_f32(hipStream_t s, const float *GU, float *act, int M, int f);
hipError_t launch_attn_f32(hipStream_t s, const float *Q, const PagedKV &kv, float *O, int M, int nq, int nkv,
                           int hd);

// ---------------------------------------------------------------- bf16 path
struct LoraDownTarget {
  const bf16 *A;   // [rank, K] or nullptr
  int rank;
  float scale;
  int ucol;        // first column of this target in U
};
// U[m, ucol_t + j] = bf16(scale_t * sum_k X[m,k] A_t[j,k]) for j < rank_pad(t)
// (zero for rank <= j < rank_pad).
// ws (nullable, ws_floats floats): workspace for splitting K over workgroups
// when M <= 16.  With `split` non-null, a split into at most four parts is
// left as unscaled fp32 partials in ws ([part][16][n_targets * rank_pad]) for
// the consuming projection to sum (split->n_parts > 0; U is not written);
// otherwise split->n_parts = 0 and U holds the result.
struct LoraSplit {
  int n_parts = 0;
  int cols = 0;
};
hipError_t launch_lora_down_bf16(hipStream_t s, const bf16 *X, int64_t ldx, int M, int K, const LoraDownTarget *t,
                                 int n_targets, int rank_pad, bf16 *U, int ldu, float *ws, int64_t ws_floats,
                                 LoraSplit *split = nullptr);

enum GemmEpi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };

struct GemmParams {
  const bf16 *X;
  int64_t ldx;
  int M, K;
  int N;                       // rows of the (virtual) weight matrix in tile space
  const bf16 *w[3];            // segment row sources, each [rows, K]
  int seg1, seg2;              // EPI_QKV: first rows of the k and v segments
  // LoRA delta: acc += U[:, ucol_s : ucol_s + kpad] * lb_s^T  per segment s
  const bf16 *U;
  int ldu, kpad, rank;
  const bf16 *lb[3];           // [seg_rows, rank] or nullptr
  int ucol[3];
  // EPI_QKV
  const bf16 *bias[3];
  bf16 *q_out;
  int dq;
  float q_scale;               // factor applied to Q (after bias and rotary) before it is stored
  PagedKV kv;
  const float2 *rope_cs;
  // EPI_QKV: token row m sits at position pos0 + m (rotary angle and page slot)
  int pos0;
  // EPI_RESID: resid[m, n] += acc (= acc when resid_overwrite); resid_out (nullable) = bf16(resid)
  float *resid;
  // EPI_RESID (nullable): the residual before the update in bf16, same layout
  // as resid, read instead of resid (the window's first update reads its
  // boundary state directly, so the fp32 copy of it is never written)
  const bf16 *resid_in;
  bf16 *resid_out;
  int resid_final;  // EPI_RESID with resid_out: the updated residual is stored only as resid_out
  int ldr;
  int resid_overwrite;
  // EPI_SWIGLU: act[m, f] = silu(gate) * up
  bf16 *act;
  int d_ffn;
  // EPI_QKV with few token rows: fp32 projections [M, N] before the rotary/paged stores
  float *proj;
  // few token rows: U given as unscaled K-split partials ([part][16][upart_cols]
  // fp32, upart_n parts) to be summed, scaled by uscale and rounded to bf16
  const float *upart;
  int upart_n, upart_cols;
  float uscale;
  // EPI_RESID: when the tiles leave the last wave of the grid at most half
  // full (n_cu compute units), the last tiles are split into K-parts that
  // write fp32 partials to split_part (split_cap floats) and a second kernel
  // adds them to the residual in a fixed order.  split_first / split_s are
  // set by the launcher.
  float *split_part;
  int64_t split_cap;
  int n_cu;
  int split_first, split_s;
  // EPI_SWIGLU: the down projection's adapter down-projection fused into the
  // epilogue (rank <= 16): dn_a = A_down [dn_rank, d_ffn].  Each workgroup sums
  // act . A_down^T over the features of consecutive items on one token tile (a
  // run) and leaves the sums in dn_part slot b * dn_runs + run ([slot][2][256][16]
  // fp32); dn_head[tm * tiles_n + tn] = slot + 1 for the first tile of a run,
  // else 0.  launch_gemm_dn_sum then forms U.
  const bf16 *dn_a;
  int dn_rank;
  float *dn_part;
  int *dn_head;
  int dn_runs;
};
// Persistent over at most n_cu workgroups (n_cu > 0).  *dn_done (nullable)
// reports whether the fused down-projection sums were produced (they are
// skipped when a workgroup would need more than dn_runs runs).
hipError_t launch_gemm_bf16(hipStream_t s, GemmEpi epi, int hd, const GemmParams &p, bool *dn_done = nullptr);
// U[m, ucol + r] = bf16(scale * sum of the fused sums) for r < dn_rank, after
// launch_gemm_bf16(EPI_SWIGLU) reported *dn_done with the same parameters.
hipError_t launch_gemm_dn_sum(hipStream_t s, const GemmParams &p, bf16 *U, int ldu, int ucol, float scale);
// The same projections for M <= 16 token rows (weight-streaming bound).
hipError_t launch_gemm_skinny_bf16(hipStream_t s, GemmEpi epi, int hd, const GemmParams &p);

// Factor the attention kernel expects the stored query rows to carry:
// log2(e) / sqrt(head_dim) (scores then come out in log2 units).
inline float attn_query_scale(int hd) { return 1.4426950408889634f / __builtin_sqrtf((float)hd); }
// Query rows 0..Mq-1 at positions q_off..q_off+Mq-1 over keys 0..q_off+Mq-1,
// Q pre-multiplied by attn_query_scale(hd).
// part (nullable, part_floats floats): workspace for splitting a few query
// rows (<= 16) over the keys of a long prefix.
hipError_t launch_attn_bf16(hipStream_t s, const bf16 *Q, const PagedKV &kv, bf16 *O, int Mq, int q_off, int nq,
                            int nkv, int hd, float *part, int64_t part_floats);

// ---------------------------------------------------------------- drift
struct DriftSeg {
  const void *a;     // current adapter tensor
  const void *b;     // stored version tensor
  int64_t count;     // elements
  int out;           // output index v * n_layers + l
};
struct DriftChunk {
  int seg;
  int64_t start, len;
};
hipError_t launch_drift_partials(hipStream_t s, const DriftSeg *segs, const DriftChunk *chunks, int n_chunks,
                                 bool f32, double *partials);
// Device address of the no-allocation drift scratch on the current device
// (CRF_DRIFT_NOALLOC_MAX_BYTES, looked up once per device).
hipError_t drift_noalloc_scratch(void **out);
hipError_t launch_drift_finalize(hipStream_t s, const double *partials, const int *chunk_first,
                                 const int *chunk_count, int n_versions, int n_layers, const int *anchor,
                                 const float *sens, int per_layer_only, float *drift, float *risk, float *sq_out,
                                 double *scratch);

}  // namespace crf
