// Host side of the C ABI (include/crf.h): validation, workspace, launch order.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <initializer_list>
#include <string>
#include <vector>

#include "../../include/crf.h"
#include "kernels.hpp"

using namespace crf;

namespace {

thread_local std::string g_last_error;

struct Timer {
  uint32_t mask = 0;            // bit k: launches of class k are bracketed by events
  std::vector<hipEvent_t> ev;   // pairs (start, stop)
  std::vector<int> kind;        // per pair
  size_t used = 0;              // pairs recorded since last read
};

}  // namespace

// runs of consecutive gate/up tiles on one token tile per workgroup whose fused
// down-projection adapter sums the context holds room for
constexpr int DN_RUNS = 4;

struct crf_context {
  crf_model_dims dims;
  int32_t max_tokens = 0, max_rank = 0, rank_pad = 0;
  int device = 0;
  size_t esz = 2;
  // workspace
  float *hres = nullptr;   // [T, d] residual stream, fp32
  void *xn = nullptr;      // [T, d] normalised input
  void *q = nullptr;       // [T, dq] rotated queries
  void *attn = nullptr;    // [T, dq] attention output
  void *act = nullptr;     // [T, f] SwiGLU output
  void *u = nullptr;       // bf16: [T, 3*rank_pad] LoRA down-projections; fp32: [T, max_rank]
  float *proj = nullptr;   // fp32 path: [T, dq + 2 dkv]
  float *gu = nullptr;     // fp32 path: [T, 2f]
  float2 *rope_cs = nullptr;
  int *d_err = nullptr;
  float *proj16 = nullptr;  // bf16 path, <= 16 token rows: fp32 Q/K/V projections [16, dq + 2 dkv]
  float *attn_part = nullptr;  // bf16 path, <= 16 query rows: key-split attention partials
  int64_t attn_part_floats = 0;
  float *lora_part = nullptr;  // bf16 path, <= 16 token rows: K-split LoRA down-projection partials
  int64_t lora_part_floats = 0;
  float *gemm_part = nullptr;  // bf16 path: K-part partials of the last residual GEMM tiles
  int64_t gemm_part_floats = 0;
  float *dn_part = nullptr;    // bf16 path: down-projection adapter sums fused into gate/up
  int *dn_head = nullptr;      //   and the table of their first tiles
  int n_cu = 0;
  // drift staging
  void *drift_host = nullptr;
  size_t drift_host_bytes = 0;
  void *drift_dev = nullptr;
  size_t drift_dev_bytes = 0;
  hipEvent_t drift_ev = nullptr;
  bool drift_ev_recorded = false;
  std::string last_error;
  Timer timer;
  // batched calls over independent caches: a second workspace (a context of
  // the same shape, made by the first such call) and two lane streams forked
  // from the caller's stream
  crf_context *lane2 = nullptr;
  hipStream_t lane_s[2] = {nullptr, nullptr};
  hipEvent_t fork_ev = nullptr, join_ev[2] = {nullptr, nullptr};
};

namespace {

crf_status fail(crf_context *ctx, crf_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (ctx)
    ctx->last_error = buf;
  else
    g_last_error = buf;
  return st;
}

#define HIP_TRY(ctx, expr)                                                                       \
  do {                                                                                           \
    hipError_t e_ = (expr);                                                                      \
    if (e_ != hipSuccess) return fail(ctx, CRF_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int dq_of(const crf_model_dims &d) { return d.n_q_heads * d.head_dim; }
int dkv_of(const crf_model_dims &d) { return d.n_kv_heads * d.head_dim; }

void target_shape(const crf_model_dims &d, int t, int &d_out, int &d_in) {
  const int dq = dq_of(d), dkv = dkv_of(d);
  switch (t) {
    case CRF_Q: d_out = dq; d_in = d.d_model; break;
    case CRF_K: case CRF_V: d_out = dkv; d_in = d.d_model; break;
    case CRF_O: d_out = d.d_model; d_in = dq; break;
    case CRF_GATE: case CRF_UP: d_out = d.d_ffn; d_in = d.d_model; break;
    default: d_out = d.d_model; d_in = d.d_ffn; break;
  }
}

crf_status check_dims(crf_context *ctx, const crf_model_dims *d) {
  if (!d) return fail(ctx, CRF_ERR_INVALID_ARG, "dims is NULL");
  if (d->n_layers <= 0 || d->d_model <= 0 || d->n_q_heads <= 0 || d->n_kv_heads <= 0 || d->head_dim <= 0 ||
      d->d_ffn <= 0)
    return fail(ctx, CRF_ERR_SHAPE, "every model dimension must be positive");
  if (!(d->rms_eps >= 0.f) || !(d->rope_theta > 0.f))
    return fail(ctx, CRF_ERR_SHAPE, "rms_eps must be >= 0 and rope_theta > 0");
  if (d->dtype != CRF_F32 && d->dtype != CRF_BF16) return fail(ctx, CRF_ERR_INVALID_ARG, "unknown dtype %d", d->dtype);
  if (d->n_q_heads % d->n_kv_heads)
    return fail(ctx, CRF_ERR_UNSUPPORTED, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", d->n_q_heads,
                d->n_kv_heads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(ctx, CRF_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", d->head_dim);
  if (d->d_model % 8 || d->d_ffn % 8)
    return fail(ctx, CRF_ERR_UNSUPPORTED, "d_model and d_ffn must be multiples of 8");
  if (d->dtype == CRF_BF16) {
    if (d->d_model % 128 || dq_of(*d) % 128 || dkv_of(*d) % 128 || d->d_ffn % 64)
      return fail(ctx, CRF_ERR_UNSUPPORTED,
                  "bf16 path needs d_model, n_q_heads*head_dim, n_kv_heads*head_dim multiples of 128 and d_ffn a "
                  "multiple of 64");
    // the projection kernels address each weight matrix through one buffer resource
    // (the largest are [d_ffn, d_model] / [d_model, d_ffn] and [dq, d_model] / [d_model, dq])
    if (std::max<int64_t>(d->d_ffn, dq_of(*d)) * d->d_model * 2 >= ((int64_t)1 << 31))
      return fail(ctx, CRF_ERR_UNSUPPORTED, "bf16 path needs every projection weight smaller than 2 GiB");
  }
  return CRF_OK;
}

// bf16 projections read their input [rows, K] through one buffer resource:
// rows * max(d_model, n_q_heads*head_dim, d_ffn) * 2 bytes must stay below 2 GiB.
crf_status check_gemm_rows(crf_context *ctx, const crf_model_dims *d, int64_t rows, const char *what) {
  if (d->dtype != CRF_BF16 || rows <= 16) return CRF_OK;  // up to 16 rows take the weight-streaming kernels
  const int64_t k = std::max<int64_t>(d->d_ffn, std::max<int64_t>(d->d_model, dq_of(*d)));
  if (rows * k * 2 >= ((int64_t)1 << 31))
    return fail(ctx, CRF_ERR_UNSUPPORTED,
                "%s: %lld token rows x %lld features of bf16 projection input reach 2 GiB (at most %lld rows)", what,
                (long long)rows, (long long)k, (long long)((((int64_t)1 << 31) - 1) / (2 * k)));
  return CRF_OK;
}

crf_status check_window(crf_context *ctx, const crf_model_dims *d, int32_t l0, int32_t h, const crf_kv_cache *kv) {
  crf_status st = check_dims(ctx, d);
  if (st != CRF_OK) return st;
  if (l0 < 0 || h < 0 || (int64_t)l0 + h > d->n_layers)
    return fail(ctx, CRF_ERR_RANGE, "window [%d, %d+%d) outside [0, %d)", l0, l0, h, d->n_layers);
  if (!kv) return fail(ctx, CRF_ERR_INVALID_ARG, "kv_cache is NULL");
  if (kv->page_size < 1 || kv->n_pages < 0 || kv->n_tokens < 0)
    return fail(ctx, CRF_ERR_SHAPE, "page_size must be >= 1, n_pages and n_tokens >= 0");
  if ((int64_t)kv->n_tokens > (int64_t)kv->n_pages * kv->page_size)
    return fail(ctx, CRF_ERR_SHAPE, "n_tokens %d exceeds n_pages*page_size = %lld", kv->n_tokens,
                (long long)kv->n_pages * kv->page_size);
  if (kv->page_stride < (int64_t)d->n_kv_heads * kv->page_size * d->head_dim)
    return fail(ctx, CRF_ERR_SHAPE, "page_stride %lld < n_kv_heads*page_size*head_dim", (long long)kv->page_stride);
  if (kv->layer_stride < (int64_t)kv->n_pages * kv->page_stride)
    return fail(ctx, CRF_ERR_SHAPE, "layer_stride %lld < n_pages*page_stride", (long long)kv->layer_stride);
  if ((int64_t)kv->n_pages * kv->page_stride * (d->dtype == CRF_BF16 ? 2 : 4) >= ((int64_t)1 << 31))
    return fail(ctx, CRF_ERR_UNSUPPORTED, "one layer of the KV pool must be smaller than 2 GiB");
  if (h > 0 && kv->n_tokens > 0 && (!kv->k_pool || !kv->v_pool || !kv->block_table))
    return fail(ctx, CRF_ERR_INVALID_ARG, "k_pool, v_pool and block_table must be non-NULL");
  return CRF_OK;
}

bool same_dims(const crf_model_dims &a, const crf_model_dims &b) {
  return a.n_layers == b.n_layers && a.d_model == b.d_model && a.n_q_heads == b.n_q_heads &&
         a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim && a.d_ffn == b.d_ffn && a.rms_eps == b.rms_eps &&
         a.rope_theta == b.rope_theta && a.dtype == b.dtype;
}

// Full validation of one window request against a context (host only).
// gemm_rows: token rows the projections run over (the window's n_tokens, or a
// decoding step's new tokens).
crf_status check_request(crf_context *ctx, const crf_model_dims *dims, const void *hb,
                         const crf_layer_weights *w, const crf_lora_layer *lora, int32_t l0, int32_t h,
                         const crf_kv_cache *kv, const void *hout, const char *what, int64_t gemm_rows) {
  crf_status st = check_window(ctx, dims, l0, h, kv);
  if (st != CRF_OK) return st;
  if (h > 0 && (st = check_gemm_rows(ctx, dims, gemm_rows, what)) != CRF_OK) return st;
  if (!same_dims(*dims, ctx->dims)) return fail(ctx, CRF_ERR_INVALID_ARG, "%s: dims differ from the context's", what);
  if (h == 0 || kv->n_tokens == 0) return CRF_OK;
  if (kv->n_tokens > ctx->max_tokens)
    return fail(ctx, CRF_ERR_WORKSPACE, "%s: n_tokens %d exceeds the context's max_tokens %d", what, kv->n_tokens,
                ctx->max_tokens);
  if (!hb || !aligned16(hb)) return fail(ctx, CRF_ERR_INVALID_ARG, "%s: hidden_at_boundary NULL or misaligned", what);
  if (hout && !aligned16(hout)) return fail(ctx, CRF_ERR_INVALID_ARG, "%s: hidden_out misaligned", what);
  if (!aligned16(kv->k_pool) || !aligned16(kv->v_pool) || kv->page_stride % 8 || kv->layer_stride % 8)
    return fail(ctx, CRF_ERR_INVALID_ARG, "%s: KV pools must be 16-byte aligned with strides multiple of 8", what);
  if (!w) return fail(ctx, CRF_ERR_INVALID_ARG, "%s: base_weights is NULL", what);
  for (int l = l0; l < l0 + h; ++l) {
    const crf_layer_weights &lw = w[l];
    if (!lw.attn_norm || !lw.mlp_norm || !aligned16(lw.attn_norm) || !aligned16(lw.mlp_norm))
      return fail(ctx, CRF_ERR_INVALID_ARG, "%s: layer %d norm gains NULL or misaligned", what, l);
    for (int t = 0; t < CRF_NUM_TARGETS; ++t)
      if (!lw.w[t] || !aligned16(lw.w[t]))
        return fail(ctx, CRF_ERR_INVALID_ARG, "%s: layer %d weight %d NULL or misaligned", what, l, t);
    if (lora) {
      const crf_lora_layer &ll = lora[l];
      if (ll.rank < 0) return fail(ctx, CRF_ERR_INVALID_ARG, "%s: layer %d negative LoRA rank", what, l);
      if (ll.rank > ctx->max_rank)
        return fail(ctx, CRF_ERR_WORKSPACE, "%s: layer %d LoRA rank %d exceeds the context's %d", what, l, ll.rank,
                    ctx->max_rank);
      if (ll.rank > 0 && ctx->dims.dtype == CRF_BF16 && ll.rank % 8)
        return fail(ctx, CRF_ERR_UNSUPPORTED, "%s: bf16 path needs LoRA rank multiple of 8 (got %d)", what, ll.rank);
      for (int t = 0; t < CRF_NUM_TARGETS && ll.rank > 0; ++t) {
        if ((ll.A[t] == nullptr) != (ll.B[t] == nullptr))
          return fail(ctx, CRF_ERR_INVALID_ARG, "%s: layer %d target %d has only one LoRA factor", what, l, t);
        if (ll.A[t] && (!aligned16(ll.A[t]) || !aligned16(ll.B[t])))
          return fail(ctx, CRF_ERR_INVALID_ARG, "%s: layer %d target %d LoRA factor misaligned", what, l, t);
      }
    }
  }
  return CRF_OK;
}

// ----------------------------------------------------------------------------- timing

struct Launch {
  crf_context *ctx;
  hipStream_t s;
  int kind;
  size_t idx = 0;
  bool on;
  Launch(crf_context *c, hipStream_t st, int k) : ctx(c), s(st), kind(k), on(((c->timer.mask >> k) & 1u) != 0) {
    Timer &t = ctx->timer;
    if (!on) return;
    idx = t.used;
    if (2 * idx + 2 > t.ev.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return;
      t.ev.push_back(a);
      t.ev.push_back(b);
      t.kind.push_back(k);
    }
    t.kind[idx] = k;
    (void)hipEventRecord(t.ev[2 * idx], s);
  }
  ~Launch() {
    Timer &t = ctx->timer;
    if (!on || 2 * idx + 2 > t.ev.size()) return;
    (void)hipEventRecord(t.ev[2 * idx + 1], s);
    t.used = idx + 1;
  }
};

#define LAUNCH(ctx, s, kind, expr)                                                                     \
  do {                                                                                                 \
    Launch lt_(ctx, s, kind);                                                                          \
    hipError_t e_ = (expr);                                                                            \
    if (e_ != hipSuccess) return fail(ctx, CRF_ERR_HIP, "launch %s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// ----------------------------------------------------------------------------- layer sequences

PagedKV layer_kv(crf_context *ctx, const crf_kv_cache *kv, int l) {
  PagedKV p;
  p.k = (char *)kv->k_pool + (size_t)l * kv->layer_stride * ctx->esz;
  p.v = (char *)kv->v_pool + (size_t)l * kv->layer_stride * ctx->esz;
  p.page_stride = kv->page_stride;
  p.block_table = kv->block_table;
  p.n_pages = kv->n_pages;
  p.page_size = kv->page_size;
  p.n_tokens = kv->n_tokens;
  p.err = ctx->d_err;
  return p;
}

bool has_lora(const crf_lora_layer *lora, int l, int t) {
  return lora && lora[l].rank > 0 && lora[l].A[t] != nullptr;
}

// Layers [l0, l0+h) over `rows` token rows at positions pos0..pos0+rows-1: a
// window (pos0 = 0, rows = the prefix) or new tokens over a cached prefix
// (pos0 = the prefix length).  kv_tail: without hidden_out the last layer runs
// its K/V projections only.
crf_status run_layers_bf16(crf_context *ctx, const void *hb, const crf_layer_weights *W,
                           const crf_lora_layer *lora, int l0, int h, const crf_kv_cache *kv, void *hout,
                           hipStream_t s, int rows, int pos0, bool kv_tail) {
  const crf_model_dims &d = ctx->dims;
  const int M = rows, D = d.d_model, dq = dq_of(d), dkv = dkv_of(d), f = d.d_ffn, hd = d.head_dim;
  const int rp = ctx->rank_pad, ldu = 3 * rp;
  bf16 *xn = (bf16 *)ctx->xn, *q = (bf16 *)ctx->q, *attn = (bf16 *)ctx->attn, *act = (bf16 *)ctx->act;
  bf16 *u = (bf16 *)ctx->u;
  for (int l = l0; l < l0 + h; ++l) {
    const crf_layer_weights &w = W[l];
    const bool first = l == l0, last = l == l0 + h - 1;
    const int rank = lora ? lora[l].rank : 0;
    const float scale = lora ? lora[l].scale : 0.f;
    auto lora_targets = [&](std::initializer_list<int> ts, LoraDownTarget *out) {
      int i = 0;
      bool any = false;
      for (int t : ts) {
        const bool on = has_lora(lora, l, t);
        out[i] = LoraDownTarget{on ? (const bf16 *)lora[l].A[t] : nullptr, rank, scale, i * rp};
        any |= on;
        ++i;
      }
      return any;
    };
    auto base_params = [&](const bf16 *X, int K, int N) {
      GemmParams p{};
      p.X = X;
      p.ldx = K;
      p.M = M;
      p.K = K;
      p.N = N;
      p.U = nullptr;
      p.ldu = ldu;
      p.kpad = rp;
      p.rank = rank;
      p.rope_cs = ctx->rope_cs;
      p.q_scale = attn_query_scale(hd);
      p.pos0 = pos0;
      p.split_part = ctx->gemm_part;
      p.split_cap = ctx->gemm_part_floats;
      p.n_cu = ctx->n_cu;
      return p;
    };
    LoraDownTarget tg[3];
    // a few token rows (a decoding step, a very short window): weight-streaming kernels
    const bool skinny = M <= 16;
    LoraSplit lsplit;  // set by the last LoRA down-projection
    auto gemm = [&](GemmEpi epi, GemmParams &p) {
      if (!skinny) return launch_gemm_bf16(s, epi, hd, p);
      p.proj = ctx->proj16;
      if (p.U && lsplit.n_parts > 0) {  // U still as K-split partials: the projection sums them
        p.upart = ctx->lora_part;
        p.upart_n = lsplit.n_parts;
        p.upart_cols = lsplit.cols;
        p.uscale = scale;
      }
      return launch_gemm_skinny_bf16(s, epi, hd, p);
    };

    // attention block
    // the window's first O projection reads the bf16 boundary state as its old
    // residual (the weight-streaming kernels of a few rows read the fp32 copy)
    const bool resid_from_boundary = first && !skinny;
    LAUNCH(ctx, s, CRF_KK_NORM,
           launch_rmsnorm(s, first ? hb : (const void *)ctx->hres, !first, w.attn_norm, false, xn, false,
                          first && !resid_from_boundary ? ctx->hres : nullptr, M, D, d.rms_eps));
    if (last && !hout && kv_tail) {
      // Nothing reads this layer's output: its cache entry depends only on its
      // input through the K and V projections, so only those run.
      const bool kv_any = lora_targets({CRF_K, CRF_V}, tg);
      if (kv_any) LAUNCH(ctx, s, CRF_KK_LORA_DOWN, launch_lora_down_bf16(s, xn, D, M, D, tg, 2, rp, u, ldu, ctx->lora_part, ctx->lora_part_floats, &lsplit));
      GemmParams p = base_params(xn, D, 2 * dkv);
      p.w[1] = (const bf16 *)w.w[CRF_K];
      p.w[2] = (const bf16 *)w.w[CRF_V];
      p.seg1 = 0;  // no query rows: [0, dkv) K, [dkv, 2 dkv) V
      p.seg2 = dkv;
      if (kv_any) {
        p.U = u;
        for (int i = 1; i < 3; ++i) {
          const int t = CRF_Q + i;
          p.lb[i] = has_lora(lora, l, t) ? (const bf16 *)lora[l].B[t] : nullptr;
          p.ucol[i] = (i - 1) * rp;
        }
      }
      p.bias[1] = (const bf16 *)w.bias_k;
      p.bias[2] = (const bf16 *)w.bias_v;
      p.dq = dq;
      p.kv = layer_kv(ctx, kv, l);
      LAUNCH(ctx, s, CRF_KK_GEMM_QKV, gemm(EPI_QKV, p));
      break;
    }
    bool any = lora_targets({CRF_Q, CRF_K, CRF_V}, tg);
    if (any) LAUNCH(ctx, s, CRF_KK_LORA_DOWN, launch_lora_down_bf16(s, xn, D, M, D, tg, 3, rp, u, ldu, ctx->lora_part, ctx->lora_part_floats, &lsplit));
    {
      GemmParams p = base_params(xn, D, dq + 2 * dkv);
      p.w[0] = (const bf16 *)w.w[CRF_Q];
      p.w[1] = (const bf16 *)w.w[CRF_K];
      p.w[2] = (const bf16 *)w.w[CRF_V];
      p.seg1 = dq;
      p.seg2 = dq + dkv;
      if (any) {
        p.U = u;
        for (int i = 0; i < 3; ++i) {
          const int t = CRF_Q + i;
          p.lb[i] = has_lora(lora, l, t) ? (const bf16 *)lora[l].B[t] : nullptr;
          p.ucol[i] = i * rp;
        }
      }
      p.bias[0] = (const bf16 *)w.bias_q;
      p.bias[1] = (const bf16 *)w.bias_k;
      p.bias[2] = (const bf16 *)w.bias_v;
      p.q_out = q;
      p.dq = dq;
      p.kv = layer_kv(ctx, kv, l);
      LAUNCH(ctx, s, CRF_KK_GEMM_QKV, gemm(EPI_QKV, p));
    }
    LAUNCH(ctx, s, CRF_KK_ATTN,
           launch_attn_bf16(s, q, layer_kv(ctx, kv, l), attn, M, pos0, d.n_q_heads, d.n_kv_heads, hd,
                            ctx->attn_part, ctx->attn_part_floats));
    any = lora_targets({CRF_O}, tg);
    if (any) LAUNCH(ctx, s, CRF_KK_LORA_DOWN, launch_lora_down_bf16(s, attn, dq, M, dq, tg, 1, rp, u, ldu, ctx->lora_part, ctx->lora_part_floats, &lsplit));
    {
      GemmParams p = base_params(attn, dq, D);
      p.w[0] = (const bf16 *)w.w[CRF_O];
      if (any) {
        p.U = u;
        p.lb[0] = (const bf16 *)lora[l].B[CRF_O];
        p.ucol[0] = 0;
      }
      p.resid = ctx->hres;
      p.resid_in = resid_from_boundary ? (const bf16 *)hb : nullptr;
      p.ldr = D;
      LAUNCH(ctx, s, CRF_KK_GEMM_O, gemm(EPI_RESID, p));
    }
    // MLP block
    LAUNCH(ctx, s, CRF_KK_NORM,
           launch_rmsnorm(s, ctx->hres, true, w.mlp_norm, false, xn, false, nullptr, M, D, d.rms_eps));
    any = lora_targets({CRF_GATE, CRF_UP}, tg);
    if (any) LAUNCH(ctx, s, CRF_KK_LORA_DOWN, launch_lora_down_bf16(s, xn, D, M, D, tg, 2, rp, u, ldu, ctx->lora_part, ctx->lora_part_floats, &lsplit));
    // the down projection's adapter down-projection rides on the gate/up
    // epilogue when its rank fits (dn_done), else it is a pass of its own
    bool dn_done = false;
    GemmParams pgu = base_params(xn, D, 2 * f);
    {
      GemmParams &p = pgu;
      p.w[0] = (const bf16 *)w.w[CRF_GATE];
      p.w[1] = (const bf16 *)w.w[CRF_UP];
      if (any) {
        p.U = u;
        p.lb[0] = has_lora(lora, l, CRF_GATE) ? (const bf16 *)lora[l].B[CRF_GATE] : nullptr;
        p.lb[1] = has_lora(lora, l, CRF_UP) ? (const bf16 *)lora[l].B[CRF_UP] : nullptr;
        p.ucol[0] = 0;
        p.ucol[1] = rp;
      }
      p.act = act;
      p.d_ffn = f;
      if (!skinny && has_lora(lora, l, CRF_DOWN) && rank <= 16 && ctx->dn_part) {
        p.dn_a = (const bf16 *)lora[l].A[CRF_DOWN];
        p.dn_rank = rank;
        p.dn_part = ctx->dn_part;
        p.dn_head = ctx->dn_head;
        p.dn_runs = DN_RUNS;
      }
      LAUNCH(ctx, s, CRF_KK_GEMM_GATEUP, skinny ? gemm(EPI_SWIGLU, p) : launch_gemm_bf16(s, EPI_SWIGLU, hd, p, &dn_done));
    }
    any = lora_targets({CRF_DOWN}, tg);
    if (any && dn_done)
      LAUNCH(ctx, s, CRF_KK_LORA_DOWN, launch_gemm_dn_sum(s, pgu, u, ldu, 0, scale));
    else if (any)
      LAUNCH(ctx, s, CRF_KK_LORA_DOWN, launch_lora_down_bf16(s, act, f, M, f, tg, 1, rp, u, ldu, ctx->lora_part, ctx->lora_part_floats, &lsplit));
    {
      GemmParams p = base_params(act, f, D);
      p.w[0] = (const bf16 *)w.w[CRF_DOWN];
      if (any) {
        p.U = u;
        p.lb[0] = (const bf16 *)lora[l].B[CRF_DOWN];
        p.ucol[0] = 0;
      }
      p.resid = ctx->hres;
      p.resid_out = (last && hout) ? (bf16 *)hout : nullptr;
      p.resid_final = p.resid_out && !skinny;  // nothing reads the fp32 residual after the window
      p.ldr = D;
      LAUNCH(ctx, s, CRF_KK_GEMM_DOWN, gemm(EPI_RESID, p));
    }
  }
  return CRF_OK;
}

crf_status run_layers_f32(crf_context *ctx, const void *hb, const crf_layer_weights *W, const crf_lora_layer *lora,
                          int l0, int h, const crf_kv_cache *kv, void *hout, hipStream_t s) {
  const crf_model_dims &d = ctx->dims;
  const int M = kv->n_tokens, D = d.d_model, dq = dq_of(d), dkv = dkv_of(d), f = d.d_ffn, hd = d.head_dim;
  const int PW = dq + 2 * dkv;
  float *xn = (float *)ctx->xn, *q = (float *)ctx->q, *attn = (float *)ctx->attn, *act = (float *)ctx->act;
  float *u = (float *)ctx->u;
  // y[:, :] (ldc) += x W^T (+ scale (x A^T) B^T)
  auto proj = [&](int l, int t, const float *x, int K, float *y, int ldc, float beta) -> crf_status {
    int d_out, d_in;
    target_shape(d, t, d_out, d_in);
    const int kind = t <= CRF_V ? CRF_KK_GEMM_QKV
                   : t == CRF_O ? CRF_KK_GEMM_O
                   : t == CRF_DOWN ? CRF_KK_GEMM_DOWN : CRF_KK_GEMM_GATEUP;
    LAUNCH(ctx, s, kind, launch_gemm_f32(s, M, d_out, K, x, K, (const float *)W[l].w[t], K, y, ldc, 1.f, beta));
    if (has_lora(lora, l, t)) {
      const int r = lora[l].rank;
      LAUNCH(ctx, s, CRF_KK_LORA_DOWN,
             launch_gemm_f32(s, M, r, K, x, K, (const float *)lora[l].A[t], K, u, r, lora[l].scale, 0.f));
      LAUNCH(ctx, s, kind, launch_gemm_f32(s, M, d_out, r, u, r, (const float *)lora[l].B[t], r, y, ldc, 1.f, 1.f));
    }
    return CRF_OK;
  };
  crf_status st;
  for (int l = l0; l < l0 + h; ++l) {
    const crf_layer_weights &w = W[l];
    const bool first = l == l0;
    LAUNCH(ctx, s, CRF_KK_NORM,
           launch_rmsnorm(s, first ? hb : (const void *)ctx->hres, true, w.attn_norm, true, xn, true,
                          first ? ctx->hres : nullptr, M, D, d.rms_eps));
    if ((st = proj(l, CRF_Q, xn, D, ctx->proj, PW, 0.f)) != CRF_OK) return st;
    if ((st = proj(l, CRF_K, xn, D, ctx->proj + dq, PW, 0.f)) != CRF_OK) return st;
    if ((st = proj(l, CRF_V, xn, D, ctx->proj + dq + dkv, PW, 0.f)) != CRF_OK) return st;
    const PagedKV pk = layer_kv(ctx, kv, l);
    LAUNCH(ctx, s, CRF_KK_OTHER,
           launch_qkv_post_f32(s, ctx->proj, (const float *)w.bias_q, (const float *)w.bias_k,
                               (const float *)w.bias_v, q, pk, ctx->rope_cs, M, d.n_q_heads, d.n_kv_heads, hd));
    LAUNCH(ctx, s, CRF_KK_ATTN, launch_attn_f32(s, q, pk, attn, M, d.n_q_heads, d.n_kv_heads, hd));
    if ((st = proj(l, CRF_O, attn, dq, ctx->hres, D, 1.f)) != CRF_OK) return st;
    LAUNCH(ctx, s, CRF_KK_NORM,
           launch_rmsnorm(s, ctx->hres, true, w.mlp_norm, true, xn, true, nullptr, M, D, d.rms_eps));
    if ((st = proj(l, CRF_GATE, xn, D, ctx->gu, 2 * f, 0.f)) != CRF_OK) return st;
    if ((st = proj(l, CRF_UP, xn, D, ctx->gu + f, 2 * f, 0.f)) != CRF_OK) return st;
    LAUNCH(ctx, s, CRF_KK_OTHER, launch_silu_mul_f32(s, ctx->gu, act, M, f));
    if ((st = proj(l, CRF_DOWN, act, f, ctx->hres, D, 1.f)) != CRF_OK) return st;
  }
  if (hout) HIP_TRY(ctx, hipMemcpyAsync(hout, ctx->hres, (size_t)M * D * sizeof(float), hipMemcpyDeviceToDevice, s));
  return CRF_OK;
}

crf_status run_window(crf_context *ctx, const void *hb, const crf_layer_weights *W, const crf_lora_layer *lora,
                      int l0, int h, const crf_kv_cache *kv, void *hout, hipStream_t s) {
  if (h == 0 || kv->n_tokens == 0) return CRF_OK;
  if (ctx->dims.dtype == CRF_BF16) return run_layers_bf16(ctx, hb, W, lora, l0, h, kv, hout, s, kv->n_tokens, 0, true);
  return run_layers_f32(ctx, hb, W, lora, l0, h, kv, hout, s);
}

template <typename T>
crf_status dmalloc(crf_context *ctx, T **p, size_t bytes) {
  void *q = nullptr;
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(&q, bytes);
  if (e != hipSuccess) return fail(ctx, CRF_ERR_HIP, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
  *p = (T *)q;
  return CRF_OK;
}

}  // namespace

namespace {

// Drift tables: segments (one per current/version factor pair), chunks of at
// most 2^16 elements, and per (version, layer) the first chunk and the chunk
// count.  Staging layout: segs | chunks | first | count | anchor, copied from
// the host, then partials (double, one per chunk) and scratch (double, one per
// (version, layer)) written by the kernels.
constexpr int64_t DRIFT_CHUNK = 1 << 16;

struct DriftPlan {
  int L = 0, V = 0;
  size_t n_segs = 0, n_chunks = 0;
  size_t o_segs = 0, o_chunks = 0, o_first = 0, o_count = 0, o_anchor = 0, host_bytes = 0, o_part = 0, o_scr = 0,
         dev_bytes = 0;
};

// Validates a drift request and sizes its tables (touches no device).
crf_status drift_plan(crf_context *ctx, const crf_model_dims *dims, const crf_lora_layer *current, int32_t n_versions,
                      const crf_lora_layer *const *versions, const int32_t *anchor_version, const float *drift_out,
                      const float *risk_out, DriftPlan &pl) {
  if (!current || !versions || !anchor_version || !drift_out || !risk_out || n_versions < 1)
    return fail(ctx, CRF_ERR_INVALID_ARG, "NULL argument or n_versions < 1");
  const int L = dims->n_layers;
  for (int l = 0; l < L; ++l)
    if (anchor_version[l] < 0 || anchor_version[l] >= n_versions)
      return fail(ctx, CRF_ERR_INVALID_ARG, "anchor_version[%d] = %d outside [0, %d)", l, anchor_version[l],
                  n_versions);
  pl = DriftPlan{};
  pl.L = L;
  pl.V = n_versions;
  for (int v = 0; v < n_versions; ++v) {
    if (!versions[v]) return fail(ctx, CRF_ERR_INVALID_ARG, "versions[%d] is NULL", v);
    for (int l = 0; l < L; ++l) {
      const crf_lora_layer &c = current[l], &vv = versions[v][l];
      for (int t = 0; t < CRF_NUM_TARGETS && c.rank > 0; ++t) {
        if (!c.A[t]) continue;
        if (!c.B[t] || !vv.A[t] || !vv.B[t] || vv.rank != c.rank)
          return fail(ctx, CRF_ERR_INVALID_ARG, "layer %d target %d missing or rank differs in version %d", l, t, v);
        int d_out, d_in;
        target_shape(*dims, t, d_out, d_in);
        const int64_t cnt[2] = {(int64_t)c.rank * d_in, (int64_t)d_out * c.rank};
        for (int k = 0; k < 2; ++k) {
          ++pl.n_segs;
          pl.n_chunks += (size_t)((cnt[k] + DRIFT_CHUNK - 1) / DRIFT_CHUNK);
        }
      }
    }
  }
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t n_out = (size_t)n_versions * L;
  pl.o_segs = 0;
  pl.o_chunks = al(pl.o_segs + pl.n_segs * sizeof(DriftSeg));
  pl.o_first = al(pl.o_chunks + pl.n_chunks * sizeof(DriftChunk));
  pl.o_count = al(pl.o_first + n_out * sizeof(int));
  pl.o_anchor = al(pl.o_count + n_out * sizeof(int));
  pl.host_bytes = al(pl.o_anchor + L * sizeof(int));
  pl.o_part = pl.host_bytes;
  pl.o_scr = al(pl.o_part + (pl.n_chunks + 1) * sizeof(double));
  pl.dev_bytes = al(pl.o_scr + n_out * sizeof(double));
  return CRF_OK;
}

// Writes the tables of a planned request into host staging hb (host_bytes).
void drift_fill(const DriftPlan &pl, const crf_model_dims *dims, const crf_lora_layer *current,
                const crf_lora_layer *const *versions, const int32_t *anchor_version, char *hb) {
  DriftSeg *segs = (DriftSeg *)(hb + pl.o_segs);
  DriftChunk *chunks = (DriftChunk *)(hb + pl.o_chunks);
  int *first = (int *)(hb + pl.o_first), *count = (int *)(hb + pl.o_count);
  int ns = 0, nc = 0;
  for (int v = 0; v < pl.V; ++v)
    for (int l = 0; l < pl.L; ++l) {
      const int o = v * pl.L + l;
      first[o] = nc;
      const crf_lora_layer &c = current[l], &vv = versions[v][l];
      for (int t = 0; t < CRF_NUM_TARGETS && c.rank > 0; ++t) {
        if (!c.A[t]) continue;
        int d_out, d_in;
        target_shape(*dims, t, d_out, d_in);
        const int64_t cnt[2] = {(int64_t)c.rank * d_in, (int64_t)d_out * c.rank};
        const void *pa[2] = {c.A[t], c.B[t]}, *pb[2] = {vv.A[t], vv.B[t]};
        for (int k = 0; k < 2; ++k) {
          const int si = ns++;
          segs[si] = DriftSeg{pa[k], pb[k], cnt[k], o};
          for (int64_t s0 = 0; s0 < cnt[k]; s0 += DRIFT_CHUNK)
            chunks[nc++] = DriftChunk{si, s0, std::min(DRIFT_CHUNK, cnt[k] - s0)};
        }
      }
      count[o] = nc - first[o];
    }
  memcpy(hb + pl.o_anchor, anchor_version, pl.L * sizeof(int));
}

// The two drift kernels over staging db (tables already there).
hipError_t drift_launch(hipStream_t s, const DriftPlan &pl, char *db, bool f32, const float *sensitivity,
                        int32_t per_layer_only, float *drift_out, float *risk_out, float *sq_partial_out) {
  hipError_t e = launch_drift_partials(s, (const DriftSeg *)(db + pl.o_segs), (const DriftChunk *)(db + pl.o_chunks),
                                       (int)pl.n_chunks, f32, (double *)(db + pl.o_part));
  if (e != hipSuccess) return e;
  return launch_drift_finalize(s, (const double *)(db + pl.o_part), (const int *)(db + pl.o_first),
                               (const int *)(db + pl.o_count), pl.V, pl.L, (const int *)(db + pl.o_anchor),
                               sensitivity, per_layer_only, drift_out, risk_out, sq_partial_out,
                               (double *)(db + pl.o_scr));
}

}  // namespace

extern "C" {

const char *crf_status_string(crf_status s) {
  switch (s) {
    case CRF_OK: return "CRF_OK";
    case CRF_ERR_INVALID_ARG: return "CRF_ERR_INVALID_ARG";
    case CRF_ERR_SHAPE: return "CRF_ERR_SHAPE";
    case CRF_ERR_RANGE: return "CRF_ERR_RANGE";
    case CRF_ERR_UNSUPPORTED: return "CRF_ERR_UNSUPPORTED";
    case CRF_ERR_WORKSPACE: return "CRF_ERR_WORKSPACE";
    case CRF_ERR_HIP: return "CRF_ERR_HIP";
    case CRF_ERR_DEVICE: return "CRF_ERR_DEVICE";
  }
  return "CRF_ERR_UNKNOWN";
}

int32_t crf_abi_version(void) { return CRF_ABI_VERSION; }

const char *crf_last_error(const crf_context *ctx) { return ctx ? ctx->last_error.c_str() : g_last_error.c_str(); }

crf_status crf_validate_dims(const crf_model_dims *dims) { return check_dims(nullptr, dims); }

crf_status crf_validate_window(const crf_model_dims *dims, int32_t l0, int32_t h, const crf_kv_cache *kv) {
  crf_status st = check_window(nullptr, dims, l0, h, kv);
  if (st == CRF_OK && h > 0) st = check_gemm_rows(nullptr, dims, kv->n_tokens, "crf_validate_window");
  return st;
}

void crf_context_destroy(crf_context *ctx) {
  if (!ctx) return;
  void *bufs[] = {ctx->hres, ctx->xn, ctx->q, ctx->attn, ctx->act, ctx->u, ctx->proj, ctx->gu, ctx->rope_cs,
                  ctx->d_err, ctx->drift_dev, ctx->proj16, ctx->attn_part, ctx->lora_part, ctx->gemm_part,
                  ctx->dn_part, ctx->dn_head};
  for (void *b : bufs)
    if (b) (void)hipFree(b);
  if (ctx->drift_host) (void)hipHostFree(ctx->drift_host);
  if (ctx->drift_ev) (void)hipEventDestroy(ctx->drift_ev);
  for (hipEvent_t e : ctx->timer.ev) (void)hipEventDestroy(e);
  for (int i = 0; i < 2; ++i) {
    if (ctx->lane_s[i]) (void)hipStreamDestroy(ctx->lane_s[i]);
    if (ctx->join_ev[i]) (void)hipEventDestroy(ctx->join_ev[i]);
  }
  if (ctx->fork_ev) (void)hipEventDestroy(ctx->fork_ev);
  crf_context_destroy(ctx->lane2);
  delete ctx;
}

crf_status crf_context_create(const crf_model_dims *dims, int32_t max_tokens, int32_t max_lora_rank,
                              crf_context **out) {
  if (!out) return fail(nullptr, CRF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  crf_status st = check_dims(nullptr, dims);
  if (st != CRF_OK) return st;
  if (max_tokens < 1) return fail(nullptr, CRF_ERR_SHAPE, "max_tokens must be >= 1");
  if (max_lora_rank < 0 || max_lora_rank > 64) return fail(nullptr, CRF_ERR_UNSUPPORTED, "max_lora_rank must be in [0, 64]");
  crf_context *ctx = new crf_context();
  ctx->dims = *dims;
  ctx->max_tokens = max_tokens;
  ctx->max_rank = max_lora_rank;
  ctx->rank_pad = ((max_lora_rank + 15) / 16) * 16;
  ctx->esz = dims->dtype == CRF_BF16 ? 2 : 4;
  (void)hipGetDevice(&ctx->device);
  const size_t T = (size_t)max_tokens, D = dims->d_model, dq = dq_of(*dims), dkv = dkv_of(*dims), f = dims->d_ffn;
  const size_t e = ctx->esz;
  auto cleanup = [&](crf_status s) {
    if (s != CRF_OK) {
      g_last_error = ctx->last_error;
      crf_context_destroy(ctx);
    }
    return s;
  };
  if ((st = dmalloc(ctx, &ctx->hres, T * D * 4)) != CRF_OK) return cleanup(st);
  if ((st = dmalloc(ctx, &ctx->xn, T * D * e)) != CRF_OK) return cleanup(st);
  if ((st = dmalloc(ctx, &ctx->q, T * dq * e)) != CRF_OK) return cleanup(st);
  if ((st = dmalloc(ctx, &ctx->attn, T * dq * e)) != CRF_OK) return cleanup(st);
  if ((st = dmalloc(ctx, &ctx->act, T * f * e)) != CRF_OK) return cleanup(st);
  if (dims->dtype == CRF_BF16) {
    if ((st = dmalloc(ctx, &ctx->u, T * 3 * ctx->rank_pad * 2)) != CRF_OK) return cleanup(st);
    if ((st = dmalloc(ctx, &ctx->proj16, 16 * (dq + 2 * dkv) * 4)) != CRF_OK) return cleanup(st);
    // key splits of >= 64 keys, up to 16 query rows per head, rows of hd + 4 floats
    ctx->attn_part_floats = (int64_t)((T + 63) / 64) * dims->n_q_heads * 16 * (dims->head_dim + 4);
    if ((st = dmalloc(ctx, &ctx->attn_part, (size_t)ctx->attn_part_floats * 4)) != CRF_OK) return cleanup(st);
    // K splits of >= 256 for up to 16 rows and three targets
    ctx->lora_part_floats = (int64_t)((std::max({D, f, dq}) + 255) / 256) * 16 * 3 * ctx->rank_pad;
    if ((st = dmalloc(ctx, &ctx->lora_part, (size_t)ctx->lora_part_floats * 4)) != CRF_OK) return cleanup(st);
    // at most one 256x256 fp32 partial per compute unit
    if (hipDeviceGetAttribute(&ctx->n_cu, hipDeviceAttributeMultiprocessorCount, ctx->device) != hipSuccess)
      ctx->n_cu = 0;
    ctx->gemm_part_floats = (int64_t)std::max(ctx->n_cu, 0) * 256 * 256;
    if (ctx->gemm_part_floats > 0 &&
        (st = dmalloc(ctx, &ctx->gemm_part, (size_t)ctx->gemm_part_floats * 4)) != CRF_OK)
      return cleanup(st);
    // fused down-projection adapter sums: DN_RUNS runs of [2][256][16] per
    // compute unit, and one table entry per gate/up tile
    if (ctx->n_cu > 0 && max_lora_rank > 0) {
      if ((st = dmalloc(ctx, &ctx->dn_part, (size_t)ctx->n_cu * DN_RUNS * 2 * 256 * 16 * 4)) != CRF_OK)
        return cleanup(st);
      if ((st = dmalloc(ctx, &ctx->dn_head, ((T + 255) / 256) * ((2 * f + 255) / 256) * sizeof(int))) != CRF_OK)
        return cleanup(st);
    }
  } else {
    if ((st = dmalloc(ctx, &ctx->u, T * (size_t)(max_lora_rank > 0 ? max_lora_rank : 1) * 4)) != CRF_OK)
      return cleanup(st);
    if ((st = dmalloc(ctx, &ctx->proj, T * (dq + 2 * dkv) * 4)) != CRF_OK) return cleanup(st);
    if ((st = dmalloc(ctx, &ctx->gu, T * 2 * f * 4)) != CRF_OK) return cleanup(st);
  }
  if ((st = dmalloc(ctx, &ctx->rope_cs, T * (dims->head_dim / 2) * sizeof(float2))) != CRF_OK) return cleanup(st);
  if ((st = dmalloc(ctx, &ctx->d_err, sizeof(int))) != CRF_OK) return cleanup(st);
  hipError_t he = hipMemset(ctx->d_err, 0, sizeof(int));
  if (he == hipSuccess) he = launch_rope_table(nullptr, ctx->rope_cs, max_tokens, dims->head_dim, dims->rope_theta);
  if (he == hipSuccess) he = hipDeviceSynchronize();
  if (he != hipSuccess) return cleanup(fail(ctx, CRF_ERR_HIP, "context init: %s", hipGetErrorString(he)));
  *out = ctx;
  return CRF_OK;
}

crf_status crf_recompute_window(crf_context *ctx, const crf_model_dims *dims, const void *hidden_at_boundary,
                                const crf_layer_weights *base_weights, const crf_lora_layer *lora, int32_t l0,
                                int32_t h, const crf_kv_cache *kv_cache, void *hidden_out, void *stream) {
  if (!ctx) return fail(nullptr, CRF_ERR_INVALID_ARG, "context is NULL");
  crf_status st = check_request(ctx, dims, hidden_at_boundary, base_weights, lora, l0, h, kv_cache, hidden_out,
                                "crf_recompute_window", kv_cache ? kv_cache->n_tokens : 0);
  if (st != CRF_OK) return st;
  return run_window(ctx, hidden_at_boundary, base_weights, lora, l0, h, kv_cache, hidden_out, (hipStream_t)stream);
}

crf_status crf_recompute_window_batched(crf_context *ctx, const crf_model_dims *dims,
                                        const crf_layer_weights *base_weights, int32_t n_items,
                                        const crf_window_item *items, void *stream) {
  if (!ctx) return fail(nullptr, CRF_ERR_INVALID_ARG, "context is NULL");
  if (n_items < 0 || (n_items > 0 && !items)) return fail(ctx, CRF_ERR_INVALID_ARG, "items NULL or n_items < 0");
  for (int i = 0; i < n_items; ++i) {
    char what[64];
    snprintf(what, sizeof what, "item %d", i);
    const crf_window_item &it = items[i];
    crf_status st = check_request(ctx, dims, it.hidden_at_boundary, base_weights, it.lora, it.l0, it.h, &it.kv,
                                  it.hidden_out, what, it.kv.n_tokens);
    if (st != CRF_OK) return st;
  }
  // Independent items (no item writes a buffer that another reads or writes)
  // run on two lanes, each a stream with its own workspace, so that small
  // windows fill the GPU together; every item's arithmetic is the same either
  // way.  While event timing is on they run in order on `stream`.
  bool lanes = n_items >= 2 && ctx->timer.mask == 0;
  // Byte ranges each item may write (its window's layers of both pools, its
  // output state) and read (the same pool layers, its boundary state, its
  // block table).  Pages are chosen by device-side block tables, so a pool's
  // range spans every page of the window's layers.
  struct Span {
    uintptr_t lo, hi;
  };
  auto overlap = [](Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; };
  std::vector<std::vector<Span>> wr(n_items), rd(n_items);
  for (int i = 0; lanes && i < n_items; ++i) {
    const crf_window_item &it = items[i];
    if (it.h == 0 || it.kv.n_tokens == 0) continue;  // launches nothing
    const size_t esz = ctx->esz;
    const size_t row = (size_t)ctx->dims.d_model * esz * it.kv.n_tokens;
    for (void *pool : {it.kv.k_pool, it.kv.v_pool}) {
      const uintptr_t b = (uintptr_t)pool + (size_t)it.l0 * it.kv.layer_stride * esz;
      const Span sp{b, b + ((size_t)(it.h - 1) * it.kv.layer_stride + (size_t)it.kv.n_pages * it.kv.page_stride) * esz};
      wr[i].push_back(sp);
      rd[i].push_back(sp);
    }
    if (it.hidden_out) wr[i].push_back(Span{(uintptr_t)it.hidden_out, (uintptr_t)it.hidden_out + row});
    rd[i].push_back(Span{(uintptr_t)it.hidden_at_boundary, (uintptr_t)it.hidden_at_boundary + row});
    const size_t bt = ((size_t)it.kv.n_tokens + it.kv.page_size - 1) / it.kv.page_size * sizeof(int32_t);
    rd[i].push_back(Span{(uintptr_t)it.kv.block_table, (uintptr_t)it.kv.block_table + bt});
  }
  for (int i = 0; lanes && i < n_items; ++i)
    for (int j = 0; lanes && j < n_items; ++j) {
      if (i == j) continue;
      for (const Span &w : wr[i]) {
        for (const Span &o : wr[j]) lanes = lanes && !overlap(w, o);
        for (const Span &o : rd[j]) lanes = lanes && !overlap(w, o);
      }
    }
  if (!lanes) {
    for (int i = 0; i < n_items; ++i) {
      const crf_window_item &it = items[i];
      crf_status st = run_window(ctx, it.hidden_at_boundary, base_weights, it.lora, it.l0, it.h, &it.kv,
                                 it.hidden_out, (hipStream_t)stream);
      if (st != CRF_OK) return st;
    }
    return CRF_OK;
  }
  if (!ctx->fork_ev) {  // set last: it marks the lanes complete
    if (!ctx->lane2) {
      crf_context *c2 = nullptr;
      if (crf_context_create(&ctx->dims, ctx->max_tokens, ctx->max_rank, &c2) != CRF_OK)
        return fail(ctx, CRF_ERR_WORKSPACE, "second workspace for concurrent batch items: %s", g_last_error.c_str());
      ctx->lane2 = c2;
    }
    for (int i = 0; i < 2; ++i) {
      if (!ctx->lane_s[i]) HIP_TRY(ctx, hipStreamCreateWithFlags(&ctx->lane_s[i], hipStreamNonBlocking));
      if (!ctx->join_ev[i]) HIP_TRY(ctx, hipEventCreateWithFlags(&ctx->join_ev[i], hipEventDisableTiming));
    }
    HIP_TRY(ctx, hipEventCreateWithFlags(&ctx->fork_ev, hipEventDisableTiming));
  }
  // longest first, each to the lane with less work so far
  std::vector<int> order(n_items);
  for (int i = 0; i < n_items; ++i) order[i] = i;
  auto work = [&](int i) { return (int64_t)items[i].kv.n_tokens * items[i].h; };
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return work(a) > work(b); });
  HIP_TRY(ctx, hipEventRecord(ctx->fork_ev, (hipStream_t)stream));
  for (int i = 0; i < 2; ++i) HIP_TRY(ctx, hipStreamWaitEvent(ctx->lane_s[i], ctx->fork_ev, 0));
  int64_t load[2] = {0, 0};
  crf_status st = CRF_OK;
  for (int i : order) {
    const int lane = load[1] < load[0] ? 1 : 0;
    load[lane] += work(i);
    crf_context *c = lane ? ctx->lane2 : ctx;
    const crf_window_item &it = items[i];
    st = run_window(c, it.hidden_at_boundary, base_weights, it.lora, it.l0, it.h, &it.kv, it.hidden_out,
                    ctx->lane_s[lane]);
    if (st != CRF_OK) {
      if (c != ctx) ctx->last_error = c->last_error;
      break;
    }
  }
  // join both lanes back into the caller's stream, also after a failed launch
  for (int i = 0; i < 2; ++i) {
    HIP_TRY(ctx, hipEventRecord(ctx->join_ev[i], ctx->lane_s[i]));
    HIP_TRY(ctx, hipStreamWaitEvent((hipStream_t)stream, ctx->join_ev[i], 0));
  }
  return st;
}

crf_status crf_decode_logits(crf_context *ctx, const crf_model_dims *dims, const void *new_tokens, int32_t n_new,
                             const crf_layer_weights *base_weights, const crf_lora_layer *lora,
                             const crf_kv_cache *kv_cache, const void *final_norm, const void *lm_head,
                             int32_t vocab, float *logits_out, void *stream) {
  if (!ctx) return fail(nullptr, CRF_ERR_INVALID_ARG, "context is NULL");
  const char *what = "crf_decode_logits";
  if (!kv_cache) return fail(ctx, CRF_ERR_INVALID_ARG, "%s: kv_cache is NULL", what);
  if (n_new < 1) return fail(ctx, CRF_ERR_SHAPE, "%s: n_new must be >= 1", what);
  if (ctx->dims.dtype != CRF_BF16) return fail(ctx, CRF_ERR_UNSUPPORTED, "%s: bf16 contexts only", what);
  // every layer, over the prefix plus the new tokens (their slots are written)
  crf_kv_cache ext = *kv_cache;
  ext.n_tokens = kv_cache->n_tokens + n_new;
  crf_status st = check_request(ctx, dims, new_tokens, base_weights, lora, 0, ctx->dims.n_layers, &ext, nullptr,
                                what, n_new);
  if (st != CRF_OK) return st;
  if (n_new > ctx->max_tokens)
    return fail(ctx, CRF_ERR_WORKSPACE, "%s: n_new %d exceeds the context's max_tokens", what, n_new);
  if (vocab < 8 || vocab % 8)
    return fail(ctx, CRF_ERR_UNSUPPORTED, "%s: vocab must be a positive multiple of 8 (got %d)", what, vocab);
  if ((int64_t)vocab * ctx->dims.d_model * 2 >= (int64_t)CRF_OOB)
    return fail(ctx, CRF_ERR_UNSUPPORTED, "%s: LM head larger than 2 GiB", what);
  if (!final_norm || !lm_head || !logits_out || !aligned16(final_norm) || !aligned16(lm_head) ||
      !aligned16(logits_out))
    return fail(ctx, CRF_ERR_INVALID_ARG, "%s: final_norm, lm_head or logits_out NULL or misaligned", what);
  hipStream_t s = (hipStream_t)stream;
  const crf_model_dims &d = ctx->dims;
  st = run_layers_bf16(ctx, new_tokens, base_weights, lora, 0, d.n_layers, &ext, nullptr, s, n_new,
                       kv_cache->n_tokens, false);
  if (st != CRF_OK) return st;
  // final RMSNorm of the last new token (fp32 residual stream) and the LM head
  const size_t D = d.d_model;
  LAUNCH(ctx, s, CRF_KK_NORM,
         launch_rmsnorm(s, ctx->hres + (size_t)(n_new - 1) * D, true, final_norm, false, ctx->xn, false, nullptr, 1,
                        (int)D, d.rms_eps));
  GemmParams p{};
  p.X = (const bf16 *)ctx->xn;
  p.ldx = D;
  p.M = 1;
  p.K = (int)D;
  p.N = vocab;
  p.w[0] = (const bf16 *)lm_head;
  p.resid = logits_out;
  p.ldr = vocab;
  p.resid_overwrite = 1;
  LAUNCH(ctx, s, CRF_KK_OTHER, launch_gemm_skinny_bf16(s, EPI_RESID, d.head_dim, p));
  return CRF_OK;
}

crf_status crf_layer_drift(crf_context *ctx, const crf_model_dims *dims, const crf_lora_layer *current,
                           int32_t n_versions, const crf_lora_layer *const *versions,
                           const int32_t *anchor_version, const float *sensitivity, int32_t per_layer_only,
                           float *drift_out, float *risk_out, float *sq_partial_out, void *stream) {
  if (!ctx) return fail(nullptr, CRF_ERR_INVALID_ARG, "context is NULL");
  crf_status st = check_dims(ctx, dims);
  if (st != CRF_OK) return st;
  if (!same_dims(*dims, ctx->dims)) return fail(ctx, CRF_ERR_INVALID_ARG, "dims differ from the context's");
  DriftPlan pl;
  if ((st = drift_plan(ctx, dims, current, n_versions, versions, anchor_version, drift_out, risk_out, pl)) != CRF_OK)
    return st;
  hipStream_t s = (hipStream_t)stream;
  if (!ctx->drift_ev) HIP_TRY(ctx, hipEventCreateWithFlags(&ctx->drift_ev, hipEventDisableTiming));
  if (ctx->drift_ev_recorded) HIP_TRY(ctx, hipEventSynchronize(ctx->drift_ev));
  if (pl.host_bytes > ctx->drift_host_bytes) {
    if (ctx->drift_host) HIP_TRY(ctx, hipHostFree(ctx->drift_host));
    ctx->drift_host = nullptr;
    ctx->drift_host_bytes = 0;
    HIP_TRY(ctx, hipHostMalloc(&ctx->drift_host, pl.host_bytes, hipHostMallocDefault));
    ctx->drift_host_bytes = pl.host_bytes;
  }
  if (pl.dev_bytes > ctx->drift_dev_bytes) {
    HIP_TRY(ctx, hipStreamSynchronize(s));
    if (ctx->drift_dev) HIP_TRY(ctx, hipFree(ctx->drift_dev));
    ctx->drift_dev = nullptr;
    ctx->drift_dev_bytes = 0;
    HIP_TRY(ctx, hipMalloc(&ctx->drift_dev, pl.dev_bytes));
    ctx->drift_dev_bytes = pl.dev_bytes;
  }
  char *hb = (char *)ctx->drift_host, *db = (char *)ctx->drift_dev;
  drift_fill(pl, dims, current, versions, anchor_version, hb);
  HIP_TRY(ctx, hipMemcpyAsync(db, hb, pl.host_bytes, hipMemcpyHostToDevice, s));
  HIP_TRY(ctx, hipEventRecord(ctx->drift_ev, s));
  ctx->drift_ev_recorded = true;
  LAUNCH(ctx, s, CRF_KK_DRIFT,
         drift_launch(s, pl, db, dims->dtype == CRF_F32, sensitivity, per_layer_only, drift_out, risk_out,
                      sq_partial_out));
  return CRF_OK;
}

crf_status crf_layer_drift_noalloc(const crf_model_dims *dims, const crf_lora_layer *current, int32_t n_versions,
                                   const crf_lora_layer *const *versions, const int32_t *anchor_version,
                                   const float *sensitivity, int32_t per_layer_only, float *drift_out,
                                   float *risk_out, float *sq_partial_out, void *stream) {
  crf_status st = check_dims(nullptr, dims);
  if (st != CRF_OK) return st;
  DriftPlan pl;
  if ((st = drift_plan(nullptr, dims, current, n_versions, versions, anchor_version, drift_out, risk_out, pl)) !=
      CRF_OK)
    return st;
  if (pl.dev_bytes > CRF_DRIFT_NOALLOC_MAX_BYTES)
    return fail(nullptr, CRF_ERR_WORKSPACE,
                "crf_layer_drift_noalloc: %zu segments in %zu chunks need %zu bytes of scratch, more than its %d",
                pl.n_segs, pl.n_chunks, pl.dev_bytes, CRF_DRIFT_NOALLOC_MAX_BYTES);
  void *scratch = nullptr;
  hipError_t e = drift_noalloc_scratch(&scratch);
  if (e != hipSuccess)
    return fail(nullptr, CRF_ERR_HIP, "crf_layer_drift_noalloc: scratch address: %s", hipGetErrorString(e));
  // host staging of the tables: one fixed buffer per host thread
  static thread_local char hstage[CRF_DRIFT_NOALLOC_MAX_BYTES];
  drift_fill(pl, dims, current, versions, anchor_version, hstage);
  hipStream_t s = (hipStream_t)stream;
  // a copy from pageable memory has read the source when it returns
  e = hipMemcpyAsync(scratch, hstage, pl.host_bytes, hipMemcpyHostToDevice, s);
  if (e == hipSuccess)
    e = drift_launch(s, pl, (char *)scratch, dims->dtype == CRF_F32, sensitivity, per_layer_only, drift_out,
                     risk_out, sq_partial_out);
  if (e != hipSuccess) return fail(nullptr, CRF_ERR_HIP, "crf_layer_drift_noalloc: %s", hipGetErrorString(e));
  return CRF_OK;
}

crf_status crf_context_device_errors(crf_context *ctx, int32_t *flags_out) {
  if (!ctx || !flags_out) return fail(ctx, CRF_ERR_INVALID_ARG, "NULL argument");
  HIP_TRY(ctx, hipDeviceSynchronize());
  int v = 0;
  HIP_TRY(ctx, hipMemcpy(&v, ctx->d_err, sizeof(int), hipMemcpyDeviceToHost));
  HIP_TRY(ctx, hipMemset(ctx->d_err, 0, sizeof(int)));
  if (ctx->lane2) {  // the second workspace's flags (concurrent batch items)
    int v2 = 0;
    HIP_TRY(ctx, hipMemcpy(&v2, ctx->lane2->d_err, sizeof(int), hipMemcpyDeviceToHost));
    HIP_TRY(ctx, hipMemset(ctx->lane2->d_err, 0, sizeof(int)));
    v |= v2;
  }
  *flags_out = v;
  return CRF_OK;
}

crf_status crf_context_set_timing(crf_context *ctx, int32_t enable) {
  return crf_context_set_timing_classes(ctx, enable ? (1u << CRF_KK_COUNT) - 1u : 0u);
}

crf_status crf_context_set_timing_classes(crf_context *ctx, uint32_t class_mask) {
  if (!ctx) return fail(nullptr, CRF_ERR_INVALID_ARG, "context is NULL");
  if (class_mask >> CRF_KK_COUNT) return fail(ctx, CRF_ERR_INVALID_ARG, "class mask 0x%x has bits past CRF_KK_COUNT", class_mask);
  ctx->timer.mask = class_mask;
  return CRF_OK;
}

crf_status crf_context_read_timing(crf_context *ctx, float *ms_out, int32_t *count_out, int32_t n_kinds) {
  if (!ctx || !ms_out || !count_out || n_kinds < 0) return fail(ctx, CRF_ERR_INVALID_ARG, "bad argument");
  for (int k = 0; k < n_kinds; ++k) {
    ms_out[k] = 0.f;
    count_out[k] = 0;
  }
  Timer &t = ctx->timer;
  if (t.used > 0) HIP_TRY(ctx, hipEventSynchronize(t.ev[2 * t.used - 1]));
  for (size_t i = 0; i < t.used; ++i) {
    float ms = 0.f;
    HIP_TRY(ctx, hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]));
    const int k = t.kind[i];
    if (k >= 0 && k < n_kinds) {
      ms_out[k] += ms;
      count_out[k] += 1;
    }
  }
  t.used = 0;
  return CRF_OK;
}

}  // extern "C"

crf_status crf_device_info(int32_t device, int32_t *n_cu_out, int32_t *max_sclk_mhz_out, char *name,
                           int32_t name_len) {
  if (!n_cu_out || !max_sclk_mhz_out) return fail(nullptr, CRF_ERR_INVALID_ARG, "null output");
  hipDeviceProp_t prop;
  const hipError_t e = hipGetDeviceProperties(&prop, device);
  if (e != hipSuccess) return fail(nullptr, CRF_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
  *n_cu_out = prop.multiProcessorCount;
  *max_sclk_mhz_out = prop.clockRate / 1000;
  if (name && name_len > 0) {
    snprintf(name, (size_t)name_len, "%s", prop.gcnArchName);
  }
  return CRF_OK;
}
