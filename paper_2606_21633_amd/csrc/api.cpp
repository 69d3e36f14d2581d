// C ABI of libherald.so: argument validation (host only, before any launch),
// workspace carve-up and the two-stream block pipeline. Kernels live in the
// .hip files of this directory.
#include <stdint.h>
#include <string.h>

#include "common.h"
#include "select.h"

using namespace herald;

namespace {

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned256(const void *p) { return ((uintptr_t)p & 255u) == 0; }

int elt_of(const herald_heads *h) { return h->dtype == HERALD_BF16 ? 2 : 4; }

herald_status check_heads(const herald_heads *h) {
  if (!h) return HERALD_ERR_INVALID_ARG;
  if (h->num_q_heads < 1 || h->num_kv_heads < 1 || h->num_q_heads % h->num_kv_heads)
    return HERALD_ERR_INVALID_ARG;
  if (h->dtype != HERALD_F32 && h->dtype != HERALD_BF16) return HERALD_ERR_INVALID_ARG;
  const int G = h->num_q_heads / h->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return HERALD_ERR_UNSUPPORTED;
  if (h->head_dim != 64 && h->head_dim != 128) return HERALD_ERR_UNSUPPORTED;
  return HERALD_OK;
}

herald_status check_block(int32_t block) {
  if (block < 1) return HERALD_ERR_INVALID_ARG;
  if (block > 64) return HERALD_ERR_UNSUPPORTED;
  return HERALD_OK;
}

bool stride_ok(int64_t s, int elt) { return s >= 0 && (s * elt) % 16 == 0; }

herald_status check_kv(const herald_heads *h, const herald_kv *kv, bool need_v) {
  if (!kv || !kv->k || (need_v && !kv->v) || !kv->seq_lens) return HERALD_ERR_INVALID_ARG;
  if (kv->max_seq_len < 1 || kv->max_seq_len > INT32_MAX) return HERALD_ERR_INVALID_ARG;
  const int elt = elt_of(h);
  if (!aligned16(kv->k) || (need_v && !aligned16(kv->v))) return HERALD_ERR_INVALID_ARG;
  if (kv->stride_s < h->head_dim || !stride_ok(kv->stride_s, elt) ||
      !stride_ok(kv->stride_h, elt))
    return HERALD_ERR_INVALID_ARG;
  if (kv->page_table) {
    const int32_t ps = kv->page_size;
    if (ps < 1 || (ps & (ps - 1))) return HERALD_ERR_INVALID_ARG;
    if (ps < 8) return HERALD_ERR_UNSUPPORTED;  // a 1 KiB load spans up to 8 rows
    if (kv->max_pages < (kv->max_seq_len + ps - 1) / ps) return HERALD_ERR_INVALID_ARG;
    if (!stride_ok(kv->stride_page, elt)) return HERALD_ERR_INVALID_ARG;
  } else if (!stride_ok(kv->stride_b, elt)) {
    return HERALD_ERR_INVALID_ARG;
  }
  return HERALD_OK;
}

herald_status check_pool(const herald_heads *h, const herald_pool *p) {
  if (!p || !p->k || !p->v || p->capacity < 1) return HERALD_ERR_INVALID_ARG;
  const int elt = elt_of(h);
  if (!aligned16(p->k) || !aligned16(p->v)) return HERALD_ERR_INVALID_ARG;
  if (p->stride_s < h->head_dim || !stride_ok(p->stride_s, elt) ||
      !stride_ok(p->stride_h, elt) || !stride_ok(p->stride_b, elt))
    return HERALD_ERR_INVALID_ARG;
  return HERALD_OK;
}

KvView view_of(const herald_kv *kv) {
  KvView v{};
  v.k = reinterpret_cast<const char *>(kv->k);
  v.v = reinterpret_cast<const char *>(kv->v);
  v.sb = kv->stride_b;
  v.sh = kv->stride_h;
  v.ss = kv->stride_s;
  v.pt = kv->page_table;
  v.page_shift = 0;
  if (kv->page_table)
    while ((1 << v.page_shift) < kv->page_size) ++v.page_shift;
  v.max_pages = kv->max_pages;
  v.sp = kv->stride_page;
  v.lens = kv->seq_lens;
  v.max_len = kv->max_seq_len;
  return v;
}

PoolView pool_of(const herald_pool *p) {
  return PoolView{reinterpret_cast<char *>(p->k), reinterpret_cast<char *>(p->v),
                  p->stride_b, p->stride_h, p->stride_s};
}

herald_kv kv_of_pool(const herald_pool *p, const int32_t *lens, int64_t max_len) {
  herald_kv kv{};
  kv.k = p->k;
  kv.v = p->v;
  kv.stride_b = p->stride_b;
  kv.stride_h = p->stride_h;
  kv.stride_s = p->stride_s;
  kv.page_table = nullptr;
  kv.seq_lens = lens;
  kv.max_seq_len = max_len;
  return kv;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t attn_ws_bytes(const AttnPlan &p) {
  if (p.nsplit_cap <= 1) return 0;
  return align256(p.part_o_bytes) + align256(p.part_ml_bytes);
}

herald_status hip_status(hipError_t e) { return e == hipSuccess ? HERALD_OK : HERALD_ERR_HIP; }

}  // namespace

extern "C" {

const char *herald_status_string(herald_status s) {
  switch (s) {
    case HERALD_OK: return "ok";
    case HERALD_ERR_INVALID_ARG: return "invalid argument";
    case HERALD_ERR_UNSUPPORTED: return "unsupported shape";
    case HERALD_ERR_WORKSPACE: return "workspace missing or too small";
    case HERALD_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

int32_t herald_budget_tokens(int64_t S, int32_t num, int32_t den) {
  if (S <= 0 || den <= 0 || num < 0) return 0;
  int64_t k = (S * (int64_t)num + den / 2) / den;
  if (k < 1) k = 1;
  if (k > S) k = S;
  return (int32_t)k;
}

size_t herald_select_workspace(const herald_heads *heads, int32_t batch, int64_t max_seq_len) {
  if (check_heads(heads) != HERALD_OK || batch < 1 || max_seq_len < 1) return 0;
  return select_ws_bytes(batch, heads->num_q_heads, heads->num_kv_heads, heads->head_dim,
                         max_seq_len, nullptr, nullptr);
}

// The selections share one path: x = 0 ranks with the mean of the block's
// queries, x >= 1 with its x centred rows; tail rows (n_tail >= 0) enter the
// softmax statistics only.
static herald_status select_common(const herald_heads *heads, int32_t batch, int32_t block,
                                   int32_t x, const void *q_sel, const herald_kv *kv,
                                   const void *tail, const void *tail_v, int32_t n_tail,
                                   const int32_t *k_per_seq, int32_t k_max, int32_t *idx_out,
                                   void *o_out, void *ws, size_t ws_bytes, hipStream_t stream) {
  herald_status st;
  if ((st = check_heads(heads)) != HERALD_OK) return st;
  if ((st = check_block(block)) != HERALD_OK) return st;
  if (batch < 1 || x < 0 || x > block || !q_sel || !aligned16(q_sel) || !k_per_seq || !idx_out)
    return HERALD_ERR_INVALID_ARG;
  if (n_tail < 0 || n_tail > 64 || (n_tail > 0 && (!tail || !aligned16(tail))))
    return HERALD_ERR_INVALID_ARG;
  if (o_out && (!aligned16(o_out) || (n_tail > 0 && (!tail_v || !aligned16(tail_v)))))
    return HERALD_ERR_INVALID_ARG;
  const int G = heads->num_q_heads / heads->num_kv_heads;
  const int V = (x == 0 ? 1 : x) * G;
  if (V > kMaxScoreRows) return HERALD_ERR_UNSUPPORTED;
  if ((st = check_kv(heads, kv, o_out != nullptr)) != HERALD_OK) return st;  // V for o_out
  if (k_max < 1 || k_max > kv->max_seq_len) return HERALD_ERR_INVALID_ARG;
  const size_t need = herald_select_xq_workspace(heads, batch, x == 0 ? 1 : x, kv->max_seq_len);
  if (!ws || !aligned256(ws) || ws_bytes < need) return HERALD_ERR_WORKSPACE;
  SelectWs layout;
  select_ws_bytes(batch, V * heads->num_kv_heads, heads->num_kv_heads, heads->head_dim,
                  kv->max_seq_len, &layout, reinterpret_cast<char *>(ws));
  if (x == 0)
    return hip_status(launch_select(*heads, batch, block, q_sel, view_of(kv), tail, tail_v,
                                    n_tail, k_per_seq, k_max, idx_out, o_out, layout, stream));
  return hip_status(launch_select_xq(*heads, batch, block, x, q_sel, view_of(kv), tail, tail_v,
                                     n_tail, k_per_seq, k_max, idx_out, o_out, layout, stream));
}

herald_status herald_select(const herald_heads *heads, int32_t batch, int32_t block,
                            const void *q_sel, const herald_kv *kv,
                            const int32_t *k_per_seq, int32_t k_max, int32_t *idx_out,
                            void *ws, size_t ws_bytes, hipStream_t stream) {
  return select_common(heads, batch, block, 0, q_sel, kv, nullptr, nullptr, 0, k_per_seq,
                       k_max, idx_out, nullptr, ws, ws_bytes, stream);
}

size_t herald_select_xq_workspace(const herald_heads *heads, int32_t batch, int32_t x,
                                  int64_t max_seq_len) {
  if (check_heads(heads) != HERALD_OK || batch < 1 || max_seq_len < 1 || x < 1) return 0;
  const int64_t V = (int64_t)x * (heads->num_q_heads / heads->num_kv_heads);
  if (V > kMaxScoreRows) return 0;
  // the selection workspace with V score rows per KV head in place of G
  return select_ws_bytes(batch, (int)V * heads->num_kv_heads, heads->num_kv_heads,
                         heads->head_dim, max_seq_len, nullptr, nullptr);
}

herald_status herald_select_xq(const herald_heads *heads, int32_t batch, int32_t block,
                               int32_t x, const void *q_sel, const herald_kv *kv,
                               const int32_t *k_per_seq, int32_t k_max, int32_t *idx_out,
                               void *ws, size_t ws_bytes, hipStream_t stream) {
  if (x < 1) return HERALD_ERR_INVALID_ARG;
  return select_common(heads, batch, block, x, q_sel, kv, nullptr, nullptr, 0, k_per_seq,
                       k_max, idx_out, nullptr, ws, ws_bytes, stream);
}

herald_status herald_select_draft(const herald_heads *heads, int32_t batch, int32_t block,
                                  int32_t x, const void *q_sel, const herald_kv *kv,
                                  const void *draft_k, int32_t n_draft,
                                  const int32_t *k_per_seq, int32_t k_max, int32_t *idx_out,
                                  void *ws, size_t ws_bytes, hipStream_t stream) {
  return select_common(heads, batch, block, x, q_sel, kv, draft_k, nullptr, n_draft, k_per_seq,
                       k_max, idx_out, nullptr, ws, ws_bytes, stream);
}

herald_status herald_select_attn(const herald_heads *heads, int32_t batch, int32_t block,
                                 int32_t x, const void *q_sel, const herald_kv *kv,
                                 const void *draft_k, const void *draft_v, int32_t n_draft,
                                 const int32_t *k_per_seq, int32_t k_max, int32_t *idx_out,
                                 void *o_out, void *ws, size_t ws_bytes, hipStream_t stream) {
  if (!o_out) return HERALD_ERR_INVALID_ARG;
  return select_common(heads, batch, block, x, q_sel, kv, draft_k, draft_v, n_draft, k_per_seq,
                       k_max, idx_out, o_out, ws, ws_bytes, stream);
}

herald_status herald_gather(const herald_heads *heads, int32_t batch, const herald_kv *kv,
                            const int32_t *idx, const int32_t *k_per_seq, int32_t k_max,
                            const herald_pool *dst, int32_t dst_row0, hipStream_t stream) {
  herald_status st;
  if ((st = check_heads(heads)) != HERALD_OK) return st;
  if (batch < 1 || !idx || !k_per_seq || k_max < 1 || dst_row0 < 0)
    return HERALD_ERR_INVALID_ARG;
  if ((st = check_kv(heads, kv, true)) != HERALD_OK) return st;
  if ((st = check_pool(heads, dst)) != HERALD_OK) return st;
  if ((int64_t)dst_row0 + k_max > dst->capacity) return HERALD_ERR_INVALID_ARG;
  return hip_status(launch_gather(*heads, batch, view_of(kv), idx, k_per_seq, k_max,
                                  pool_of(dst), dst_row0, stream));
}

size_t herald_block_attn_workspace(const herald_heads *heads, int32_t batch, int32_t block,
                                   int64_t max_ctx) {
  if (check_heads(heads) != HERALD_OK || check_block(block) != HERALD_OK || batch < 1 ||
      max_ctx < 0)
    return 0;
  // at least one byte so that "0" always means invalid
  const size_t b = attn_ws_bytes(attn_plan(*heads, batch, block, max_ctx));
  return b ? b : 256;
}

herald_status herald_block_attn(const herald_heads *heads, int32_t batch, int32_t block,
                                const void *q, const herald_kv *ctx, const void *blk_k,
                                const void *blk_v, void *out, void *ws, size_t ws_bytes,
                                hipStream_t stream) {
  return herald_block_attn_groups(heads, batch, block, 1, q, ctx, blk_k, blk_v, out, ws,
                                  ws_bytes, stream);
}

herald_status herald_block_attn_groups(const herald_heads *heads, int32_t batch, int32_t block,
                                       int32_t groups, const void *q, const herald_kv *ctx,
                                       const void *blk_k, const void *blk_v, void *out,
                                       void *ws, size_t ws_bytes, hipStream_t stream) {
  herald_status st;
  if ((st = check_heads(heads)) != HERALD_OK) return st;
  if ((st = check_block(block)) != HERALD_OK) return st;
  if (batch < 1 || groups < 1 || (int64_t)batch * groups > INT32_MAX / 1024 || !q || !blk_k ||
      !blk_v || !out || !aligned16(q) || !aligned16(blk_k) || !aligned16(blk_v) ||
      !aligned16(out))
    return HERALD_ERR_INVALID_ARG;
  if (!ctx || !ctx->seq_lens || ctx->max_seq_len < 0 || ctx->max_seq_len > INT32_MAX)
    return HERALD_ERR_INVALID_ARG;
  if (ctx->max_seq_len > 0) {
    herald_kv c = *ctx;
    if ((st = check_kv(heads, &c, true)) != HERALD_OK) return st;
  }
  const size_t need = herald_block_attn_workspace(heads, batch * groups, block,
                                                  ctx->max_seq_len);
  const AttnPlan p = attn_plan(*heads, batch * groups, block, ctx->max_seq_len);
  if (p.nsplit > 1 && (!ws || !aligned256(ws) || ws_bytes < need)) return HERALD_ERR_WORKSPACE;
  return hip_status(launch_block_attn(*heads, batch, block, groups, q, view_of(ctx),
                                      ctx->max_seq_len, blk_k, blk_v, out, ws, stream));
}

size_t herald_decode_block_workspace(const herald_heads *heads, int32_t batch, int32_t block,
                                     int64_t max_seq_len, int32_t k_max) {
  if (check_heads(heads) != HERALD_OK || check_block(block) != HERALD_OK || batch < 1 ||
      max_seq_len < 1 || k_max < 1)
    return 0;
  const size_t sel = align256(herald_select_workspace(heads, batch, max_seq_len));
  const size_t idx = align256((size_t)batch * heads->num_kv_heads * k_max * sizeof(int32_t));
  int64_t max_ctx = max_seq_len > (int64_t)k_max + block ? max_seq_len : (int64_t)k_max + block;
  const size_t att = align256(herald_block_attn_workspace(heads, batch, block, max_ctx));
  return sel + idx + att;
}

herald_status herald_decode_block(const herald_heads *heads, int32_t num_layers,
                                  int32_t batch, int32_t block, int32_t steps,
                                  const herald_layer *layers, int32_t *seq_lens,
                                  int64_t max_seq_len, const int32_t *n_active,
                                  int64_t max_active, int32_t *n_idle,
                                  const int32_t *k_next, int32_t k_max, int32_t dense,
                                  void *ws, size_t ws_bytes, hipStream_t s_main,
                                  hipStream_t s_retr) {
  herald_status st;
  if ((st = check_heads(heads)) != HERALD_OK) return st;
  if ((st = check_block(block)) != HERALD_OK) return st;
  if (num_layers < 1 || batch < 1 || steps < 1 || !layers || !seq_lens || max_seq_len < 1 ||
      max_seq_len > INT32_MAX)
    return HERALD_ERR_INVALID_ARG;
  // a layer is dense if the call is (the all-dense baseline) or its own flag is set
  auto layer_dense = [&](int l) { return dense != 0 || layers[l].dense != 0; };
  bool any_sparse = false;
  for (int l = 0; l < num_layers; ++l) any_sparse = any_sparse || !layer_dense(l);
  if (any_sparse && (!n_active || max_active < 0 || !n_idle || !k_next || k_max < 1 ||
                     k_max > max_seq_len))
    return HERALD_ERR_INVALID_ARG;
  const int elt = elt_of(heads);
  for (int l = 0; l < num_layers; ++l) {
    const herald_layer &L = layers[l];
    if ((st = check_pool(heads, &L.cache)) != HERALD_OK) return st;
    if ((int64_t)L.cache.capacity < max_seq_len + block) return HERALD_ERR_INVALID_ARG;
    if (!layer_dense(l)) {
      if ((st = check_pool(heads, &L.active)) != HERALD_OK) return st;
      if ((st = check_pool(heads, &L.idle)) != HERALD_OK) return st;
      if ((int64_t)L.active.capacity < max_active) return HERALD_ERR_INVALID_ARG;
      if ((int64_t)L.idle.capacity < (int64_t)k_max + block) return HERALD_ERR_INVALID_ARG;
      if (!L.q_next || !aligned16(L.q_next)) return HERALD_ERR_INVALID_ARG;
    }
    const void *ptrs[6] = {L.q_steps, L.blk_k, L.blk_v, L.done_k, L.done_v, L.out};
    for (const void *p : ptrs)
      if (!p || !aligned16(p)) return HERALD_ERR_INVALID_ARG;
    if (L.out_step_stride < 0 || !stride_ok(L.out_step_stride, elt)) return HERALD_ERR_INVALID_ARG;
    if (L.select_x != 0 && L.select_x != 1) return HERALD_ERR_INVALID_ARG;
    if (L.q_draft) {
      const void *dp[4] = {L.q_draft, L.draft_k, L.draft_v, L.out_draft};
      for (const void *p : dp)
        if (!p || !aligned16(p)) return HERALD_ERR_INVALID_ARG;
      if (steps < 2) return HERALD_ERR_INVALID_ARG;  // the draft runs with step 1
    }
  }
  bool any_draft = false;
  for (int l = 0; l < num_layers; ++l) any_draft = any_draft || layers[l].q_draft != nullptr;
  const size_t need = herald_decode_block_workspace(heads, batch, block, max_seq_len,
                                                    any_sparse ? k_max : 1);
  if (!ws || !aligned256(ws) || ws_bytes < need) return HERALD_ERR_WORKSPACE;

  // workspace: [selection][idx][attention partials]
  char *w = reinterpret_cast<char *>(ws);
  const size_t sel_bytes = align256(herald_select_workspace(heads, batch, max_seq_len));
  const size_t idx_bytes =
      align256((size_t)batch * heads->num_kv_heads * (any_sparse ? k_max : 1) * sizeof(int32_t));
  SelectWs sel;
  select_ws_bytes(batch, heads->num_q_heads, heads->num_kv_heads, heads->head_dim, max_seq_len,
                  &sel, w);
  int32_t *idx = reinterpret_cast<int32_t *>(w + sel_bytes);
  void *attn_ws = w + sel_bytes + idx_bytes;

  const int64_t Hq = heads->num_q_heads, Hkv = heads->num_kv_heads, D = heads->head_dim;
  const int64_t q_step = (int64_t)batch * block * Hq * D;   // elements per step
  const int64_t kv_step = (int64_t)batch * block * Hkv * D;

  hipEvent_t ev_start = nullptr, ev_sel = nullptr, ev_draft = nullptr;
  hipError_t e = hipEventCreateWithFlags(&ev_start, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&ev_sel, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&ev_draft, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventRecord(ev_start, s_main);

  // retrieval stream, once `after` has been reached on the main stream: the
  // next block's selection (with the layer's draft as normalisation tail, if
  // it has one) and the gather into the idle pools
  auto retrieval = [&](hipEvent_t after) -> hipError_t {
    hipError_t r = hipStreamWaitEvent(s_retr, after, 0);
    for (int l = 0; l < num_layers && r == hipSuccess; ++l) {
      if (layer_dense(l)) continue;
      const herald_layer &L = layers[l];
      herald_kv cache = kv_of_pool(&L.cache, seq_lens, max_seq_len);
      const void *tail = L.q_draft ? L.draft_k : nullptr;
      const int n_tail = L.q_draft ? block : 0;
      r = L.select_x == 0
              ? launch_select(*heads, batch, block, L.q_next, view_of(&cache), tail, nullptr,
                              n_tail, k_next, k_max, idx, nullptr, sel, s_retr)
              : launch_select_xq(*heads, batch, block, 1, L.q_next, view_of(&cache), tail,
                                 nullptr, n_tail, k_next, k_max, idx, nullptr, sel, s_retr);
      if (r == hipSuccess)
        r = launch_gather(*heads, batch, view_of(&cache), idx, k_next, k_max, pool_of(&L.idle),
                          0, s_retr);
    }
    if (r == hipSuccess) r = hipEventRecord(ev_sel, s_retr);
    return r;
  };
  // main stream: denoising step t of every layer (step 1 with the draft group)
  auto step = [&](int t) -> hipError_t {
    hipError_t r = hipSuccess;
    for (int l = 0; l < num_layers && r == hipSuccess; ++l) {
      const herald_layer &L = layers[l];
      herald_kv ctx = layer_dense(l) ? kv_of_pool(&L.cache, seq_lens, max_seq_len)
                                     : kv_of_pool(&L.active, n_active, max_active);
      const char *q = reinterpret_cast<const char *>(L.q_steps) + t * q_step * elt;
      const char *bk = reinterpret_cast<const char *>(L.blk_k) + t * kv_step * elt;
      const char *bv = reinterpret_cast<const char *>(L.blk_v) + t * kv_step * elt;
      char *o = reinterpret_cast<char *>(L.out) + t * L.out_step_stride * elt;
      r = launch_block_attn(*heads, batch, block, 1, q, view_of(&ctx), ctx.max_seq_len, bk, bv,
                            o, attn_ws, s_main);
      if (r == hipSuccess && t == 1 && L.q_draft)
        r = launch_block_attn(*heads, batch, block, 1, L.q_draft, view_of(&ctx),
                              ctx.max_seq_len, L.draft_k, L.draft_v, L.out_draft, attn_ws,
                              s_main);
    }
    return r;
  };
  if (!any_draft) {
    if (e == hipSuccess && any_sparse) e = retrieval(ev_start);
    for (int t = 0; t < steps && e == hipSuccess; ++t) e = step(t);
  } else {
    // the selection needs the draft, which the 2B-token step 1 produces
    for (int t = 0; t < 2 && e == hipSuccess; ++t) e = step(t);
    if (e == hipSuccess) e = hipEventRecord(ev_draft, s_main);
    if (e == hipSuccess && any_sparse) e = retrieval(ev_draft);
    for (int t = 2; t < steps && e == hipSuccess; ++t) e = step(t);
  }
  // join, append the completed block, advance the lengths
  if (e == hipSuccess && any_sparse) e = hipStreamWaitEvent(s_main, ev_sel, 0);
  for (int l = 0; l < num_layers && e == hipSuccess; ++l) {
    const herald_layer &L = layers[l];
    const PoolView idle = pool_of(&L.idle);
    e = launch_append(*heads, batch, block, L.done_k, L.done_v, pool_of(&L.cache), seq_lens,
                      layer_dense(l) ? nullptr : &idle, k_next, k_max, L.cache.capacity, s_main);
  }
  if (e == hipSuccess)
    e = launch_bump(batch, block, seq_lens, any_sparse ? n_idle : nullptr, k_next, k_max,
                    s_main);
  if (ev_start) hipEventDestroy(ev_start);
  if (ev_sel) hipEventDestroy(ev_sel);
  if (ev_draft) hipEventDestroy(ev_draft);
  return hip_status(e);
}

}  // extern "C"
