/*
 * herald.h — C ABI of libherald.so, the MI355X (gfx950) hot path of HERALD's
 * sparse block-diffusion-LLM decode (arXiv 2606.21633).
 *
 * A block dLLM decodes a block of B tokens over T denoising steps; only
 * completed blocks enter the KV cache (sec. II-A). HERALD splits sparse
 * attention into a selection phase run once per block over the full cache and
 * a denoising phase that reuses the selected entries for all T steps
 * (sec. I, sec. III-C). This library runs both phases out of HBM:
 *
 *   herald_select      representative query (mean of the block's B queries,
 *                      sec. IV-A.2), scores over every cached token, GQA
 *                      importance s_hat_h[s] = sum_g exp(s[g,s]-m_g)/l_g and
 *                      one top-k per KV head (sec. IV-B.4).
 *   herald_select_xq   the same selection with x query rows of the block
 *                      used as they are: x = 1 is the paper's centre [MASK]
 *                      query (sec. IV-A.2, Eq. 2), x = B every block query;
 *                      the cost grows with x (the query-count trade-off of
 *                      sec. IV-A.2).
 *   herald_select_draft the next block's selection with the current
 *                      block's draft KV appended for normalisation
 *                      (draft-based lookahead, sec. IV-A.1, sec. IV-B.2);
 *                      herald_select_attn also returns the representative
 *                      queries' attention output (sec. IV-B.4).
 *   herald_gather      copies the selected K/V rows into a sparse pool
 *                      (sec. IV-B.3).
 *   herald_block_attn  B-query GQA attention over a context (a pool, or a
 *                      full cache for the dense baseline) plus the block's
 *                      own KV (sec. II-A, sec. V); herald_block_attn_groups
 *                      runs several query groups that share the context
 *                      (the 2B-token denoising + draft step, sec. IV-B.2).
 *   herald_decode_block one block over L layers as a two-stream pipeline:
 *                      the next block's selection on one stream, the T
 *                      denoising steps on the other, double-buffered pools
 *                      (sec. IV-A.1, sec. IV-B.1, sec. IV-B.2).
 *
 * Conventions
 *   - Ownership: the caller owns every buffer (device memory) and every
 *     stream. The library allocates no device memory; scratch space is the
 *     caller's workspace, sized by the *_workspace functions.
 *   - Errors: every function returns a status and never aborts. All argument
 *     checks that can be made on the host run before anything is enqueued; a
 *     failing check enqueues nothing. HIP launch errors are HERALD_ERR_HIP.
 *   - Asynchrony: work is enqueued on the given stream(s) and returns at once.
 *     Calls are re-entrant across streams when their workspaces and outputs
 *     are disjoint.
 *   - Layout: tensors are row-major with the last (head_dim) axis contiguous;
 *     every row start must be 16-byte aligned (128-bit loads). Element strides
 *     are in elements of the tensor's dtype.
 *   - Shapes supported: head_dim in {64, 128}; num_q_heads a multiple of
 *     num_kv_heads with group G = num_q_heads / num_kv_heads in {1,2,4,8};
 *     1 <= block <= 64. Query head hq reads KV head hq / G.
 *   - Device-side per-sequence values (seq_lens, k_per_seq) are clamped by
 *     the kernels: k_b is taken as min(max(k_b, 0), seq_len_b, k_max).
 */
#ifndef HERALD_H
#define HERALD_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HERALD_OK = 0,
  HERALD_ERR_INVALID_ARG = 1, /* null pointer, bad size, misaligned row   */
  HERALD_ERR_UNSUPPORTED = 2, /* head_dim, group size or block not built  */
  HERALD_ERR_WORKSPACE = 3,   /* workspace missing or smaller than needed */
  HERALD_ERR_HIP = 4          /* a HIP runtime call or launch failed      */
} herald_status;

typedef enum { HERALD_F32 = 0, HERALD_BF16 = 1 } herald_dtype;

/* Attention head layout shared by every tensor of one call. */
typedef struct {
  int32_t num_q_heads;  /* H_q */
  int32_t num_kv_heads; /* H_kv; G = H_q / H_kv query heads share a KV head */
  int32_t head_dim;     /* d: 64 or 128 */
  herald_dtype dtype;   /* element type of Q, K, V, pools and outputs */
} herald_heads;

/*
 * Read-only view of a KV cache (or of a pool). Row s of KV head h of
 * sequence b starts at element
 *   contiguous (page_table == NULL):
 *       b*stride_b + h*stride_h + s*stride_s
 *   paged:
 *       page_table[b*max_pages + s/page_size]*stride_page + h*stride_h
 *       + (s % page_size)*stride_s
 * of k (and of v). seq_lens[b] (device int32) is the number of valid rows of
 * sequence b; max_seq_len (host) bounds them (larger values are clamped to
 * it). page_size must be a power of two >= 8 (HERALD_ERR_UNSUPPORTED below 8).
 */
typedef struct {
  const void *k;
  const void *v;
  int64_t stride_b;
  int64_t stride_h;
  int64_t stride_s;
  const int32_t *page_table; /* device [batch][max_pages], or NULL */
  int32_t page_size;         /* tokens per page (paged only) */
  int32_t max_pages;         /* row length of page_table (paged only) */
  int64_t stride_page;       /* elements between pages (paged only) */
  const int32_t *seq_lens;   /* device [batch] */
  int64_t max_seq_len;       /* host upper bound of seq_lens */
} herald_kv;

/* Writable contiguous pool (or cache): row j of KV head h of sequence b at
 * b*stride_b + h*stride_h + j*stride_s; capacity rows per (b, h). */
typedef struct {
  void *k;
  void *v;
  int64_t stride_b;
  int64_t stride_h;
  int64_t stride_s;
  int32_t capacity;
} herald_pool;

/*
 * Per-KV-head budget k = clamp(floor(S*num/den + 1/2), 1, S) in exact integer
 * arithmetic (the paper's budget is a fraction of the prefix per KV head,
 * sec. IV-B.4; the rounding is this library's choice). Returns 0 if S <= 0,
 * den <= 0 or num < 0.
 */
int32_t herald_budget_tokens(int64_t S, int32_t num, int32_t den);

/* Workspace bytes needed by herald_select for these sizes (0 if invalid). */
size_t herald_select_workspace(const herald_heads *heads, int32_t batch,
                               int64_t max_seq_len);

/*
 * Selection phase of one layer (sec. IV-A.2, sec. IV-B.4).
 *   q_sel     device [batch][block][H_q][d]: the block's selection queries;
 *             their mean per head is the representative query.
 *   kv        K is read (V is not): every valid row of every sequence.
 *   k_per_seq device [batch]: per-KV-head budget of each sequence (clamped,
 *             see above).
 *   k_max     host: row length of idx_out (>= 1, <= kv->max_seq_len).
 *   idx_out   device [batch][H_kv][k_max] int32: for each (b, h) the k_b row
 *             indices with the largest importance, ties to the lower index,
 *             in ascending order, then -1 up to k_max.
 * Ranking keys are fp64 (representative query, dot products, exp, softmax
 * normaliser and importance). ws must hold herald_select_workspace() bytes
 * and be 256-byte aligned; its contents on entry are ignored.
 */
herald_status herald_select(const herald_heads *heads, int32_t batch,
                            int32_t block, const void *q_sel,
                            const herald_kv *kv, const int32_t *k_per_seq,
                            int32_t k_max, int32_t *idx_out, void *ws,
                            size_t ws_bytes, hipStream_t stream);

/* Workspace bytes needed by herald_select_xq for these sizes (0 if invalid,
 * including x < 1 or x * H_q / H_kv > 512). Grows with x: the fp64 scores of
 * x * H_q / H_kv score rows per cached row are kept. */
size_t herald_select_xq_workspace(const herald_heads *heads, int32_t batch,
                                  int32_t x, int64_t max_seq_len);

/*
 * Selection with x query rows (sec. IV-A.2). The rows are the x centred in
 * the block, c0 = floor((block - x) / 2) to c0 + x - 1, each used as it is
 * (no mean): x = 1 takes the centre [MASK] position, which Eq. 2 makes the
 * representative (for even block sizes the two middle rows tie; the lower is
 * taken); x = block takes every query of the block. Every (row, query head)
 * pair is a score row with its own softmax statistics over the full cache,
 * and the importance of a cached row for KV head h is the sum of its
 * softmax-normalised scores over the x rows and the G = H_q / H_kv query
 * heads of h (the G-sum of sec. IV-B.4 taken over query rows as well; the
 * paper states no rule for x > 1, this is the library's reading).
 *   x         host: 1 <= x <= block, x * G <= 512.
 * Every other argument, the output, the fp64 ranking keys and the tie rule
 * are as for herald_select; ws must hold herald_select_xq_workspace() bytes
 * for this x and be 256-byte aligned.
 */
herald_status herald_select_xq(const herald_heads *heads, int32_t batch,
                               int32_t block, int32_t x, const void *q_sel,
                               const herald_kv *kv, const int32_t *k_per_seq,
                               int32_t k_max, int32_t *idx_out, void *ws,
                               size_t ws_bytes, hipStream_t stream);

/*
 * Selection of block n+1 with block n's draft KV appended (sec. IV-B.2,
 * steps 7 and 8; sec. IV-A.1): the draft rows are scored with the cache and
 * enter every score row's softmax statistics (m, l), so they shape the
 * importance of the cached rows, but they are never candidates: the
 * completed block replaces them (the library's reading; the paper appends
 * the draft to the pool it ranks).
 *   x         host: 0 ranks with the mean of the block's queries (as
 *             herald_select), x >= 1 with its x centred rows (as
 *             herald_select_xq; the paper's pipeline uses x = 1).
 *   draft_k   device [batch][n_draft][H_kv][d] (the draft's K; V is not
 *             read), 16-byte aligned; may be NULL if n_draft = 0.
 *   n_draft   host, 0 <= n_draft <= 64 (n_draft = 0: no draft).
 * Other arguments as herald_select; ws holds
 * herald_select_xq_workspace(heads, batch, max(x, 1), kv->max_seq_len) bytes.
 */
herald_status herald_select_draft(const herald_heads *heads, int32_t batch,
                                  int32_t block, int32_t x, const void *q_sel,
                                  const herald_kv *kv, const void *draft_k,
                                  int32_t n_draft, const int32_t *k_per_seq,
                                  int32_t k_max, int32_t *idx_out, void *ws,
                                  size_t ws_bytes, hipStream_t stream);

/*
 * herald_select_draft plus the attention output of the representative
 * queries over the cache and the draft: for every score row (representative
 * row i, query head hq = h * G + g), o = sum_s exp(z[s] - m) / l * v_s over
 * the kv->seq_lens[b] cached rows and the n_draft draft rows, with the same
 * fp64 scores and statistics as the ranking (the running output o_g that the
 * paper's fused selection kernel keeps beside (m, l) and hands to the FFN,
 * sec. IV-B.4). Weights in fp32, fp32 accumulation, then heads->dtype (bf16
 * rounded to nearest-even).
 *   kv        K and V are read.
 *   draft_v   device [batch][n_draft][H_kv][d] (the draft's V); may be NULL
 *             if n_draft = 0.
 *   o_out     device [batch][max(x, 1)][H_q][d], 16-byte aligned (not NULL).
 * Other arguments and the workspace as herald_select_draft.
 */
herald_status herald_select_attn(const herald_heads *heads, int32_t batch,
                                 int32_t block, int32_t x, const void *q_sel,
                                 const herald_kv *kv, const void *draft_k,
                                 const void *draft_v, int32_t n_draft,
                                 const int32_t *k_per_seq, int32_t k_max,
                                 int32_t *idx_out, void *o_out, void *ws,
                                 size_t ws_bytes, hipStream_t stream);

/*
 * Gather (sec. IV-B.3): for each (b, h) and j < k_b, copies row idx[b][h][j]
 * of kv's K and V into row dst_row0 + j of dst (bit-exact). Rows of dst
 * outside [dst_row0, dst_row0 + k_b) are not touched. idx is the output of
 * herald_select ([batch][H_kv][k_max]); dst_row0 + k_max <= dst->capacity.
 */
herald_status herald_gather(const herald_heads *heads, int32_t batch,
                            const herald_kv *kv, const int32_t *idx,
                            const int32_t *k_per_seq, int32_t k_max,
                            const herald_pool *dst, int32_t dst_row0,
                            hipStream_t stream);

/* Workspace bytes needed by herald_block_attn (0 if invalid). */
size_t herald_block_attn_workspace(const herald_heads *heads, int32_t batch,
                                   int32_t block, int64_t max_ctx);

/*
 * One denoising step of block attention (sec. II-A; the denoising phase of
 * sec. IV-B.2). For every sequence b, block row i < block and query head hq,
 * with h = hq / G: the keys are the ctx->seq_lens[b] context rows of KV head
 * h followed by the block's own rows blk_k[b][0..block)[h]; with
 * p = softmax(q . key / sqrt(d)), out[b][i][hq] = sum_j p_j value_j. No mask.
 *   q            device [batch][block][H_q][d]
 *   ctx          the sparse pool (or the full cache for dense attention),
 *                contiguous or paged; max_seq_len bounds the rows used.
 *   blk_k, blk_v device [batch][block][H_kv][d]
 *   out          device [batch][block][H_q][d] in heads->dtype
 * bf16 inputs run on bf16 MFMA with fp32 accumulation and softmax; the output
 * is rounded to nearest-even bf16. fp32 inputs run in fp32. ws holds
 * herald_block_attn_workspace() bytes (split-KV partials), 256-byte aligned.
 */
herald_status herald_block_attn(const herald_heads *heads, int32_t batch,
                                int32_t block, const void *q,
                                const herald_kv *ctx, const void *blk_k,
                                const void *blk_v, void *out, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/*
 * Block attention of several query groups per sequence: the 2B-token step of
 * sec. IV-B.2 (step 3), in which the denoising group and the draft group of
 * block n attend to the same completed prefix but not to each other. Group j
 * of sequence b is the block b * groups + j of a herald_block_attn call over
 * batch * groups blocks whose context is ctx's sequence b:
 *   q, out       device [batch][groups * block][H_q][d]
 *   blk_k, blk_v device [batch][groups * block][H_kv][d]; group j's queries
 *                see rows j * block .. j * block + block - 1 only.
 *   ctx          as herald_block_attn, batch sequences (shared by groups).
 *   groups       host, >= 1; groups = 1 is herald_block_attn.
 * ws holds herald_block_attn_workspace(heads, batch * groups, block,
 * ctx->max_seq_len) bytes.
 */
herald_status herald_block_attn_groups(const herald_heads *heads, int32_t batch,
                                       int32_t block, int32_t groups,
                                       const void *q, const herald_kv *ctx,
                                       const void *blk_k, const void *blk_v,
                                       void *out, void *ws, size_t ws_bytes,
                                       hipStream_t stream);

/* Tensors of one layer for herald_decode_block. */
typedef struct {
  herald_pool cache;    /* full KV cache, contiguous; rows [0, seq_len) */
  herald_pool active;   /* pool denoised over (this block's selection)  */
  herald_pool idle;     /* pool filled for the next block               */
  const void *q_steps;  /* [T][batch][block][H_q][d] denoising queries  */
  const void *blk_k;    /* [T][batch][block][H_kv][d] block K per step  */
  const void *blk_v;    /* [T][batch][block][H_kv][d] block V per step  */
  const void *done_k;   /* [batch][block][H_kv][d] completed block's K  */
  const void *done_v;   /* [batch][block][H_kv][d] completed block's V  */
  const void *q_next;   /* [batch][block][H_q][d] next block's selection queries */
  void *out;            /* step t's output at out + t*out_step_stride     */
  int64_t out_step_stride; /* elements; 0 = every step overwrites out     */
  int32_t dense;        /* nonzero: this layer keeps exact attention over its
                           full cache (the paper keeps its first layers so,
                           sec. IV-B.2); it has no pools and no selection  */
  /* Draft-based lookahead (sec. IV-A.1, sec. IV-B.2): NULL q_draft = none.
   * With a draft, step 1 is the 2B-token step: the draft group (q_draft over
   * the same context, with draft_k/draft_v as its own block KV) runs beside
   * the denoising group, and the next block's selection waits for it and
   * takes draft_k as a normalisation tail (herald_select_draft). */
  const void *q_draft;  /* [batch][block][H_q][d] draft group's queries    */
  const void *draft_k;  /* [batch][block][H_kv][d] the draft's K            */
  const void *draft_v;  /* [batch][block][H_kv][d] the draft's V            */
  void *out_draft;      /* [batch][block][H_q][d] draft group's output      */
  int32_t select_x;     /* next block's representative query: 0 the mean of
                           q_next, 1 its centre row (the paper's choice)     */
} herald_layer;

/* Workspace bytes needed by herald_decode_block (0 if invalid). */
size_t herald_decode_block_workspace(const herald_heads *heads,
                                     int32_t batch, int32_t block,
                                     int64_t max_seq_len, int32_t k_max);

/*
 * One block n over num_layers layers as the dual-stream pipeline of
 * sec. IV-B.1-2, on one GPU:
 *   s_retr: for every layer, select the next block's entries from the
 *           prefix before block n (seq_lens = S_n, the draft-lookahead
 *           schedule of sec. IV-A.1) with q_next, and gather them into
 *           rows [0, k_b) of the idle pool;
 *   s_main: for t < steps, for every layer, block attention of q_steps[t]
 *           over the active pool (n_active[b] rows) plus blk_k/blk_v[t];
 *   join:   s_main waits for s_retr; then, per layer, the completed block
 *           (done_k/done_v) is appended to the cache at rows
 *           [S_n, S_n + block) and to the idle pool at rows
 *           [k_b, k_b + block); n_idle[b] = k_b + block; seq_lens[b] += block.
 * The caller swaps active and idle for block n+1 (sec. IV-B.1). With dense
 * != 0 the main stream attends over the full cache (rows [0, S_n)) instead of
 * the pool and no selection runs (the GPU-only dense baseline); the append
 * still runs. A layer whose own dense flag is set is treated so in any case
 * (its active and idle pools are not read and may be null views).
 * Draft lookahead: if any layer has a q_draft, step 1 of those layers also
 * runs their draft group (q_draft over the same context with draft_k/draft_v
 * as its block KV, output out_draft), and the retrieval stream starts only
 * after step 1 of every layer (the draft is that step's product, sec. IV-B.2
 * steps 3 and 7); each such layer's selection then takes draft_k as its
 * normalisation tail (herald_select_draft); steps must be >= 2. select_x
 * picks the representative (0: mean of q_next, 1: its centre row).
 * Everything is ordered on s_main when the call's work ends; the
 * retrieval stream first waits for work already enqueued on s_main. k_next
 * (device [batch]) is the next pool's budget; k_max bounds it and
 * k_max + block <= idle.capacity. The cache capacity must hold S_n + block.
 */
herald_status herald_decode_block(const herald_heads *heads,
                                  int32_t num_layers, int32_t batch,
                                  int32_t block, int32_t steps,
                                  const herald_layer *layers,
                                  int32_t *seq_lens, int64_t max_seq_len,
                                  const int32_t *n_active, int64_t max_active,
                                  int32_t *n_idle, const int32_t *k_next,
                                  int32_t k_max, int32_t dense, void *ws,
                                  size_t ws_bytes, hipStream_t s_main,
                                  hipStream_t s_retr);

/* Static description of a status code. */
const char *herald_status_string(herald_status status);

#ifdef __cplusplus
}
#endif

#endif /* HERALD_H */
