/*
 * HERALD reference oracle: plain, slow, fp64 CPU implementation of the
 * sparse block-dLLM decode hot path. TEST INFRASTRUCTURE ONLY: it is used by
 * the tests, the smoke check and the CPU-baseline leg of the benchmark, and
 * never by the product library. It shares no code with the GPU path.
 *
 * Every input element (fp32, bf16 or fp64) is first decoded exactly to fp64;
 * all arithmetic is fp64 with libm exp/sqrt, written as the definitions read,
 * with no blocking, fusion or reordering.
 *
 * What each function follows:
 *   herald_oracle_budget   per-KV-head budget k from a fraction of the prefix
 *                          length (sec. IV-B.4 defines k per KV head; the
 *                          rounding rule is a reading, half-up).
 *   herald_oracle_select   representative-query selection (sec. IV-A.2) with
 *                          the mean of the block's queries as the
 *                          representative, scores over every prefix entry,
 *                          per-query-head softmax statistics (m_g, l_g) and
 *                          the GQA importance vector
 *                          s_hat_h[s] = sum_g exp(s[g,s]-m_g)/l_g followed by
 *                          one top-k per KV head (sec. IV-B.4). Ties go to the
 *                          lower index; the output is in ascending index order.
 *   herald_oracle_select_xq
 *                          selection with x query rows of the block used as
 *                          they are: the x rows centred in the block, rows
 *                          floor((B-x)/2) .. floor((B-x)/2)+x-1, each with its
 *                          own softmax statistics per query head, and the
 *                          importance summed over all x*G softmax-normalised
 *                          score rows (the G-sum of sec. IV-B.4 extended over
 *                          query rows; the paper gives no rule for x > 1, this
 *                          is a reading). x = 1 is the centre [MASK] query of
 *                          sec. IV-A.2 (Eq. 2 is minimised by the row nearest
 *                          the block centre; for even B the two middle rows
 *                          tie and the lower is taken); x = B uses every
 *                          query of the block. Same top-k and tie rule.
 *   herald_oracle_select_draft
 *                          the selection of block n+1 with block n's draft KV
 *                          appended for normalisation (sec. IV-B.2, steps 7
 *                          and 8): the representative is the mean of the
 *                          block's queries (x = 0) or the x centred rows; the
 *                          draft rows' scores enter every score row's softmax
 *                          statistics (m, l) but the draft rows are never
 *                          candidates, since the completed block replaces
 *                          them (a reading: the paper appends the draft to
 *                          the pool it ranks). Optionally also the attention
 *                          output of every score row over cache and draft,
 *                          o = sum_s exp(z[s]-m)/l v_s (the running output o_g
 *                          that the paper's fused selection kernel keeps,
 *                          sec. IV-B.4).
 *   herald_oracle_gather   copy of the selected K/V rows into a dense pool
 *                          (sec. IV-B.3, the gather of the selected entries).
 *   herald_oracle_attn     B-query GQA attention of a block over a context
 *                          (the sparse pool or the full prefix) plus the
 *                          block's own KV, no mask: bidirectional inside the
 *                          block, the context is all prefix (sec. II-A).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* element types of the raw input buffers */
enum { OR_F32 = 0, OR_BF16 = 1, OR_F64 = 2 };

/* Exact decode of one element to fp64. bf16 is the top half of an fp32. */
static double load_elem(const void *p, int type, int64_t i) {
  if (type == OR_F64) return ((const double *)p)[i];
  if (type == OR_F32) return (double)((const float *)p)[i];
  uint32_t bits = ((uint32_t)((const uint16_t *)p)[i]) << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

static size_t elem_size(int type) {
  return type == OR_F64 ? 8 : (type == OR_F32 ? 4 : 2);
}

/* Threads the OpenMP loops below run on. */
int herald_oracle_threads(void) { return omp_get_max_threads(); }

/* Sets the threads of the OpenMP loops (n >= 1), e.g. 1 to time one core. */
void herald_oracle_set_threads(int n) { omp_set_num_threads(n < 1 ? 1 : n); }

int64_t herald_oracle_budget(int64_t S, int64_t num, int64_t den) {
  /* k = clamp(floor(S*num/den + 1/2), 1, S) evaluated exactly in integers */
  if (S <= 0 || den <= 0 || num < 0) return 0;
  int64_t k = (S * num + den / 2) / den;
  if (k < 1) k = 1;
  if (k > S) k = S;
  return k;
}

typedef struct {
  double key;
  int64_t idx;
} ranked;

/* total order: larger importance first, lower index first on equal values */
static int cmp_rank(const void *a, const void *b) {
  const ranked *x = (const ranked *)a, *y = (const ranked *)b;
  if (x->key > y->key) return -1;
  if (x->key < y->key) return 1;
  return (x->idx < y->idx) ? -1 : (x->idx > y->idx);
}

static int cmp_i32(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

/* one top-k per KV head: the first k under (importance desc, index asc),
 * written in ascending index order */
static void topk_ascending(ranked *r, int64_t S, int64_t k, int32_t *out) {
  qsort(r, (size_t)S, sizeof(ranked), cmp_rank);
  for (int64_t j = 0; j < k; ++j) out[j] = (int32_t)r[j].idx;
  qsort(out, (size_t)k, sizeof(int32_t), cmp_i32);
}

/*
 * One sequence. q_sel [B][Hq][d]; K [Hkv][S][d] (row s of head h at
 * (h*S + s)*d). Writes s_hat [Hkv][S] (if non-NULL), and idx [Hkv][k]
 * (ascending). Query head hq belongs to KV head hq / (Hq/Hkv).
 * Returns 0 on success, -1 on bad arguments or allocation failure.
 */
int herald_oracle_select(int B, int Hq, int Hkv, int d, int64_t S,
                         const void *q_sel, int q_type, const void *K,
                         int k_type, int64_t k, double *s_hat_out,
                         double *m_out, double *l_out, int32_t *idx_out) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || S < 1 || k < 1 ||
      k > S)
    return -1;
  const int G = Hq / Hkv;
  const double scale = 1.0 / sqrt((double)d);
  int fail = 0;

#pragma omp parallel for schedule(dynamic) reduction(| : fail)
  for (int h = 0; h < Hkv; ++h) {
    double *qbar = (double *)malloc(sizeof(double) * (size_t)G * d);
    double *z = (double *)malloc(sizeof(double) * (size_t)G * S);
    double *m = (double *)malloc(sizeof(double) * G);
    double *l = (double *)malloc(sizeof(double) * G);
    ranked *r = (ranked *)malloc(sizeof(ranked) * (size_t)S);
    if (!qbar || !z || !m || !l || !r) {
      fail = 1;
      free(qbar); free(z); free(m); free(l); free(r);
      continue;
    }
    /* representative query: mean of the B block queries of each head */
    for (int g = 0; g < G; ++g) {
      const int hq = h * G + g;
      for (int e = 0; e < d; ++e) {
        double acc = 0.0;
        for (int i = 0; i < B; ++i)
          acc += load_elem(q_sel, q_type, ((int64_t)i * Hq + hq) * d + e);
        qbar[g * d + e] = acc / (double)B;
      }
    }
    /* raw scores s[g,s] = scale * <qbar_g, k_s> over every prefix entry */
    for (int g = 0; g < G; ++g)
      for (int64_t s = 0; s < S; ++s) {
        double acc = 0.0;
        for (int e = 0; e < d; ++e)
          acc += qbar[g * d + e] *
                 load_elem(K, k_type, ((int64_t)h * S + s) * d + e);
        z[g * S + s] = acc * scale;
      }
    /* softmax statistics per query head */
    for (int g = 0; g < G; ++g) {
      double mx = -INFINITY;
      for (int64_t s = 0; s < S; ++s)
        if (z[g * S + s] > mx) mx = z[g * S + s];
      double sum = 0.0;
      for (int64_t s = 0; s < S; ++s) sum += exp(z[g * S + s] - mx);
      m[g] = mx;
      l[g] = sum;
      if (m_out) m_out[h * G + g] = mx;
      if (l_out) l_out[h * G + g] = sum;
    }
    /* GQA importance: sum over the group of softmax-normalised scores */
    for (int64_t s = 0; s < S; ++s) {
      double acc = 0.0;
      for (int g = 0; g < G; ++g) acc += exp(z[g * S + s] - m[g]) / l[g];
      r[s].key = acc;
      r[s].idx = s;
      if (s_hat_out) s_hat_out[(int64_t)h * S + s] = acc;
    }
    topk_ascending(r, S, k, idx_out + (int64_t)h * k);
    free(qbar); free(z); free(m); free(l); free(r);
  }
  return fail ? -1 : 0;
}

/*
 * One sequence, x query rows. Shapes as herald_oracle_select; 1 <= x <= B.
 * Writes s_hat [Hkv][S] (if non-NULL) and idx [Hkv][k] (ascending).
 */
int herald_oracle_select_xq(int B, int x, int Hq, int Hkv, int d, int64_t S,
                            const void *q_sel, int q_type, const void *K,
                            int k_type, int64_t k, double *s_hat_out,
                            int32_t *idx_out) {
  if (B < 1 || x < 1 || x > B || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 ||
      S < 1 || k < 1 || k > S)
    return -1;
  const int G = Hq / Hkv;
  const int c0 = (B - x) / 2; /* first row of the centred window */
  const int V = x * G;        /* score rows: query row i, head g -> v = i*G+g */
  const double scale = 1.0 / sqrt((double)d);
  int fail = 0;

#pragma omp parallel for schedule(dynamic) reduction(| : fail)
  for (int h = 0; h < Hkv; ++h) {
    double *z = (double *)malloc(sizeof(double) * (size_t)V * S);
    double *m = (double *)malloc(sizeof(double) * V);
    double *l = (double *)malloc(sizeof(double) * V);
    ranked *r = (ranked *)malloc(sizeof(ranked) * (size_t)S);
    if (!z || !m || !l || !r) {
      fail = 1;
      free(z); free(m); free(l); free(r);
      continue;
    }
    /* raw scores of every window row and head over every prefix entry */
    for (int i = 0; i < x; ++i)
      for (int g = 0; g < G; ++g) {
        const int v = i * G + g, hq = h * G + g;
        const int64_t q0 = ((int64_t)(c0 + i) * Hq + hq) * d;
        for (int64_t s = 0; s < S; ++s) {
          double acc = 0.0;
          for (int e = 0; e < d; ++e)
            acc += load_elem(q_sel, q_type, q0 + e) *
                   load_elem(K, k_type, ((int64_t)h * S + s) * d + e);
          z[(int64_t)v * S + s] = acc * scale;
        }
      }
    /* softmax statistics of every score row */
    for (int v = 0; v < V; ++v) {
      double mx = -INFINITY;
      for (int64_t s = 0; s < S; ++s)
        if (z[(int64_t)v * S + s] > mx) mx = z[(int64_t)v * S + s];
      double sum = 0.0;
      for (int64_t s = 0; s < S; ++s) sum += exp(z[(int64_t)v * S + s] - mx);
      m[v] = mx;
      l[v] = sum;
    }
    /* importance: sum over the x*G softmax-normalised score rows */
    for (int64_t s = 0; s < S; ++s) {
      double acc = 0.0;
      for (int v = 0; v < V; ++v) acc += exp(z[(int64_t)v * S + s] - m[v]) / l[v];
      r[s].key = acc;
      r[s].idx = s;
      if (s_hat_out) s_hat_out[(int64_t)h * S + s] = acc;
    }
    topk_ascending(r, S, k, idx_out + (int64_t)h * k);
    free(z); free(m); free(l); free(r);
  }
  return fail ? -1 : 0;
}

/*
 * One sequence with a normalisation tail. q_sel [B][Hq][d]; K [Hkv][S][d];
 * tail [n_tail][Hkv][d] (row t of head h at (t*Hkv + h)*d), n_tail >= 0.
 * x = 0: one score row per query head, the mean of the B queries; x >= 1:
 * the x centred rows as herald_oracle_select_xq. Writes s_hat [Hkv][S] (if
 * non-NULL) and idx [Hkv][k] (ascending), candidates 0 .. S-1 only. With
 * o_out: Vc [Hkv][S][d] (type k_type) and tail_v (type t_type, like tail)
 * give the values, and o_out [max(x,1)][Hq][d] the attention outputs.
 */
int herald_oracle_select_draft(int B, int x, int Hq, int Hkv, int d, int64_t S,
                               const void *q_sel, int q_type, const void *K,
                               int k_type, const void *tail, int t_type,
                               int64_t n_tail, int64_t k, double *s_hat_out,
                               int32_t *idx_out, const void *Vc, const void *tail_v,
                               double *o_out) {
  if (B < 1 || x < 0 || x > B || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 ||
      S < 1 || k < 1 || k > S || n_tail < 0 || (n_tail > 0 && !tail) ||
      (o_out && (!Vc || (n_tail > 0 && !tail_v))))
    return -1;
  const int G = Hq / Hkv;
  const int nrow = x == 0 ? 1 : x;   /* query rows per head */
  const int c0 = (B - nrow) / 2;     /* first row of the centred window */
  const int V = nrow * G;
  const int64_t N = S + n_tail;      /* scored rows: prefix, then the tail */
  const double scale = 1.0 / sqrt((double)d);
  int fail = 0;

#pragma omp parallel for schedule(dynamic) reduction(| : fail)
  for (int h = 0; h < Hkv; ++h) {
    double *qv = (double *)malloc(sizeof(double) * (size_t)V * d);
    double *z = (double *)malloc(sizeof(double) * (size_t)V * N);
    double *m = (double *)malloc(sizeof(double) * V);
    double *l = (double *)malloc(sizeof(double) * V);
    ranked *r = (ranked *)malloc(sizeof(ranked) * (size_t)S);
    if (!qv || !z || !m || !l || !r) {
      fail = 1;
      free(qv); free(z); free(m); free(l); free(r);
      continue;
    }
    /* the query of every score row v = i*G + g */
    for (int i = 0; i < nrow; ++i)
      for (int g = 0; g < G; ++g) {
        const int v = i * G + g, hq = h * G + g;
        for (int e = 0; e < d; ++e) {
          if (x == 0) {
            double acc = 0.0;
            for (int j = 0; j < B; ++j)
              acc += load_elem(q_sel, q_type, ((int64_t)j * Hq + hq) * d + e);
            qv[v * d + e] = acc / (double)B;
          } else {
            qv[v * d + e] = load_elem(q_sel, q_type, ((int64_t)(c0 + i) * Hq + hq) * d + e);
          }
        }
      }
    /* scores over the prefix rows, then over the tail rows */
    for (int v = 0; v < V; ++v)
      for (int64_t s = 0; s < N; ++s) {
        double acc = 0.0;
        for (int e = 0; e < d; ++e) {
          const double kv = s < S ? load_elem(K, k_type, ((int64_t)h * S + s) * d + e)
                                  : load_elem(tail, t_type, ((s - S) * Hkv + h) * d + e);
          acc += qv[v * d + e] * kv;
        }
        z[(int64_t)v * N + s] = acc * scale;
      }
    /* softmax statistics over prefix and tail */
    for (int v = 0; v < V; ++v) {
      double mx = -INFINITY;
      for (int64_t s = 0; s < N; ++s)
        if (z[(int64_t)v * N + s] > mx) mx = z[(int64_t)v * N + s];
      double sum = 0.0;
      for (int64_t s = 0; s < N; ++s) sum += exp(z[(int64_t)v * N + s] - mx);
      m[v] = mx;
      l[v] = sum;
    }
    /* importance of the prefix rows only: they are the candidates */
    for (int64_t s = 0; s < S; ++s) {
      double acc = 0.0;
      for (int v = 0; v < V; ++v) acc += exp(z[(int64_t)v * N + s] - m[v]) / l[v];
      r[s].key = acc;
      r[s].idx = s;
      if (s_hat_out) s_hat_out[(int64_t)h * S + s] = acc;
    }
    /* attention output of every score row over prefix and tail, written at
     * [v / G][h * G + v % G][e] of o_out [nrow][Hq][d] */
    if (o_out)
      for (int v = 0; v < V; ++v)
        for (int e = 0; e < d; ++e) {
          double acc = 0.0;
          for (int64_t s = 0; s < N; ++s) {
            const double vv = s < S ? load_elem(Vc, k_type, ((int64_t)h * S + s) * d + e)
                                    : load_elem(tail_v, t_type, ((s - S) * Hkv + h) * d + e);
            acc += exp(z[(int64_t)v * N + s] - m[v]) / l[v] * vv;
          }
          o_out[((int64_t)(v / G) * Hq + h * G + v % G) * d + e] = acc;
        }
    topk_ascending(r, S, k, idx_out + (int64_t)h * k);
    free(qv); free(z); free(m); free(l); free(r);
  }
  return fail ? -1 : 0;
}

/*
 * Gather of one sequence: pool[h][j][:] = K[h][idx[h][j]][:] for j < k,
 * a byte copy. K is [Hkv][S][d]; pool is [Hkv][cap][d], cap >= k.
 */
int herald_oracle_gather(int Hkv, int d, int64_t S, const void *K, int type,
                         const int32_t *idx, int64_t k, int64_t cap,
                         void *pool) {
  if (Hkv < 1 || d < 1 || k < 0 || k > cap) return -1;
  const size_t row = elem_size(type) * (size_t)d;
  for (int h = 0; h < Hkv; ++h)
    for (int64_t j = 0; j < k; ++j) {
      int64_t s = idx[(int64_t)h * k + j];
      if (s < 0 || s >= S) return -1;
      memcpy((char *)pool + ((int64_t)h * cap + j) * row,
             (const char *)K + ((int64_t)h * S + s) * row, row);
    }
  return 0;
}

/*
 * Block attention of one sequence. q [B][Hq][d]; context keys/values
 * ctx_k/ctx_v [Hkv][n_ctx][d] (row stride d, head stride ctx_stride_h rows);
 * the block's own keys/values blk_k/blk_v [B][Hkv][d]. For every block row i
 * and query head hq: keys are the n_ctx context rows of KV head hq/G followed
 * by the B block rows of that head, p = softmax(scale * q . key), and
 * out[i][hq] = sum_j p_j value_j. out is fp64 [B][Hq][d].
 */
int herald_oracle_attn(int B, int Hq, int Hkv, int d, int64_t n_ctx,
                       int64_t ctx_stride_h, const void *q, int q_type,
                       const void *ctx_k, const void *ctx_v, int kv_type,
                       const void *blk_k, const void *blk_v, int blk_type,
                       double *out) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || n_ctx < 0 ||
      ctx_stride_h < n_ctx)
    return -1;
  const int G = Hq / Hkv;
  const double scale = 1.0 / sqrt((double)d);
  const int64_t nkeys = n_ctx + B;
  int fail = 0;

#pragma omp parallel for collapse(2) schedule(dynamic) reduction(| : fail)
  for (int i = 0; i < B; ++i)
    for (int hq = 0; hq < Hq; ++hq) {
      const int h = hq / G;
      double *logit = (double *)malloc(sizeof(double) * (size_t)nkeys);
      double *qv = (double *)malloc(sizeof(double) * (size_t)d);
      if (!logit || !qv) {
        fail = 1;
        free(logit); free(qv);
        continue;
      }
      for (int e = 0; e < d; ++e)
        qv[e] = load_elem(q, q_type, ((int64_t)i * Hq + hq) * d + e);
      for (int64_t j = 0; j < nkeys; ++j) {
        double acc = 0.0;
        for (int e = 0; e < d; ++e) {
          double kv =
              j < n_ctx
                  ? load_elem(ctx_k, kv_type, ((int64_t)h * ctx_stride_h + j) * d + e)
                  : load_elem(blk_k, blk_type,
                              ((j - n_ctx) * Hkv + h) * (int64_t)d + e);
          acc += qv[e] * kv;
        }
        logit[j] = acc * scale;
      }
      double mx = -INFINITY;
      for (int64_t j = 0; j < nkeys; ++j)
        if (logit[j] > mx) mx = logit[j];
      double den = 0.0;
      for (int64_t j = 0; j < nkeys; ++j) den += exp(logit[j] - mx);
      /* logit[] now holds the attention probabilities p_j */
      for (int64_t j = 0; j < nkeys; ++j) logit[j] = exp(logit[j] - mx) / den;
      for (int e = 0; e < d; ++e) {
        double acc = 0.0;
        for (int64_t j = 0; j < nkeys; ++j) {
          double v =
              j < n_ctx
                  ? load_elem(ctx_v, kv_type, ((int64_t)h * ctx_stride_h + j) * d + e)
                  : load_elem(blk_v, blk_type,
                              ((j - n_ctx) * Hkv + h) * (int64_t)d + e);
          acc += logit[j] * v;
        }
        out[((int64_t)i * Hq + hq) * d + e] = acc;
      }
      free(logit);
      free(qv);
    }
  return fail ? -1 : 0;
}
