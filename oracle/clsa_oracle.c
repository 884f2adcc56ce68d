/*
 * CPU oracle for the CLSA shared-routing sparse attention path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * loads this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header, table or helper with the GPU
 * kernels.
 *
 * Plain, slow and meant to be checked by eye against the paper
 * ("You Only Index Once: Cross-Layer Sparse Attention with Shared Routing"):
 *   - every bfloat16 input is widened exactly to double;
 *   - every sum is accumulated in double, in plain loop order;
 *   - the top-k is a full sort, not a selection algorithm;
 *   - rows (and, for attention, query heads; for the index scores, blocks of
 *     keys) may be spread over host threads (oracle_set_threads): each such
 *     item computes and writes only its own outputs, with the same arithmetic
 *     in the same order, so the thread count never changes a result.  The
 *     loss of Eq. (6), whose sums run across rows, stays on one thread.
 *
 * Functions and the passage each follows:
 *   oracle_index_scores  Section 2.1, Eq. (3): I = Q_idx K_idx^T, one indexing
 *                        head of width d_idx = idx_heads * idx_dim (the per-token
 *                        index key is stored as idx_heads blocks of idx_dim).
 *   oracle_topk          Section 2.1, Eq. (3): S_t = TopK(I_t, k).
 *   oracle_sparse_attn   Section 2.1, Eq. (4): O_t = Attn(Q_t, K_{S_t}, V_{S_t}),
 *                        softmax attention of Eq. (1) restricted to S_t, with GQA.
 *   oracle_project       Section 2.1, Eq. (2): Q_idx = H W_idx^Q, K_idx = H W_idx^K,
 *                        and the shared K = H W^K, V = H W^V of the same hidden
 *                        states, for new tokens, with the cache row each of
 *                        them occupies.
 *   oracle_kd_target     Section 2.2, Eq. (5): the average over layers and query
 *                        heads of the attention distributions (each layer's own
 *                        scaled softmax over the row's valid keys).
 *   oracle_kd_loss       Section 2.2, Eq. (6): the mean over rows of
 *                        KL(A_bar_t || softmax(I_t)), I from Eq. (3), and its
 *                        gradient with respect to the index queries and keys
 *                        (A_bar held constant, the stop-gradient of Eq. (6)).
 *   oracle_decode_step   Section 2.1 last paragraph and Section 2.3 ("compute
 *                        top-k once"): one index pass, one top-k, then every
 *                        layer reuses the same S_t.
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes):
 *   - valid keys of row (b,t) are j < seq_lens[b], and also j <= q_pos[b,t]
 *     when causal (inclusive: the current token's cache entry exists);
 *   - the selection order is (score descending, token index ascending), so ties
 *     at the k-th score go to the lowest token index; S is written ascending,
 *     padded with -1, n_sel = min(k, |valid|);
 *   - the selection is decided on scores rounded to float32 (the precision the
 *     GPU path decides in); -0.0 and +0.0 compare equal;
 *   - query head h uses key/value head floor(h / (q_heads / kv_heads));
 *   - no positional encoding on this path; scale = softmax_scale;
 *   - an empty index set (n_sel = 0) gives output 0 and lse = -inf.
 */
#include "clsa_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* Host threads for the row / head loops (1 = plain serial loops).  Work items
 * are independent: each writes only its own outputs, with the same arithmetic
 * in the same order whatever thread runs it, so the results do not depend on
 * the thread count. */
static int g_threads = 1;

void oracle_set_threads(int n)
{
    g_threads = n < 1 ? 1 : (n > 256 ? 256 : n);
}

int oracle_get_threads(void)
{
    return g_threads;
}

typedef void (*item_fn)(void *ctx, size_t item, void *scratch);

typedef struct {
    item_fn fn;
    void *ctx;
    size_t items, stride, first, scratch_bytes;
} item_range;

static void *run_items(void *arg)
{
    const item_range *r = (const item_range *)arg;
    void *scratch = r->scratch_bytes ? malloc(r->scratch_bytes) : NULL;
    for (size_t i = r->first; i < r->items; i += r->stride)
        r->fn(r->ctx, i, scratch);
    free(scratch);
    return NULL;
}

/* fn(ctx, i, scratch) for i in [0, items); thread w takes items w, w + T, ...;
 * each thread has its own scratch buffer of scratch_bytes. */
static void for_items(size_t items, item_fn fn, void *ctx, size_t scratch_bytes)
{
    size_t nt = (size_t)g_threads;
    if (nt > items)
        nt = items;
    if (nt <= 1) {
        item_range r = {fn, ctx, items, 1, 0, scratch_bytes};
        run_items(&r);
        return;
    }
    pthread_t tid[256];
    int joined[256];
    item_range rng[256];
    for (size_t w = 0; w < nt; w++)
        rng[w] = (item_range){fn, ctx, items, nt, w, scratch_bytes};
    for (size_t w = 1; w < nt; w++)
        joined[w] = pthread_create(&tid[w], NULL, run_items, &rng[w]) == 0;
    run_items(&rng[0]);
    for (size_t w = 1; w < nt; w++) {
        if (joined[w])
            pthread_join(tid[w], NULL);
        else
            run_items(&rng[w]);  /* the thread could not start: run its share here */
    }
}

double oracle_bf16_to_double(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Element offset of token j of sequence b in a cache whose token rows hold
 * row_elems elements: contiguous [B, max_len, ...] or paged [P, page, ...]. */
static size_t token_row(const oracle_shape *s, const int32_t *page_table, int b, int j,
                        size_t row_elems)
{
    if (s->page_size == 0)
        return ((size_t)b * (size_t)s->max_len + (size_t)j) * row_elems;
    int32_t page = page_table[(size_t)b * (size_t)s->max_pages + (size_t)(j / s->page_size)];
    return ((size_t)page * (size_t)s->page_size + (size_t)(j % s->page_size)) * row_elems;
}

/* Number of valid keys of query row (b,t); the valid keys are 0..n-1. */
int oracle_valid_len(const oracle_shape *s, const int32_t *seq_lens, const int32_t *q_pos,
                     int b, int t)
{
    int n = seq_lens[b];
    if (s->causal) {
        int lim = q_pos[(size_t)b * s->n_q + t] + 1;
        if (lim < n)
            n = lim;
    }
    return n < 0 ? 0 : n;
}

/* Eq. (3), first half: s[b,t,j] = sum_i q_idx[b,t,i] * k_idx[b,j,i], i over the
 * d_idx = idx_heads*idx_dim components of the single indexing head. */
typedef struct {
    const oracle_shape *s;
    const uint16_t *q_idx, *k_idx;
    const int32_t *page_table, *seq_lens, *q_pos;
    double *scores;
} index_job;

enum { kKeyBlock = 4096 };  /* keys per work item of the index scores */

static void index_item(void *ctx, size_t item, void *scratch)
{
    (void)scratch;
    const index_job *a = (const index_job *)ctx;
    const oracle_shape *s = a->s;
    const int d_idx = s->idx_heads * s->idx_dim;
    const size_t blocks = ((size_t)s->max_len + kKeyBlock - 1) / kKeyBlock;
    const size_t r = item / blocks;
    const int b = (int)(r / (size_t)s->n_q), t = (int)(r % (size_t)s->n_q);
    const int j0 = (int)(item % blocks) * kKeyBlock;
    const uint16_t *q = a->q_idx + r * d_idx;
    double *row = a->scores + r * (size_t)s->max_len;
    int n = oracle_valid_len(s, a->seq_lens, a->q_pos, b, t);
    if (n > j0 + kKeyBlock)
        n = j0 + kKeyBlock;
    for (int j = j0; j < n; j++) {
        const uint16_t *k = a->k_idx + token_row(s, a->page_table, b, j, (size_t)d_idx);
        double acc = 0.0;
        for (int i = 0; i < d_idx; i++)
            acc += oracle_bf16_to_double(q[i]) * oracle_bf16_to_double(k[i]);
        row[j] = acc;
    }
}

void oracle_index_scores(const oracle_shape *s, const uint16_t *q_idx, const uint16_t *k_idx,
                         const int32_t *page_table, const int32_t *seq_lens,
                         const int32_t *q_pos, double *scores)
{
    index_job a = {s, q_idx, k_idx, page_table, seq_lens, q_pos, scores};
    const size_t blocks = ((size_t)s->max_len + kKeyBlock - 1) / kKeyBlock;
    for_items((size_t)s->batch * s->n_q * blocks, index_item, &a, 0);
}

typedef struct {
    float s;
    int32_t j;
} scored_token;

/* Selection order: higher score first; equal scores: lower token index first. */
static int by_score_then_index(const void *pa, const void *pb)
{
    const scored_token *a = (const scored_token *)pa, *b = (const scored_token *)pb;
    if (a->s > b->s) return -1;
    if (a->s < b->s) return 1;
    return (a->j > b->j) - (a->j < b->j);
}

static int by_int(const void *pa, const void *pb)
{
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

/* Eq. (3), second half: S = the first min(k, n) valid tokens in selection order,
 * written in ascending token order and padded with -1. */
typedef struct {
    const oracle_shape *s;
    const float *scores;
    const int32_t *seq_lens, *q_pos;
    int32_t *idx, *n_sel;
} topk_job;

static void topk_item(void *ctx, size_t r, void *scratch)
{
    const topk_job *a = (const topk_job *)ctx;
    const oracle_shape *s = a->s;
    const int k = s->top_k;
    scored_token *buf = (scored_token *)scratch;
    const int b = (int)(r / (size_t)s->n_q), t = (int)(r % (size_t)s->n_q);
    const float *row = a->scores + r * (size_t)s->max_len;
    int n = oracle_valid_len(s, a->seq_lens, a->q_pos, b, t);
    for (int j = 0; j < n; j++) {
        buf[j].s = row[j];
        buf[j].j = j;
    }
    qsort(buf, (size_t)n, sizeof *buf, by_score_then_index);
    int m = n < k ? n : k;
    int32_t *out = a->idx + r * (size_t)k;
    for (int i = 0; i < m; i++)
        out[i] = buf[i].j;
    qsort(out, (size_t)m, sizeof *out, by_int);
    for (int i = m; i < k; i++)
        out[i] = -1;
    a->n_sel[r] = m;
}

void oracle_topk(const oracle_shape *s, const float *scores, const int32_t *seq_lens,
                 const int32_t *q_pos, int32_t *idx, int32_t *n_sel)
{
    topk_job a = {s, scores, seq_lens, q_pos, idx, n_sel};
    for_items((size_t)s->batch * s->n_q, topk_item, &a,
              sizeof(scored_token) * (size_t)(s->max_len > 0 ? s->max_len : 1));
}

/* Eq. (4) with the softmax attention of Eq. (1), one layer:
 *   z_i = scale * <q[b,t,h], K[b, S_i, g]>,  w = softmax(z),
 *   out[b,t,h] = sum_i w_i V[b, S_i, g],     lse[b,t,h] = log sum_i exp(z_i),
 * with g = floor(h / (q_heads / kv_heads)). */
typedef struct {
    const oracle_shape *s;
    const uint16_t *q, *k_cache, *v_cache;
    const int32_t *page_table, *idx, *n_sel;
    double *out, *lse;
} attn_job;

static void attn_item(void *ctx, size_t item, void *scratch)
{
    const attn_job *a = (const attn_job *)ctx;
    const oracle_shape *s = a->s;
    const int D = s->head_dim, Hq = s->q_heads, Hkv = s->kv_heads, k = s->top_k;
    const int group = Hq / Hkv;
    const size_t kv_row = (size_t)Hkv * D;
    double *z = (double *)scratch;
    double *lse = a->lse;
    const size_t r = item / (size_t)Hq;
    const int h = (int)(item % (size_t)Hq);
    const int b = (int)(r / (size_t)s->n_q);
    const int32_t *S = a->idx + r * (size_t)k;
    const int m = a->n_sel[r];
    const int g = h / group;
    const uint16_t *qh = a->q + (r * Hq + h) * D;
    double *o = a->out + (r * Hq + h) * D;
    for (int e = 0; e < D; e++)
        o[e] = 0.0;
    if (m == 0) {
        if (lse) lse[r * Hq + h] = -INFINITY;
        return;
    }
    double zmax = -INFINITY;
    for (int i = 0; i < m; i++) {
        const uint16_t *kr = a->k_cache + token_row(s, a->page_table, b, S[i], kv_row) + (size_t)g * D;
        double acc = 0.0;
        for (int e = 0; e < D; e++)
            acc += oracle_bf16_to_double(qh[e]) * oracle_bf16_to_double(kr[e]);
        z[i] = s->softmax_scale * acc;
        if (z[i] > zmax)
            zmax = z[i];
    }
    double denom = 0.0;
    for (int i = 0; i < m; i++)
        denom += exp(z[i] - zmax);
    for (int i = 0; i < m; i++) {
        const double w = exp(z[i] - zmax) / denom;
        const uint16_t *vr = a->v_cache + token_row(s, a->page_table, b, S[i], kv_row) + (size_t)g * D;
        for (int e = 0; e < D; e++)
            o[e] += w * oracle_bf16_to_double(vr[e]);
    }
    if (lse) lse[r * Hq + h] = zmax + log(denom);
}

void oracle_sparse_attn(const oracle_shape *s, const uint16_t *q, const uint16_t *k_cache,
                        const uint16_t *v_cache, const int32_t *page_table, const int32_t *idx,
                        const int32_t *n_sel, double *out, double *lse)
{
    attn_job a = {s, q, k_cache, v_cache, page_table, idx, n_sel, out, lse};
    for_items((size_t)s->batch * s->n_q * s->q_heads, attn_item, &a,
              sizeof(double) * (size_t)(s->top_k > 0 ? s->top_k : 1));
}

/* One decode (or chunked-prefill) step: index once, select once, then every one
 * of the n_layers layers attends over the same S with its own query. */
void oracle_decode_step(const oracle_shape *s, const uint16_t *q_idx, const uint16_t *k_idx,
                        const uint16_t *k_cache, const uint16_t *v_cache,
                        const int32_t *page_table, const int32_t *seq_lens, const int32_t *q_pos,
                        int n_layers, const uint16_t *q_layers, double *out_layers,
                        double *lse_layers, int32_t *idx, int32_t *n_sel, double *scores)
{
    const size_t rows = (size_t)s->batch * s->n_q;
    const size_t nsc = rows * (size_t)s->max_len;
    float *s32 = (float *)malloc(sizeof(float) * (nsc > 0 ? nsc : 1));
    for (size_t i = 0; i < nsc; i++)
        scores[i] = 0.0;
    oracle_index_scores(s, q_idx, k_idx, page_table, seq_lens, q_pos, scores);
    for (size_t i = 0; i < nsc; i++)
        s32[i] = (float)scores[i];
    oracle_topk(s, s32, seq_lens, q_pos, idx, n_sel);
    free(s32);
    const size_t per_layer_q = rows * (size_t)s->q_heads * s->head_dim;
    const size_t per_layer_lse = rows * (size_t)s->q_heads;
    for (int l = 0; l < n_layers; l++)
        oracle_sparse_attn(s, q_layers + l * per_layer_q, k_cache, v_cache, page_table, idx, n_sel,
                           out_layers + l * per_layer_q,
                           lse_layers ? lse_layers + l * per_layer_lse : NULL);
}

/* Eq. (2) for the new tokens of a step: out[r, c] = sum_i h[r, i] * w[c, i],
 * with the output features' weight vectors stacked in w (rows 0..255 the index
 * query W_idx^Q, then the index key W_idx^K, then K, then V), and dest[r] the
 * cache row that token pos[r] of sequence r / n_q occupies (-1 when pos[r] is
 * outside [0, max_len)). */
void oracle_project(const oracle_shape *s, int d_model, const uint16_t *h, const uint16_t *w,
                    int n_out, const int32_t *pos, const int32_t *page_table, double *out,
                    int64_t *dest)
{
    const int rows = s->batch * s->n_q;
    for (int r = 0; r < rows; r++) {
        for (int c = 0; c < n_out; c++) {
            double acc = 0.0;
            for (int i = 0; i < d_model; i++)
                acc += oracle_bf16_to_double(h[(size_t)r * d_model + i]) *
                       oracle_bf16_to_double(w[(size_t)c * d_model + i]);
            out[(size_t)r * n_out + c] = acc;
        }
        const int b = r / s->n_q;
        const int p = pos[r];
        dest[r] = (p < 0 || p >= s->max_len) ? -1 : (int64_t)token_row(s, page_table, b, p, 1);
    }
}

/* Eq. (5): abar[b,t,j] = (1 / (L * Hq)) * sum over layers l and query heads h of
 * softmax_j(scale * <q_l[b,t,h], K[b,j,g(h)]>), j over the valid keys of row
 * (b,t); positions outside them are left untouched.  q_layers [L, B, T, Hq, D]. */
typedef struct {
    const oracle_shape *s;
    int n_layers;
    const uint16_t *q_layers, *k_cache;
    const int32_t *page_table, *seq_lens, *q_pos;
    double *abar;
} target_job;

static void target_item(void *ctx, size_t r, void *scratch)
{
    const target_job *tj = (const target_job *)ctx;
    const oracle_shape *s = tj->s;
    const int n_layers = tj->n_layers;
    const int D = s->head_dim, Hq = s->q_heads, Hkv = s->kv_heads;
    const int group = Hq / Hkv;
    const size_t kv_row = (size_t)Hkv * D;
    const size_t rows = (size_t)s->batch * s->n_q;
    double *z = (double *)scratch;
    const int b = (int)(r / (size_t)s->n_q), t = (int)(r % (size_t)s->n_q);
    const int n = oracle_valid_len(s, tj->seq_lens, tj->q_pos, b, t);
    double *a = tj->abar + r * (size_t)s->max_len;
    for (int j = 0; j < n; j++)
        a[j] = 0.0;
    if (n == 0)
        return;
    for (int l = 0; l < n_layers; l++) {
        for (int h = 0; h < Hq; h++) {
            const int g = h / group;
            const uint16_t *qh = tj->q_layers + (((size_t)l * rows + r) * Hq + h) * D;
            double zmax = -INFINITY;
            for (int j = 0; j < n; j++) {
                const uint16_t *kr = tj->k_cache + token_row(s, tj->page_table, b, j, kv_row) + (size_t)g * D;
                double acc = 0.0;
                for (int e = 0; e < D; e++)
                    acc += oracle_bf16_to_double(qh[e]) * oracle_bf16_to_double(kr[e]);
                z[j] = s->softmax_scale * acc;
                if (z[j] > zmax)
                    zmax = z[j];
            }
            double denom = 0.0;
            for (int j = 0; j < n; j++)
                denom += exp(z[j] - zmax);
            for (int j = 0; j < n; j++)
                a[j] += exp(z[j] - zmax) / denom;
        }
    }
    for (int j = 0; j < n; j++)
        a[j] /= (double)n_layers * (double)Hq;
}

void oracle_kd_target(const oracle_shape *s, int n_layers, const uint16_t *q_layers,
                      const uint16_t *k_cache, const int32_t *page_table,
                      const int32_t *seq_lens, const int32_t *q_pos, double *abar)
{
    target_job a = {s, n_layers, q_layers, k_cache, page_table, seq_lens, q_pos, abar};
    for_items((size_t)s->batch * s->n_q, target_item, &a,
              sizeof(double) * (size_t)(s->max_len > 0 ? s->max_len : 1));
}

/* Eq. (6) and its gradient.  For every row with at least one valid key,
 * P = abar (the target, held constant) and Q = softmax(I_t) over the valid keys,
 * I_t[j] = <q_idx[b,t], k_idx[b,j]> (Eq. 3, unscaled); the loss is the mean over
 * those rows of KL(P || Q) = sum_j P_j (log P_j - log Q_j), with 0 log 0 = 0.
 * dL/dI_t[j] = (Q_j - P_j) / n_rows, and by the chain rule
 *   dq_idx[b,t] = sum_j dL/dI_t[j] k_idx[b,j],   dk_idx[b,j] = sum_t dL/dI_t[j] q_idx[b,t].
 * dk_idx has the index-key cache's layout; its rows for positions j < seq_lens[b]
 * are written (zero when no row sees j), the others are left untouched. */
void oracle_kd_loss(const oracle_shape *s, const double *abar, const uint16_t *q_idx,
                    const uint16_t *k_idx, const int32_t *page_table, const int32_t *seq_lens,
                    const int32_t *q_pos, double *loss, double *dq_idx, double *dk_idx)
{
    const int d = s->idx_heads * s->idx_dim;
    double *sc = (double *)malloc(sizeof(double) * (size_t)(s->max_len > 0 ? s->max_len : 1));
    int n_rows = 0;
    for (int b = 0; b < s->batch; b++)
        for (int t = 0; t < s->n_q; t++)
            if (oracle_valid_len(s, seq_lens, q_pos, b, t) > 0)
                n_rows++;
    for (int b = 0; b < s->batch; b++)
        for (int j = 0; j < seq_lens[b] && j < s->max_len; j++) {
            double *dk = dk_idx + token_row(s, page_table, b, j, (size_t)d);
            for (int e = 0; e < d; e++)
                dk[e] = 0.0;
        }
    double total = 0.0;
    for (int b = 0; b < s->batch; b++) {
        for (int t = 0; t < s->n_q; t++) {
            const size_t r = (size_t)b * s->n_q + t;
            const int n = oracle_valid_len(s, seq_lens, q_pos, b, t);
            double *dq = dq_idx + r * (size_t)d;
            for (int e = 0; e < d; e++)
                dq[e] = 0.0;
            if (n == 0)
                continue;
            const uint16_t *qr = q_idx + r * (size_t)d;
            double smax = -INFINITY;
            for (int j = 0; j < n; j++) {
                const uint16_t *kr = k_idx + token_row(s, page_table, b, j, (size_t)d);
                double acc = 0.0;
                for (int e = 0; e < d; e++)
                    acc += oracle_bf16_to_double(qr[e]) * oracle_bf16_to_double(kr[e]);
                sc[j] = acc;
                if (acc > smax)
                    smax = acc;
            }
            double denom = 0.0;
            for (int j = 0; j < n; j++)
                denom += exp(sc[j] - smax);
            const double lse = smax + log(denom);
            const double *p = abar + r * (size_t)s->max_len;
            for (int j = 0; j < n; j++) {
                if (p[j] > 0.0)
                    total += p[j] * (log(p[j]) - (sc[j] - lse));
                const double g = (exp(sc[j] - lse) - p[j]) / (double)n_rows;
                const uint16_t *kr = k_idx + token_row(s, page_table, b, j, (size_t)d);
                double *dk = dk_idx + token_row(s, page_table, b, j, (size_t)d);
                for (int e = 0; e < d; e++) {
                    dq[e] += g * oracle_bf16_to_double(kr[e]);
                    dk[e] += g * oracle_bf16_to_double(qr[e]);
                }
            }
        }
    }
    *loss = n_rows > 0 ? total / (double)n_rows : 0.0;
    free(sc);
}
