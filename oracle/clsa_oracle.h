/*
 * CPU oracle for the CLSA shared-routing sparse attention path.
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * benchmark's CPU baseline; never by the product library.
 *
 * All buffers are host memory owned by the caller.  bfloat16 values are passed
 * as their uint16 bit patterns.  Layouts (row-major):
 *   q_idx   [batch, n_q, idx_heads, idx_dim]
 *   k_idx   [batch, max_len, idx_heads, idx_dim]      (page_size == 0)
 *           [pages, page_size, idx_heads, idx_dim]    (paged)
 *   k/v     [batch, max_len, kv_heads, head_dim] or [pages, page_size, kv_heads, head_dim]
 *   page_table [batch, max_pages] (physical page of each logical page)
 *   q       [batch, n_q, q_heads, head_dim]
 *   scores  [batch, n_q, max_len]   only valid positions are written
 *   idx     [batch, n_q, top_k]     ascending token indices, -1 padding
 *   n_sel   [batch, n_q]
 *   out     [batch, n_q, q_heads, head_dim]   lse [batch, n_q, q_heads]
 */
#ifndef CLSA_ORACLE_H
#define CLSA_ORACLE_H

#include <stddef.h>
#include <stdint.h>

typedef struct {
    int32_t batch, n_q;
    int32_t idx_heads, idx_dim;
    int32_t q_heads, kv_heads, head_dim;
    int32_t max_len;
    int32_t page_size, max_pages;
    int32_t top_k;
    int32_t causal;
    double softmax_scale;
} oracle_shape;

/* Host threads used by the index, top-k, attention and distillation-target
 * loops (default 1).  Results are identical for every thread count. */
void oracle_set_threads(int n);
int oracle_get_threads(void);
double oracle_bf16_to_double(uint16_t h);
int oracle_valid_len(const oracle_shape *s, const int32_t *seq_lens, const int32_t *q_pos, int b,
                     int t);
void oracle_index_scores(const oracle_shape *s, const uint16_t *q_idx, const uint16_t *k_idx,
                         const int32_t *page_table, const int32_t *seq_lens,
                         const int32_t *q_pos, double *scores);
void oracle_topk(const oracle_shape *s, const float *scores, const int32_t *seq_lens,
                 const int32_t *q_pos, int32_t *idx, int32_t *n_sel);
void oracle_sparse_attn(const oracle_shape *s, const uint16_t *q, const uint16_t *k_cache,
                        const uint16_t *v_cache, const int32_t *page_table, const int32_t *idx,
                        const int32_t *n_sel, double *out, double *lse);
void oracle_project(const oracle_shape *s, int d_model, const uint16_t *h, const uint16_t *w,
                    int n_out, const int32_t *pos, const int32_t *page_table, double *out,
                    int64_t *dest);
void oracle_kd_target(const oracle_shape *s, int n_layers, const uint16_t *q_layers,
                      const uint16_t *k_cache, const int32_t *page_table,
                      const int32_t *seq_lens, const int32_t *q_pos, double *abar);
void oracle_kd_loss(const oracle_shape *s, const double *abar, const uint16_t *q_idx,
                    const uint16_t *k_idx, const int32_t *page_table, const int32_t *seq_lens,
                    const int32_t *q_pos, double *loss, double *dq_idx, double *dk_idx);
void oracle_decode_step(const oracle_shape *s, const uint16_t *q_idx, const uint16_t *k_idx,
                        const uint16_t *k_cache, const uint16_t *v_cache,
                        const int32_t *page_table, const int32_t *seq_lens, const int32_t *q_pos,
                        int n_layers, const uint16_t *q_layers, double *out_layers,
                        double *lse_layers, int32_t *idx, int32_t *n_sel, double *scores);

#endif
