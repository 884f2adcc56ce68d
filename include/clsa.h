/*
 * libclsa -- MI355X (gfx950) kernels for the decode hot path of Cross-Layer
 * Sparse Attention ("You Only Index Once: Cross-Layer Sparse Attention with
 * Shared Routing").
 *
 * The path: one indexer pass scores the current query against every cached
 * token's index key (Section 2.1, Eq. 3, I = Q_idx K_idx^T), one token-level
 * top-k is taken (Eq. 3, S_t = TopK(I_t, k)), and every cross-decoder layer
 * attends only to the selected rows of the one shared KV cache (Eq. 4,
 * O_t = Attn(Q_t, K_{S_t}, V_{S_t})), reusing the same S_t (Section 2.1, last
 * paragraph; Section 2.3: top-k is computed once per step).
 *
 * Conventions for every entry point
 *   - All tensor arguments are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or retains them.  bfloat16 tensors are passed as
 *     void* and must be 16-byte aligned; int32/float tensors 4-byte aligned.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Every call only
 *     enqueues work on that stream and returns without synchronising; errors
 *     inside kernels are not reported back.
 *   - `ws` is caller-owned device scratch of at least clsa_workspace_bytes()
 *     bytes, 256-byte aligned.  Its contents need not be initialised and are
 *     undefined afterwards.  Two calls that overlap in time must not share one
 *     workspace.
 *   - Arguments are validated on the host before anything is enqueued; on any
 *     error nothing is enqueued.  No C++ exception crosses this interface.
 *   - Device-side values are trusted within documented ranges: seq_lens[b] is
 *     clamped to [0, max_len] and n_sel[r] (an input of clsa_sparse_attn) to
 *     [0, top_k], and a value outside its range raises a device error bit that
 *     clsa_get_device_error() reports; q_pos (causal) limits row (b,t) to keys
 *     j <= q_pos[b,t]; page_table entries for pages that hold valid tokens
 *     must be valid physical page numbers (they are not range-checked).
 *   - Thread safety: entry points may be called concurrently from several host
 *     threads (each with its own workspace and outputs).  The library keeps no
 *     mutable state shared between calls except a per-device cache of one
 *     device property (filled atomically) and the device error bits; the
 *     profiling hook (clsa_set_phase_events) is per host thread.
 *
 * Tensor layouts (row-major, R = batch * n_q query rows, row r = b * n_q + t):
 *   q_idx       bf16 [batch, n_q, idx_heads, idx_dim]   index query (Eq. 2)
 *   k_idx       bf16 [batch, max_len, idx_heads, idx_dim]          contiguous
 *               bf16 [num_pages, page_size, idx_heads, idx_dim]    paged
 *   k_cache,    bf16 [batch, max_len, kv_heads, head_dim]          contiguous
 *   v_cache     bf16 [num_pages, page_size, kv_heads, head_dim]    paged
 *   page_table  int32 [batch, max_pages]: physical page of logical page p of
 *               sequence b; shared by k_idx, k_cache and v_cache (the routing
 *               index is bound to the shared KV cache, Section 2.1)
 *   seq_lens    int32 [batch]: cached tokens per sequence (incl. the current one)
 *   q_pos       int32 [batch, n_q]: absolute position of each query (causal only)
 *   scores      fp32 [batch, n_q, max_len]: only valid positions are written
 *   idx         int32 [batch, n_q, top_k]: selected token positions, ascending,
 *               padded with -1
 *   n_sel       int32 [batch, n_q]: min(top_k, number of valid keys)
 *   q, out      bf16 [batch, n_q, q_heads, head_dim]
 *   lse         fp32 [batch, n_q, q_heads] natural-log sum of exp of the scaled
 *               logits over S (-inf for an empty S), or NULL
 *   q_layers,   bf16 [n_layers, batch, n_q, q_heads, head_dim]
 *   out_layers
 *   lse_layers  fp32 [n_layers, batch, n_q, q_heads] or NULL
 *
 * Semantics fixed where the paper is silent
 *   - valid keys of row (b,t): j < seq_lens[b] and, when causal, j <= q_pos[b,t];
 *   - selection order: score descending, then token index ascending, i.e. ties
 *     at the k-th score go to the lowest index; -0.0 and +0.0 are equal; NaN
 *     scores are not supported;
 *   - query head h reads key/value head h / (q_heads / kv_heads) (GQA);
 *   - no positional encoding is applied on this path;
 *   - an empty S (no valid key) yields out = 0 and lse = -inf.
 *
 * Supported shapes (CLSA_ERR_UNSUPPORTED otherwise; there is no fallback):
 *   idx_heads * idx_dim == 256, head_dim == 128,
 *   q_heads / kv_heads in {1, 2, 4, 5, 8}, 1 <= top_k <= 8192,
 *   max_len <= 262144, page_size 0 or a power of two in [16, 4096];
 *   contiguous key/value caches (page_size 0): one sequence's cache below
 *   4 GiB, i.e. max_len * kv_heads * 256 bytes < 2^32 (the attention kernels
 *   address it with 32-bit offsets; the paged layout has no such limit).
 */
#ifndef CLSA_H
#define CLSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CLSA_OK = 0,
    CLSA_ERR_INVALID_ARG = -1, /* null/misaligned pointer, non-positive size, ... */
    CLSA_ERR_UNSUPPORTED = -2, /* a shape outside the compiled set               */
    CLSA_ERR_WORKSPACE = -3,   /* ws NULL or smaller than clsa_workspace_bytes()  */
    CLSA_ERR_HIP = -4,         /* the HIP runtime reported an error on enqueue   */
    CLSA_ERR_SCRATCH_LIMIT = -5 /* clsa_decode_step_noalloc: the step needs more  */
                                /* scratch than CLSA_NOALLOC_SCRATCH_BYTES        */
} clsa_status;

/* Size of the fixed per-device scratch of clsa_decode_step_noalloc. */
#define CLSA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/* Bits reported by clsa_get_device_error(). */
enum {
    CLSA_DEVERR_SEQ_LEN = 1, /* a seq_lens[b] outside [0, max_len] was clamped        */
    CLSA_DEVERR_N_SEL = 2    /* an n_sel[r] outside [0, top_k] was clamped            */
};

typedef enum {
    CLSA_OP_INDEX = 0,  /* clsa_index_scores (needs no workspace) */
    CLSA_OP_TOPK = 1,   /* clsa_topk */
    CLSA_OP_ATTN = 2,   /* clsa_sparse_attn */
    CLSA_OP_DECODE = 3, /* clsa_decode_step and clsa_decode_step_grouped */
    CLSA_OP_DENSE = 4,  /* clsa_dense_attn */
    CLSA_OP_KD_TARGET = 5, /* clsa_kd_target (size grows with n_layers) */
    CLSA_OP_KD_LOSS = 6    /* clsa_kd_loss */
} clsa_op;

typedef struct clsa_shape {
    int32_t batch;       /* B sequences                                          */
    int32_t n_q;         /* T query tokens per sequence (1 = decode)              */
    int32_t idx_heads;   /* index key stored as idx_heads blocks of idx_dim: one  */
    int32_t idx_dim;     /*   indexing head of width d_idx = idx_heads * idx_dim  */
    int32_t q_heads;     /* attention query heads                                 */
    int32_t kv_heads;    /* key/value heads of the shared cache                   */
    int32_t head_dim;    /* D                                                     */
    int32_t max_len;     /* capacity per sequence; row stride of scores and of    */
                         /*   contiguous caches; a multiple of page_size if paged */
    int32_t page_size;   /* 0 = contiguous caches, else tokens per page           */
    int32_t max_pages;   /* columns of page_table (>= max_len / page_size)        */
    int32_t top_k;       /* k                                                     */
    int32_t causal;      /* 1: row (b,t) also limited to keys j <= q_pos[b,t]     */
    float softmax_scale; /* logit scale of Eq. 4's softmax (1/sqrt(head_dim))     */
} clsa_shape;

/* Bytes of workspace `op` needs for `shape` (n_layers matters for
 * CLSA_OP_KD_TARGET only, whose statistics buffer grows with the layer count;
 * for CLSA_OP_DECODE it never changes the size: layers reuse the same buffers).
 * Returns 0 for CLSA_OP_INDEX, and also 0 when the shape is invalid or
 * unsupported (the entry point then reports the reason). */
size_t clsa_workspace_bytes(const clsa_shape *shape, int32_t op, int32_t n_layers);

/* Eq. 3, first half: scores[b,t,j] = sum_i q_idx[b,t,i] * k_idx[b,j,i] over the
 * d_idx components of the single indexing head, for every valid j; bf16 inputs,
 * fp32 products and accumulation; no scale and no nonlinearity.  page_table
 * may be NULL when page_size == 0; q_pos may be NULL unless causal. */
clsa_status clsa_index_scores(const clsa_shape *shape, const void *q_idx, const void *k_idx,
                              const int32_t *page_table, const int32_t *seq_lens,
                              const int32_t *q_pos, float *scores, void *stream);

/* Eq. 3, second half: for every row (b,t), the min(top_k, n_valid) valid
 * positions with the largest scores (ties to the lowest index), written in
 * ascending order to idx[b,t,:], padded with -1; n_sel[b,t] = their count.
 * Exact: the set is decided on the given fp32 scores with no approximation. */
clsa_status clsa_topk(const clsa_shape *shape, const float *scores, const int32_t *seq_lens,
                      const int32_t *q_pos, int32_t *idx, int32_t *n_sel, void *ws,
                      size_t ws_bytes, void *stream);

/* Eq. 4, one layer: for every row (b,t) and query head h, softmax attention of
 * q[b,t,h] over the rows idx[b,t,0..n_sel-1] of head g = h/(q_heads/kv_heads)
 * of the shared K/V cache, logits scaled by softmax_scale; fp32 math, bf16
 * out, optional fp32 lse.  idx entries beyond n_sel are ignored; entries below
 * n_sel must be valid positions (< seq_lens[b]) of sequence b. */
clsa_status clsa_sparse_attn(const clsa_shape *shape, const void *q, const void *k_cache,
                             const void *v_cache, const int32_t *page_table, const int32_t *idx,
                             const int32_t *n_sel, void *out, float *lse, void *ws,
                             size_t ws_bytes, void *stream);

/* One step of the shared-routing path (Section 2.1; Section 2.3): one indexer
 * pass and one top-k over the whole cache, then n_layers attention passes
 * in layer order, layer l using q_layers[l] and the same index set.  The index
 * set is also returned in idx / n_sel.  The scores live in the workspace. */
clsa_status clsa_decode_step(const clsa_shape *shape, const void *q_idx, const void *k_idx,
                             const void *k_cache, const void *v_cache,
                             const int32_t *page_table, const int32_t *seq_lens,
                             const int32_t *q_pos, int32_t n_layers, const void *q_layers,
                             void *out_layers, float *lse_layers, int32_t *idx, int32_t *n_sel,
                             void *ws, size_t ws_bytes, void *stream);

/* clsa_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same computation, arguments and results, but no workspace argument.  The
 * step's scratch is a fixed device array inside the library, one per device,
 * of CLSA_NOALLOC_SCRATCH_BYTES (32 MiB), held until the process ends; its
 * address is looked up on the first call on each device.  The call allocates
 * nothing and calls no allocating routine.  A shape whose step needs more
 * than that (clsa_workspace_bytes(shape, CLSA_OP_DECODE, n_layers) >
 * CLSA_NOALLOC_SCRATCH_BYTES, e.g. thousands of query rows) is rejected with
 * CLSA_ERR_SCRATCH_LIMIT before anything is enqueued.  Every call on one
 * device uses that device's one array (whatever is left in it from the last
 * call is cleared or overwritten as the step needs): calls that overlap in
 * time on one device, from any stream or thread, race and must not be made. */
clsa_status clsa_decode_step_noalloc(const clsa_shape *shape, const void *q_idx,
                                     const void *k_idx, const void *k_cache, const void *v_cache,
                                     const int32_t *page_table, const int32_t *seq_lens,
                                     const int32_t *q_pos, int32_t n_layers, const void *q_layers,
                                     void *out_layers, float *lse_layers, int32_t *idx,
                                     int32_t *n_sel, void *stream);

/* The same step with the routing refreshed every `group` layers, for measuring
 * what the shared routing saves (Section 3.4 and Appendix D compare per-layer
 * and every-few-layers routing with it): layers s*group .. s*group+group-1
 * attend over index set s, which is computed from the index query
 * q_idx + s * q_idx_group_stride and the index keys k_idx + s *
 * k_idx_group_stride (strides in bf16 elements, multiples of 8, >= 0; 0 reuses
 * the same index keys for every set).  group >= n_layers is clsa_decode_step;
 * group = 1 selects a fresh set before every layer.  idx / n_sel receive every
 * set: [n_sets, batch, n_q, top_k] / [n_sets, batch, n_q] with
 * n_sets = max(1, ceil(n_layers / group)).  Workspace: CLSA_OP_DECODE.  The
 * profiling hook's first three marks bracket the first set's index pass and
 * top-k; the fourth follows the last layer. */
clsa_status clsa_decode_step_grouped(const clsa_shape *shape, const void *q_idx,
                                     int64_t q_idx_group_stride, const void *k_idx,
                                     int64_t k_idx_group_stride, const void *k_cache,
                                     const void *v_cache, const int32_t *page_table,
                                     const int32_t *seq_lens, const int32_t *q_pos,
                                     int32_t n_layers, int32_t group, const void *q_layers,
                                     void *out_layers, float *lse_layers, int32_t *idx,
                                     int32_t *n_sel, void *ws, size_t ws_bytes, void *stream);

/* Dense GQA attention (Eq. 1 with GQA: the attention that Eq. 4 restricts to
 * S_t), for every row (b,t) and query head h over every valid key of sequence
 * b (j < seq_lens[b], and j <= q_pos[b,t] when causal), as the reference
 * point for the cost of the sparse path.  Same layouts, scale, output and lse
 * conventions as clsa_sparse_attn; top_k is not used (it must still be a valid
 * value); max_len <= 262144.  Workspace: CLSA_OP_DENSE. */
clsa_status clsa_dense_attn(const clsa_shape *shape, const void *q, const void *k_cache,
                            const void *v_cache, const int32_t *page_table,
                            const int32_t *seq_lens, const int32_t *q_pos, void *out, float *lse,
                            void *ws, size_t ws_bytes, void *stream);

/* Section 2.1, Eq. 2 for the new tokens of a step, with their cache write:
 * for every row r = (b,t) of the new hidden states h[b,t,0..d_model-1],
 *   q_idx[b,t,:]                  = h W_idx^Q             (256 values),
 *   index-key cache row of pos[r] = h W_idx^K             (256 values),
 *   key cache row of pos[r]       = h W^K, value row = h W^V (kv_heads*head_dim each),
 * where pos[b,t] is the token's absolute position in sequence b (paged caches
 * through page_table; positions outside [0, max_len) are not written to the
 * caches).  w is one bf16 matrix [512 + 2*kv_heads*head_dim, d_model]: row c
 * is the weight vector of output feature c, in the order W_idx^Q, W_idx^K,
 * W^K, W^V (each head's 128 features consecutive).  bf16 inputs, fp32 products
 * and accumulation, bf16 results rounded to nearest even.  d_model: a multiple
 * of 512 up to 8192.  Two rows must not write the same cache row.  Needs no
 * workspace. */
clsa_status clsa_project_append(const clsa_shape *shape, int32_t d_model, const void *h,
                                const void *w, const int32_t *pos, const int32_t *page_table,
                                void *q_idx, void *k_idx, void *k_cache, void *v_cache,
                                void *stream);

/* Section 2.2, Eq. 5: the distillation target of the indexer,
 *   abar[b,t,j] = 1/(n_layers*q_heads) * sum_l sum_h softmax_j(softmax_scale *
 *                 q_layers[l,b,t,h] . K[b,j,g(h)]),
 * each softmax over the valid keys j of row (b,t) (j < seq_lens[b], and
 * j <= q_pos[b,t] when causal) of the one shared key cache, g(h) =
 * h / (q_heads / kv_heads).  abar: fp32 [batch, n_q, max_len]; only the valid
 * positions of each row are written (a row without valid keys is left as it
 * is).  bf16 inputs, fp32 logits and softmax.  n_layers >= 1 and
 * softmax_scale > 0; v_cache is not read.  lse_layers: fp32
 * [n_layers, batch, n_q, q_heads], the natural-log log-sum-exp of each layer's
 * scaled logits over the row's valid keys -- what clsa_dense_attn returns as
 * lse for that layer, i.e. what the dense forward pass of the cross-decoder
 * already has -- or NULL, and the call computes them itself (one more pass
 * over every layer's logits).  Workspace: CLSA_OP_KD_TARGET with the same
 * n_layers. */
clsa_status clsa_kd_target(const clsa_shape *shape, int32_t n_layers, const void *q_layers,
                           const void *k_cache, const int32_t *page_table,
                           const int32_t *seq_lens, const int32_t *q_pos,
                           const float *lse_layers, float *abar, void *ws, size_t ws_bytes,
                           void *stream);

/* Section 2.2, Eq. 6 and its gradient.  With P = abar[b,t,:] (the target,
 * held constant: the stop-gradient of Eq. 6) and Q = softmax(I_t) over the
 * valid keys of row (b,t), I the unscaled index scores of Eq. 3 computed here
 * from q_idx and k_idx, the loss is the mean of KL(P || Q) =
 * sum_j P_j (log P_j - log Q_j) (0 log 0 = 0) over the n_rows rows that have a
 * valid key, and dL/dI_t[j] = (Q_j - P_j) / n_rows, so that
 *   dq_idx[b,t,:]            = sum_j dL/dI_t[j] k_idx[b,j,:],
 *   dk_idx row of token j    = sum_t dL/dI_t[j] q_idx[b,t,:].
 * loss: one fp32 value (0 when n_rows == 0).  dq_idx: fp32 [batch, n_q, 256],
 * every row written (zero for rows without keys).  dk_idx: fp32 with the
 * layout of the index-key cache (256 values per token, through page_table when
 * paged), written for every token j < seq_lens[b] (zero when no row sees it);
 * other rows are left as they are.  abar is read at valid positions only and
 * should be a distribution over them.  fp32 scores, softmax and products;
 * the loss is summed in double.  Workspace: CLSA_OP_KD_LOSS. */
clsa_status clsa_kd_loss(const clsa_shape *shape, const float *abar, const void *q_idx,
                         const void *k_idx, const int32_t *page_table, const int32_t *seq_lens,
                         const int32_t *q_pos, float *loss, float *dq_idx, float *dk_idx,
                         void *ws, size_t ws_bytes, void *stream);

/* Static, human-readable name of a status code. */
const char *clsa_status_string(clsa_status status);

/* Debug call for device-side range errors: *bits receives the CLSA_DEVERR_*
 * bits raised on the current device by any kernel of this library since the
 * last call (0 if none), and the bits are cleared.  Unlike every other entry
 * point it synchronises: it waits for the whole device (hipDeviceSynchronize)
 * before reading.  Calls overlapping on one device may each see a part of the
 * bits.  bits NULL: CLSA_ERR_INVALID_ARG. */
clsa_status clsa_get_device_error(uint32_t *bits);

/* Profiling hook, per host thread: it applies only to the calls made from
 * the thread that set it (a benchmarking facility, not meant for serving).  With
 * n = 4 + 2m (0 <= m <= 64) non-null hipEvent_t handles, the next
 * clsa_decode_step calls record, on the call's stream: events[0] right before
 * the indexer kernel, events[1] after it, events[2] after the top-k and
 * events[3] after the last layer; and for each layer l < m, events[4 + 2l]
 * right before the layer's sparse-attention kernel and events[5 + 2l] right
 * after it (before its split merge, if any).  clsa_kd_target records
 * events[0] before its statistics kernel, events[1] between it and the target
 * kernel and events[2] after the target kernel; clsa_kd_loss records events[0]
 * before the index scores, events[1] after them, events[2] after the loss
 * kernels and events[3] after the gradient kernels.  The handles are kept, not
 * copied: they must stay valid while the hook is on.  n == 0 (events may be
 * NULL) switches the hook off.  Any other n, or a NULL handle, is
 * CLSA_ERR_INVALID_ARG and leaves the hook as it was. */
clsa_status clsa_set_phase_events(void *const *events, int32_t n);

#ifdef __cplusplus
}
#endif

#endif /* CLSA_H */
