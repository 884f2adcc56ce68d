// Internal interface between the C-ABI host code (api.cpp) and the kernel
// translation units.  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace clsa {

// Geometry shared by the kernels, resolved and checked once on the host.
struct Geometry {
    int batch, n_q, rows;          // rows = batch * n_q
    int max_len;
    int page_shift;                // log2(page_size), or -1 for contiguous caches
    int max_pages;
    int top_k;
    int causal;
    int q_heads, kv_heads, group;  // group = q_heads / kv_heads
    float softmax_scale;
};

// Longest supported sequence capacity (max_len) and largest top_k.
constexpr int kMaxLen = 262144;
constexpr int kMaxTopK = 8192;
// Tokens scored by one indexer workgroup (4 waves x 32 tokens).
constexpr int kIndexTile = 128;
// Bins of the coarse score histogram made by the indexer (top 11 key bits,
// i.e. quarter-octave bins of the score).
constexpr int kCoarseShift = 21;  // top 11 key bits: sign, exponent, 2 mantissa bits
constexpr int kCoarseBins = 1 << (32 - kCoarseShift);
// Candidate list capacity of the per-row top-k kernel (LDS entries of 8 bytes).
constexpr int kTopkCandCap = 8192;
// Rows up to which the top-k splits each row over many workgroups, when the
// rows are longer than kTopkRowMaxLen keys.
constexpr int kTopkWideMaxRows = 128;
constexpr int kTopkRowMaxLen = 16384;

__host__ __device__ inline int div_up(int a, int b) { return (a + b - 1) / b; }

// Devices for which host-side per-device tables have an entry.
constexpr int kMaxDevices = 64;

// ---- noalloc.hip ----
// Size of the fixed per-device scratch of clsa_decode_step_noalloc (covers the
// decode steps of up to 32 sequences of 65536 tokens, or 4 of 131072).
constexpr size_t kNoallocScratchBytes = (size_t)32 << 20;
// Device address of the current device's copy of that scratch (looked up once
// per device with that device current).
hipError_t noalloc_scratch(void **ptr);

// Device error bits (CLSA_DEVERR_* of clsa.h) raised by the kernels of each
// source file on the current device: OR-ed into *bits, then cleared there.
// Synchronous copies (a debug path).
hipError_t take_device_error_index_decode(uint32_t *bits);
hipError_t take_device_error_index_prefill(uint32_t *bits);
hipError_t take_device_error_topk(uint32_t *bits);
hipError_t take_device_error_sparse_attn(uint32_t *bits);
hipError_t take_device_error_kd(uint32_t *bits);

// ---- index_decode.hip ----
// coarse_hist: [rows, kCoarseBins], zero on entry, or NULL for no histogram.
// attn_tickets: [rows, kv_heads] counters of the attention that follows, set to
// zero by this launch, or NULL.
hipError_t launch_index_scores(const Geometry &g, const void *q_idx, const void *k_idx,
                               const int32_t *page_table, const int32_t *seq_lens,
                               const int32_t *q_pos, float *scores, uint32_t *coarse_hist,
                               uint32_t *attn_tickets, hipStream_t stream);

// ---- index_prefill.hip ----
// Query rows per sequence from which the indexer runs on the matrix cores.
constexpr int kPrefillMinRows = 32;
bool index_uses_mfma(const Geometry &g);
// Scores only (no coarse histogram).  attn_tickets: [rows, kv_heads] counters
// of the attention that follows, set to zero by this launch, or NULL (also for
// the sampled pass below).
hipError_t launch_index_prefill(const Geometry &g, const void *q_idx, const void *k_idx,
                                const int32_t *page_table, const int32_t *seq_lens,
                                const int32_t *q_pos, float *scores, uint32_t *attn_tickets,
                                hipStream_t stream);

// ---- two-pass chunked-prefill top-k (index_prefill.hip, topk.hip) ----
// Every kTopkSampleStride-th key of each row is scored first; the threshold of
// the candidate pass is the rank-th largest sampled score, rank =
// topk_sample_rank(g).  Used for many causal rows with top_k <= kTopkTwoPassMaxK.
constexpr int kTopkSampleStride = 32;
constexpr int kTopkTwoPassMaxK = 2048;
// Candidate slots per (row, block of kTopkKeyBlock keys) of the second pass.
// The path is chosen only where a full-length row expects at most
// kTopkBlockMean candidates per block (Poisson tail past 48: ~1e-14).
constexpr int kTopkKeyBlock = 256;
constexpr int kTopkBlockSlots = 48;
constexpr int kTopkBlockMean = 12;
inline int topk_sample_cols(const Geometry &g) { return div_up(g.max_len, kTopkSampleStride); }
inline int topk_key_blocks(const Geometry &g) { return div_up(g.max_len, kTopkKeyBlock); }
bool topk_uses_two_pass(const Geometry &g);
int topk_sample_rank(const Geometry &g);
// Pass 1: sampled scores [rows, topk_sample_cols(g)].
hipError_t launch_index_prefill_sample(const Geometry &g, const void *q_idx, const void *k_idx,
                                       const int32_t *page_table, const int32_t *seq_lens,
                                       const int32_t *q_pos, float *samples, uint32_t *attn_tickets,
                                       hipStream_t stream);
// Per-row thresholds (order-preserving keys) from the samples; also clears the
// count of the slow list (slow: [1 + rows]) that the selection fills.
hipError_t launch_topk_sample_thresh(const Geometry &g, const float *samples,
                                     const int32_t *seq_lens, const int32_t *q_pos,
                                     uint32_t *thresh, uint32_t *slow, hipStream_t stream);
// Pass 2: cand_count [rows, topk_key_blocks(g)] and cands [rows,
// topk_key_blocks(g), kTopkBlockSlots] of (key, position) pairs (every block a
// row sees gets its count written; no clearing needed).
hipError_t launch_index_prefill_emit(const Geometry &g, const void *q_idx, const void *k_idx,
                                     const int32_t *page_table, const int32_t *seq_lens,
                                     const int32_t *q_pos, const uint32_t *thresh,
                                     uint32_t *cand_count, uint32_t *cands, hipStream_t stream);
// Exact selection from the candidates; rows whose candidates do not decide
// the set go to the slow list and recompute their scores into scores
// [rows, max_len].
hipError_t launch_topk_cands(const Geometry &g, const uint32_t *cand_count, const uint32_t *cands,
                             const int32_t *seq_lens, const int32_t *q_pos, const void *q_idx,
                             const void *k_idx, const int32_t *page_table, float *scores,
                             uint32_t *slow, int32_t *idx, int32_t *n_sel, hipStream_t stream);

// ---- topk.hip ----
struct TopkWideLayout {
    int words_max, regions;  // per row: bitmap words, 1024-key candidate regions
    size_t hist_u32, bitmap_u32, cand_u32, count_u32;  // per buffer, all rows
};
struct TopkBuffers {
    uint32_t *hist;      // [rows, kCoarseBins]; zero on entry unless already filled
    uint32_t *bitmaps;   // bitmap_u32: keys above the coarse bin (wide path)
    uint32_t *cands;     // cand_u32: candidate regions (wide path)
    uint32_t *counts;    // count_u32: candidates per region (wide path)
};
bool topk_uses_wide(const Geometry &g);
bool topk_small_rows(const Geometry &g);
TopkWideLayout topk_wide_layout(const Geometry &g);
size_t topk_lds_bytes(const Geometry &g);  // LDS per workgroup of the largest top-k kernel
// hist_ready: buf.hist already holds the coarse histogram of these scores.
hipError_t launch_topk(const Geometry &g, const float *scores, const int32_t *seq_lens,
                       const int32_t *q_pos, const TopkBuffers &buf, bool hist_ready,
                       int32_t *idx, int32_t *n_sel, hipStream_t stream);
hipError_t launch_zero_u32(uint32_t *p, size_t n, hipStream_t stream);

// ---- sparse_attn.hip ----
// Partial buffer floats (0 when one split per (row, KV head)); dense: over max_len keys.
size_t attn_partial_floats(const Geometry &g, bool dense = false);
// Attention gathering K/V rows from the cache through idx (and the page table).
// split_done, if not null, is recorded right after the attention kernel, before
// the split merge.  tickets: [rows, kv_heads] arrival counters, zero on entry and
// zero again on return, or NULL; with them, grids of at most kFusedMaxSplits
// splits per (row, KV head) merge the splits inside the attention kernel.
hipError_t launch_sparse_attn(const Geometry &g, const void *q, const void *k_cache,
                              const void *v_cache, const int32_t *page_table,
                              const int32_t *idx, const int32_t *n_sel, void *out, float *lse,
                              float *partials, uint32_t *tickets, hipStream_t stream,
                              hipEvent_t split_done = nullptr);
// Dense attention of every row over all of its valid keys (seq_lens, and q_pos
// when causal), same layouts as the sparse call.
hipError_t launch_dense_attn(const Geometry &g, const void *q, const void *k_cache,
                             const void *v_cache, const int32_t *page_table,
                             const int32_t *seq_lens, const int32_t *q_pos, void *out, float *lse,
                             float *partials, hipStream_t stream);

// ---- project.hip ----
// d_model values the projection kernels support (multiples of 512 up to 8192).
bool project_supported(int d_model);
// Eq. 2 for new tokens + cache write; w: [512 + 2 * kv_heads * 128, d_model].
hipError_t launch_project(const Geometry &g, int d_model, const void *h, const void *w,
                          const int32_t *pos, const int32_t *page_table, void *q_idx,
                          void *k_idx, void *k_cache, void *v_cache, hipStream_t stream);

// ---- kd.hip ----
// Eq. 5 target: lse2 workspace of kd_target_ws_floats floats; lse_in, if not
// null, holds the natural-log log-sum-exp of every (layer, row, query head)
// and replaces the statistics pass; `between`, if not null, is recorded after
// the statistics (or import) kernel, before the target kernel.
bool kd_target_supported(const Geometry &g, int n_layers);
size_t kd_target_ws_floats(const Geometry &g, int n_layers);
hipError_t launch_kd_target(const Geometry &g, int n_layers, const void *q_layers,
                            const void *k_cache, const int32_t *page_table,
                            const int32_t *seq_lens, const int32_t *q_pos, const float *lse_in,
                            float *abar, float *lse2, hipStream_t stream,
                            hipEvent_t between = nullptr);
// Eq. 6 loss and its gradient: workspace of kd_loss_ws_floats floats; the
// events, if not null, are recorded after the index scores and after the loss.
bool kd_loss_supported(const Geometry &g);
size_t kd_loss_ws_floats(const Geometry &g);
hipError_t launch_kd_loss(const Geometry &g, const float *abar, const void *q_idx,
                          const void *k_idx, const int32_t *page_table, const int32_t *seq_lens,
                          const int32_t *q_pos, float *loss, float *dq, float *dk, float *ws,
                          hipStream_t stream, hipEvent_t after_scores = nullptr,
                          hipEvent_t after_loss = nullptr);

}  // namespace clsa
