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

// Tokens scored by one indexer workgroup (4 waves x 32 tokens).
constexpr int kIndexTile = 128;
// Bins of the coarse score histogram made by the indexer (top 8 key bits).
constexpr int kCoarseBins = 256;
// Selected tokens handled by one sparse-attention workgroup.
constexpr int kAttnSplit = 64;
// Candidate list capacity of the per-row top-k kernel (entries of 8 bytes).
constexpr int kTopkCandCap = 8192;

__host__ __device__ inline int div_up(int a, int b) { return (a + b - 1) / b; }

// ---- index_decode.hip ----
hipError_t launch_index_scores(const Geometry &g, const void *q_idx, const void *k_idx,
                               const int32_t *page_table, const int32_t *seq_lens,
                               const int32_t *q_pos, float *scores, uint32_t *coarse_hist,
                               hipStream_t stream);

// ---- topk.hip ----
// coarse_hist: [rows, kCoarseBins] made by launch_index_scores, or NULL to have
// the top-k kernel build it itself.
hipError_t launch_topk(const Geometry &g, const float *scores, const int32_t *seq_lens,
                       const int32_t *q_pos, const uint32_t *coarse_hist, int32_t *idx,
                       int32_t *n_sel, hipStream_t stream);
hipError_t launch_zero_u32(uint32_t *p, size_t n, hipStream_t stream);
size_t topk_lds_bytes(int max_len);

// ---- sparse_attn.hip ----
size_t attn_partial_floats(const Geometry &g);
hipError_t launch_sparse_attn(const Geometry &g, const void *q, const void *k_cache,
                              const void *v_cache, const int32_t *page_table,
                              const int32_t *idx, const int32_t *n_sel, void *out, float *lse,
                              float *partials, hipStream_t stream);

}  // namespace clsa
