// Indexer scoring for decode (Section 2.1, Eq. 3: I = Q_idx K_idx^T, one head
// of width 256 held as 4 x 64).
//
// The pass is bound by HBM: every token contributes one 512-byte index key and
// 256 multiply-adds.  Layout of the work:
//   * one workgroup = 4 waves = 128 consecutive tokens of one query row;
//   * a half-wave (32 lanes x 16 bytes) reads one token's 512-byte key, so each
//     load instruction of a wave moves 1 KiB of contiguous HBM; a wave keeps 16
//     such loads (16 KiB) in flight;
//   * each lane dots its 8 bf16 with the matching 8 query values
//     (v_dot2_f32_bf16, fp32 accumulate), then a transpose-reduction over the
//     32 lanes of the half-wave turns 16 partial sums per lane into one full
//     score per lane pair with 16 cross-lane exchanges instead of 16 x 5;
//   * optionally the workgroup also counts the top 8 bits of each score's
//     order-preserving key in LDS and adds the non-empty bins to a per-row
//     histogram, which lets the top-k skip one full pass over the scores.
// Index keys are read with non-temporal loads so that streaming them does not
// evict the K/V rows the attention layers reuse from the caches.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

struct IndexArgs {
    const uint16_t *q_idx;
    const uint16_t *k_idx;
    const int32_t *page_table;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    float *scores;
    uint32_t *hist;
    int n_q, max_len, page_shift, max_pages, causal, tiles_per_row;
};

constexpr int kIdxWidth = 256;  // d_idx in bf16 elements (512 bytes per token)

template <bool HIST>
__global__ __launch_bounds__(256) void index_decode_kernel(IndexArgs a) {
    __shared__ uint32_t hist_s[kCoarseBins];
    const int row = blockIdx.x / a.tiles_per_row;
    const int tile = blockIdx.x - row * a.tiles_per_row;
    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int tile0 = tile * kIndexTile;
    if (tile0 >= n) return;  // uniform over the workgroup

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int half = lane >> 5, sub = lane & 31;
    if (HIST) {
        hist_s[threadIdx.x] = 0u;  // 256 threads, 256 bins
        __syncthreads();
    }

    const uint4 qv = *reinterpret_cast<const uint4 *>(a.q_idx + (size_t)row * kIdxWidth + sub * 8);
    const int tok0 = tile0 + wave * 32;
    uint4 kv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int tok = tok0 + 2 * i + half;
        if (tok < n) {
            const size_t off = token_offset(a.page_table, a.page_shift, a.max_pages, a.max_len, b,
                                            tok, kIdxWidth);
            kv[i] = load16_nt(a.k_idx + off + sub * 8);
        } else {
            kv[i] = make_uint4(0u, 0u, 0u, 0u);
        }
    }

    float p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = dot8_bf16(kv[i], qv, 0.0f);

    // Transpose-reduce over the 32 lanes of this half-wave.  At the exchange
    // with lane ^ m a lane keeps the half of its values selected by (sub & m)
    // and adds the partner's copy of the same half, so after the four halving
    // steps lane `sub` holds token slot (sub >> 1) summed over 16 lanes, and
    // the last exchange completes the sum over all 32.
#pragma unroll
    for (int v = 0; v < 8; ++v) {
        const bool up = sub & 16;
        const float keep = up ? p[v + 8] : p[v], send = up ? p[v] : p[v + 8];
        p[v] = keep + __shfl_xor(send, 16);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const bool up = sub & 8;
        const float keep = up ? p[v + 4] : p[v], send = up ? p[v] : p[v + 4];
        p[v] = keep + __shfl_xor(send, 8);
    }
#pragma unroll
    for (int v = 0; v < 2; ++v) {
        const bool up = sub & 4;
        const float keep = up ? p[v + 2] : p[v], send = up ? p[v] : p[v + 2];
        p[v] = keep + __shfl_xor(send, 4);
    }
    {
        const bool up = sub & 2;
        const float keep = up ? p[1] : p[0], send = up ? p[0] : p[1];
        p[0] = keep + __shfl_xor(send, 2);
    }
    p[0] += __shfl_xor(p[0], 1);

    const int slot = (sub >> 1) & 15;
    const int tok = tok0 + 2 * slot + half;
    if (!(sub & 1) && tok < n) {
        a.scores[(size_t)row * a.max_len + tok] = p[0];
        if (HIST) atomicAdd(&hist_s[score_key(p[0]) >> 24], 1u);
    }
    if (HIST) {
        __syncthreads();
        const uint32_t c = hist_s[threadIdx.x];
        if (c) atomicAdd(&a.hist[(size_t)row * kCoarseBins + threadIdx.x], c);
    }
}

hipError_t launch_index_scores(const Geometry &g, const void *q_idx, const void *k_idx,
                               const int32_t *page_table, const int32_t *seq_lens,
                               const int32_t *q_pos, float *scores, uint32_t *coarse_hist,
                               hipStream_t stream) {
    IndexArgs a;
    a.q_idx = static_cast<const uint16_t *>(q_idx);
    a.k_idx = static_cast<const uint16_t *>(k_idx);
    a.page_table = page_table;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.scores = scores;
    a.hist = coarse_hist;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.causal = g.causal;
    a.tiles_per_row = div_up(g.max_len, kIndexTile);
    const size_t blocks = (size_t)g.rows * a.tiles_per_row;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    if (coarse_hist)
        index_decode_kernel<true><<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(a);
    else
        index_decode_kernel<false><<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace clsa
