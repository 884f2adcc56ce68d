// Indexer scoring for decode (Section 2.1, Eq. 3: I = Q_idx K_idx^T, one head
// of width 256 held as 4 x 64).
//
// The pass is bound by HBM: every token contributes one 512-byte index key and
// 256 multiply-adds.  Layout of the work:
//   * one workgroup = 4 waves = up to kIndexTilesPerGroup consecutive 128-token
//     tiles of one query row (each wave takes 32 tokens of a tile);
//   * a half-wave (32 lanes x 16 bytes) reads one token's 512-byte key, so each
//     load instruction of a wave moves 1 KiB of contiguous HBM; a wave issues
//     all 16 loads of its 32 tokens (16 KiB) before it waits;
//   * each lane dots its 8 bf16 with the matching 8 query values
//     (v_dot2_f32_bf16, fp32 accumulate), then a transpose-reduction over the
//     32 lanes of the half-wave turns 16 partial sums per lane into one full
//     score per lane pair with 16 cross-lane exchanges instead of 16 x 5;
//   * optionally the workgroup also counts the top 11 bits of each score's
//     order-preserving key in LDS (quarter-octave bins) and adds the non-empty
//     bins to a per-row histogram, which lets the top-k skip a full pass.
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
    int n_q, max_len, page_shift, max_pages, causal, groups_per_row, tiles_per_group;
    uint32_t *attn_tickets;  // [rows, kv_heads], cleared here, or NULL
    int kv_heads;
};

constexpr int kIdxWidth = 256;  // d_idx in bf16 elements (512 bytes per token)
// Tiles per workgroup, fewer when the grid would otherwise leave CUs idle
// (one short sequence): each tile is one dependent memory round trip.
constexpr int kIndexTilesPerGroup = 4;
constexpr int kIndexMinGroups = 256;

// Scores of the 32 tokens tok0 .. tok0+31 of one wave.
template <bool HIST, bool PAGED>
__device__ __forceinline__ void index_tile(const IndexArgs &a, int row, int b, int n, int tok0,
                                           int half, int sub, uint4 qv, uint32_t *hist_s) {
    // All addresses first (tokens past the end are clamped to the last valid one
    // and their results dropped), then all 16 loads back to back.
    uint32_t trow[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int tok = min(tok0 + 2 * i + half, n - 1);
        if (PAGED) {
            const int page = a.page_table[(size_t)b * a.max_pages + (tok >> a.page_shift)];
            trow[i] = ((uint32_t)page << a.page_shift) + (tok & ((1 << a.page_shift) - 1));
        } else {
            trow[i] = (uint32_t)b * a.max_len + tok;
        }
    }
    uint4 kv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) kv[i] = load16_nt(a.k_idx + (size_t)trow[i] * kIdxWidth + sub * 8);
    __builtin_amdgcn_sched_barrier(0);  // keep the 16 loads together, ahead of the math

    float p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = dot8_bf16(kv[i], qv, 0.0f);

    // Transpose-reduce over the 32 lanes of this half-wave: after the four
    // halving exchanges (lane ^ 16, 8, 4, 2) lane `sub` holds token slot
    // sub >> 1 summed over 16 lanes, and the exchange with lane ^ 1 completes
    // the sum over all 32.
    transpose_reduce<16, 16, 1, 16>(p, sub);

    const int slot = (sub >> 1) & 15;
    const int tok = tok0 + 2 * slot + half;
    if (!(sub & 1) && tok < n) {
        a.scores[(size_t)row * a.max_len + tok] = p[0];
        if (HIST) atomicAdd(&hist_s[score_key(p[0]) >> kCoarseShift], 1u);
    }
}

template <bool HIST, bool PAGED>
__global__ __launch_bounds__(256) void index_decode_kernel(IndexArgs a) {
    __shared__ uint32_t hist_s[kCoarseBins];
    const int row = blockIdx.x / a.groups_per_row;
    const int grp = blockIdx.x - row * a.groups_per_row;
    const int b = row / a.n_q;
    if (a.attn_tickets && grp == 0 && (int)threadIdx.x < a.kv_heads)
        a.attn_tickets[(size_t)row * a.kv_heads + threadIdx.x] = 0u;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int tile_first = grp * a.tiles_per_group;
    if (tile_first * kIndexTile >= n) return;  // uniform over the workgroup

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int half = lane >> 5, sub = lane & 31;
    if (HIST) {
        for (int x = threadIdx.x; x < kCoarseBins; x += 256) hist_s[x] = 0u;
        __syncthreads();
    }
    const uint4 qv = *reinterpret_cast<const uint4 *>(a.q_idx + (size_t)row * kIdxWidth + sub * 8);
    const int tile_end = min(tile_first + a.tiles_per_group, div_up(n, kIndexTile));
    for (int tile = tile_first; tile < tile_end; ++tile)
        index_tile<HIST, PAGED>(a, row, b, n, tile * kIndexTile + wave * 32, half, sub, qv, hist_s);
    if (HIST) {
        __syncthreads();
        for (int x = threadIdx.x; x < kCoarseBins; x += 256) {
            const uint32_t c = hist_s[x];
            if (c) atomicAdd(&a.hist[(size_t)row * kCoarseBins + x], c);
        }
    }
}

hipError_t launch_index_scores(const Geometry &g, const void *q_idx, const void *k_idx,
                               const int32_t *page_table, const int32_t *seq_lens,
                               const int32_t *q_pos, float *scores, uint32_t *coarse_hist,
                               uint32_t *attn_tickets, hipStream_t stream) {
    IndexArgs a;
    a.attn_tickets = attn_tickets;
    a.kv_heads = g.kv_heads;
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
    const int tiles = div_up(g.max_len, kIndexTile);
    a.tiles_per_group = kIndexTilesPerGroup;
    while (a.tiles_per_group > 1 && (size_t)g.rows * div_up(tiles, a.tiles_per_group) < kIndexMinGroups)
        a.tiles_per_group /= 2;
    a.groups_per_row = div_up(tiles, a.tiles_per_group);
    const size_t blocks = (size_t)g.rows * a.groups_per_row;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)blocks), block(256);
    const bool paged = g.page_shift >= 0;
    if (coarse_hist && paged) index_decode_kernel<true, true><<<grid, block, 0, stream>>>(a);
    else if (coarse_hist) index_decode_kernel<true, false><<<grid, block, 0, stream>>>(a);
    else if (paged) index_decode_kernel<false, true><<<grid, block, 0, stream>>>(a);
    else index_decode_kernel<false, false><<<grid, block, 0, stream>>>(a);
    return hipGetLastError();
}

hipError_t take_device_error_index_decode(uint32_t *bits) { return take_source_device_error(bits); }

}  // namespace clsa
