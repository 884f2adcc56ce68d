// Indexer scoring for chunked prefill (Section 2.1, Eq. 3: I = Q_idx K_idx^T)
// on the matrix cores.  With many query rows per sequence the scores form a
// dense [T x N] contraction over d_idx = 256, masked causally (row t sees keys
// j <= q_pos[t]).
//
// MFMA mapping (v_mfma_f32_16x16x32_bf16, C[i][j] += sum_k A[i][k] B[k][j]):
//   * A = 16 index keys x 32 index dims, B = 32 dims x 16 queries, so C is
//     keys x queries.  Lane l supplies A row / B column (l & 15) for dims
//     (l >> 4) * 8 .. +8 of a 32-dim step, and receives C rows 4 * (l >> 4) + r
//     (r = 0..3) of column (l & 15): four consecutive keys of one query.
// Key-stationary work split: a workgroup owns 256 consecutive keys of one
// sequence (each of its 4 waves holds 64 of them, all 256 dims, as A operands
// in registers for the whole kernel) and streams that sequence's queries 16 at
// a time (the B operands: 8 loads of 16 bytes per lane, the next tile's loads
// issued before the current tile's products).  The keys are read from HBM
// exactly once; the queries (512 bytes each, 4 MiB for 8192 of them) are read
// by every workgroup and stay in the L2.  Query tiles whose rows all end
// before the block's first key (causal) are skipped.  The score block is
// written once, non-temporally (the top-k reads it back), which bounds the
// kernel by HBM writes (4 bytes per 512 FLOP) rather than by the matrix cores;
// each query tile's 16 x 256 scores are therefore staged in LDS and written as
// whole 1 KiB row segments (direct 16-byte stores of 64-byte row pieces
// reached only about 3 TB/s).
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kPfWaveKeys = 64;                // keys per wave (four 16-row tiles)
constexpr int kPfKeys = 4 * kPfWaveKeys;        // keys per workgroup
constexpr int kIdxDim = 256;

struct PrefillArgs {
    const uint16_t *q_idx;
    const uint16_t *k_idx;
    const int32_t *page_table;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    float *scores;
    int n_q, max_len, page_shift, max_pages, causal;
    int kblocks;      // key blocks per sequence
    int vec_store;    // max_len % 4 == 0: rows are 16-byte aligned
};

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// B operands of query tile qt: lane (col, grp) reads dims kb*32 + grp*8 .. +8
// of query qt*16 + col (clamped to the last query; extra rows are not stored).
__device__ __forceinline__ void load_queries(const PrefillArgs &a, int b, int qt, int col,
                                             int grp, bf16x8 (&qv)[8]) {
    const int t = min(qt * 16 + col, a.n_q - 1);
    const uint16_t *p = a.q_idx + ((size_t)b * a.n_q + t) * kIdxDim + grp * 8;
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) qv[kb] = load_bf16x8(p + kb * 32);
}

// Number of keys query t may see (0 past the last query).  Branch-free: the
// position load is unconditional (clamped), so no wait is placed inside a branch.
template <bool CAUSAL>
__device__ __forceinline__ int key_limit(const int32_t *qpos, int len, int n_q, int t) {
    int n = len;
    if (CAUSAL) n = min(len, max(qpos[min(t, n_q - 1)] + 1, 0));
    return t < n_q ? n : 0;
}

// LDS staging of one query tile's scores: 16 rows x the workgroup's 256 keys
// (padded rows against bank conflicts), two buffers used alternately.
constexpr int kTileStride = kPfKeys + 4;

// Scores of query tile qt against the workgroup's 256 keys.  Each wave writes
// its 16 x 64 part into the LDS tile; after a barrier each wave stores four
// whole rows (one 1 KiB row segment per store instruction).  n: key limit of
// this lane's query (qt*16 + (lane & 15)).  The early exit is uniform over the
// workgroup (every wave holds the same 16 queries); it still passes a barrier
// so that a buffer is never rewritten while another wave reads it.
__device__ __forceinline__ void score_tile(const PrefillArgs &a, const bf16x8 (&kv)[4][8],
                                           const bf16x8 (&qv)[8], int n, int b, int qt, int jg,
                                           int wave, int lane, float (*tile)[kTileStride]) {
    const int col = lane & 15, grp = lane >> 4;
    int nmax = n;
#pragma unroll
    for (int m = 8; m >= 1; m >>= 1) nmax = max(nmax, __shfl_xor(nmax, m));
    if (nmax <= jg) {  // no query of the tile reaches the workgroup's keys
        __syncthreads();
        return;
    }
    f32x4 c[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) c[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 8; ++kb)
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
            c[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv[kt][kb], qv[kb], c[kt], 0, 0, 0);
    // lane holds keys wave*64 + 16*kt + 4*grp + r (r = 0..3) of query col
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
        *reinterpret_cast<f32x4 *>(&tile[col][wave * kPfWaveKeys + 16 * kt + 4 * grp]) = c[kt];
    __syncthreads();
    const int j0 = jg + 4 * lane;  // this lane's 4 keys of every row
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rr = wave * 4 + i;
        const int nr = __builtin_amdgcn_readlane(n, rr);  // lane rr holds query rr's limit
        if (j0 >= nr) continue;
        const f32x4 v = *reinterpret_cast<const f32x4 *>(&tile[rr][4 * lane]);
        float *dst = a.scores + ((size_t)b * a.n_q + qt * 16 + rr) * a.max_len + j0;
        if (a.vec_store && j0 + 4 <= nr) {
            __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(dst));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (j0 + r < nr) dst[r] = v[r];
        }
    }
}

template <bool PAGED, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void index_prefill_kernel(PrefillArgs a) {
    const int b = blockIdx.x / a.kblocks;
    const int kblk = blockIdx.x - b * a.kblocks;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int len = clamp_len(a.seq_lens[b], a.max_len);
    const int jg = kblk * kPfKeys;                       // first key of this workgroup
    const int jw = jg + wave * kPfWaveKeys;              // first key of this wave
    if (jg >= len) return;                               // uniform over the workgroup
    __shared__ float tile[2][16][kTileStride];

    // the wave's 64 keys as A operands: key tile kt, row col = key jw + 16*kt + col
    bf16x8 kv[4][8];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        const int j = min(jw + 16 * kt + col, len - 1);  // clamped keys are never stored
        size_t off;
        if (PAGED) {
            const int page = a.page_table[(size_t)b * a.max_pages + (j >> a.page_shift)];
            off = (((size_t)page << a.page_shift) + (j & ((1 << a.page_shift) - 1))) * kIdxDim;
        } else {
            off = ((size_t)b * a.max_len + j) * kIdxDim;
        }
#pragma unroll
        for (int kb = 0; kb < 8; ++kb) kv[kt][kb] = load_bf16x8(a.k_idx + off + grp * 8 + kb * 32);
    }

    // Tile qt+1's inputs (its queries' key limits, then its queries) are loaded
    // before tile qt is computed.  The limit load is issued first: loads
    // complete in order, so waiting for it must not wait for the queries.  The
    // loop is unrolled by two so that both query buffers keep fixed registers.
    const int ntiles = div_up(a.n_q, 16);
    const int32_t *qpos = CAUSAL ? a.q_pos + (size_t)b * a.n_q : nullptr;
    bf16x8 qa[8], qb[8];
    int n_a = key_limit<CAUSAL>(qpos, len, a.n_q, col), n_b = 0;
    load_queries(a, b, 0, col, grp, qa);
    for (int qt = 0; qt < ntiles; qt += 2) {
        if (qt + 1 < ntiles) {
            n_b = key_limit<CAUSAL>(qpos, len, a.n_q, (qt + 1) * 16 + col);
            load_queries(a, b, qt + 1, col, grp, qb);
        }
        score_tile(a, kv, qa, n_a, b, qt, jg, wave, lane, tile[0]);
        if (qt + 1 >= ntiles) break;
        if (qt + 2 < ntiles) {
            n_a = key_limit<CAUSAL>(qpos, len, a.n_q, (qt + 2) * 16 + col);
            load_queries(a, b, qt + 2, col, grp, qa);
        }
        score_tile(a, kv, qb, n_b, b, qt + 1, jg, wave, lane, tile[1]);
    }
}

bool index_uses_mfma(const Geometry &g) { return g.n_q >= kPrefillMinRows; }

hipError_t launch_index_prefill(const Geometry &g, const void *q_idx, const void *k_idx,
                                const int32_t *page_table, const int32_t *seq_lens,
                                const int32_t *q_pos, float *scores, hipStream_t stream) {
    PrefillArgs a;
    a.q_idx = static_cast<const uint16_t *>(q_idx);
    a.k_idx = static_cast<const uint16_t *>(k_idx);
    a.page_table = page_table;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.scores = scores;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.causal = g.causal;
    a.kblocks = div_up(g.max_len, kPfKeys);
    a.vec_store = (g.max_len % 4) == 0;
    const size_t blocks = (size_t)g.batch * a.kblocks;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)blocks), block(256);
    const bool paged = g.page_shift >= 0;
    if (paged && g.causal) index_prefill_kernel<true, true><<<grid, block, 0, stream>>>(a);
    else if (paged) index_prefill_kernel<true, false><<<grid, block, 0, stream>>>(a);
    else if (g.causal) index_prefill_kernel<false, true><<<grid, block, 0, stream>>>(a);
    else index_prefill_kernel<false, false><<<grid, block, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace clsa
