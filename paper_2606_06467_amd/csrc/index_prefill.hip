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
// a time as B operands.  Each query tile is loaded once per workgroup (a
// quarter per wave, a tile ahead) and shared through LDS; the keys are read
// from HBM exactly once and the queries (512 bytes each, 4 MiB for 8192 of
// them) from the L2.  Query tiles whose rows all end before the block's first
// key (causal) are skipped.  The score block is written once,
// non-temporally (the top-k reads it back): each tile's 16 x 256 scores are
// staged in LDS and written as whole 1 KiB row segments (direct 16-byte stores
// of 64-byte row pieces reached only about 3 TB/s), one tile later, after the
// next wait, so that waiting for loads never waits for fresh stores.
// Three kernels share this mapping: index_prefill_kernel writes the scores
// (clsa_index_scores, the distillation loss, the top-k over full score rows)
// or, with a key stride, the sampled scores of the two-pass chunked-prefill
// top-k; index_emit_kernel is that top-k's second pass, which writes only each
// row's candidates.
#include <type_traits>

#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kPfWaveKeys = 64;                // keys per wave (four 16-row tiles)
constexpr int kPfKeys = 4 * kPfWaveKeys;        // keys per workgroup
constexpr int kIdxDim = 256;
static_assert(kPfKeys == kTopkKeyBlock, "a workgroup's keys are one candidate block");

struct PrefillArgs {
    const uint16_t *q_idx;
    const uint16_t *k_idx;
    const int32_t *page_table;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    float *scores;            // scores: [rows, row_stride]
    const uint32_t *thresh;   // candidate pass: [rows] candidate threshold (order-preserving key)
    uint32_t *cand_count;     // candidate pass: [rows, kblocks] candidates per key block (may exceed the slots)
    uint2 *cands;             // candidate pass: [rows, kblocks, kTopkBlockSlots] (key, position)
    int n_q, max_len, page_shift, max_pages, causal;
    int kblocks;      // key blocks per sequence (of sampled keys when key_stride > 1)
    int vec_store;    // row_stride % 4 == 0: rows are 16-byte aligned
    int key_stride;   // 1, or S: a block's keys are positions 0, S, 2S, ... (the sample pass)
    int row_stride;   // floats per score row
    int qsplit;       // query-tile ranges per sequence (workgroups per key block)
    uint32_t *attn_tickets;  // arrival counters of the attention that follows, cleared here, or NULL
    int n_tickets;
};

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// Number of keys query t may see (0 past the last query), in two steps so that
// the position load can be issued a tile ahead and its result used only after
// the next wait: key_pos loads the raw position (clamped index: no branch),
// key_limit turns it into the limit.
template <bool CAUSAL>
__device__ __forceinline__ int key_pos(const int32_t *qpos, int n_q, int t) {
    return CAUSAL ? qpos[min(t, n_q - 1)] : 0;
}
template <bool CAUSAL>
__device__ __forceinline__ int key_limit(int pos, int len, int n_q, int t) {
    const int n = CAUSAL ? min(len, max(pos + 1, 0)) : len;
    return t < n_q ? n : 0;
}

// Keys of the workgroup are key indices m (positions m * key_stride); a row
// that sees the first n positions sees the first ceil(n / key_stride) of them.
__device__ __forceinline__ int strided_limit(int n, int stride) {
    return stride == 1 ? n : (n + stride - 1) / stride;
}

// LDS staging of one query tile's scores: 16 rows x the workgroup's 256 keys
// (padded rows against bank conflicts), two buffers used alternately.
constexpr int kTileStride = kPfKeys + 4;
// Query tile rows in LDS: 256 bf16 + 8 of padding (528 bytes), so that the 16
// rows read by one operand load fall on different banks.
constexpr int kQStride = kIdxDim + 8;

// s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt in
// 6:4, lgkmcnt in 11:8; a field at its maximum does not wait).
constexpr int kPfWaitLgkm0 = 0xC07F;  // lgkmcnt(0)
constexpr int kPfWaitVm0 = 0x0F70;    // vmcnt(0)

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations,
// not for its global loads and stores in flight (which __syncthreads would
// also wait for), with compiler fences so that no LDS access moves across it.
__device__ __forceinline__ void pf_lds_barrier() {
    __builtin_amdgcn_s_waitcnt(kPfWaitLgkm0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Largest / smallest key limit over the 16 queries of a tile (every lane gets
// it; the same in every wave of the workgroup, which holds the same queries).
// A butterfly inside each 16-lane row with DPP operand permutes (lane ^ 1,
// lane ^ 2, then the half-row and row mirrors, which pair the quads and the
// halves), four dependent VALU steps instead of four LDS permutes.  Called
// with every lane active.
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int x) {
    return __builtin_amdgcn_mov_dpp(x, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ int tile_limit(int n) {
    n = max(n, dpp_i32<0xB1>(n));
    n = max(n, dpp_i32<0x4E>(n));
    n = max(n, dpp_i32<0x141>(n));
    return max(n, dpp_i32<0x140>(n));
}
__device__ __forceinline__ int tile_limit_min(int n) {
    n = min(n, dpp_i32<0xB1>(n));
    n = min(n, dpp_i32<0x4E>(n));
    n = min(n, dpp_i32<0x141>(n));
    return min(n, dpp_i32<0x140>(n));
}

// The fp32 threshold equivalent to an order-preserving key threshold th:
// score_key(s) >= th exactly when s >= thresh_float(th), for every non-NaN s
// (the inverse of score_key; keys below that of -inf give -inf, keys above
// that of +inf give NaN, which no score reaches).  Denormal flushing can only
// turn a strict comparison into an equality, i.e. admit more candidates.
__device__ __forceinline__ float thresh_float(uint32_t th) {
    if (th < 0x007FFFFFu) return -INFINITY;
    return __uint_as_float((th & 0x80000000u) ? (th & 0x7FFFFFFFu) : ~th);
}

// Scores of one query tile against the workgroup's 256 keys into the LDS tile:
// each wave writes its 16 x 64 part (lane holds keys wave*64 + 16*kt + 4*grp + r
// of query col).
__device__ __forceinline__ void score_tile(const bf16x8 (&kv)[4][8], const bf16x8 (&qv)[8],
                                           int wave, int lane, float (*tile)[kTileStride]) {
    const int col = lane & 15, grp = lane >> 4;
    f32x4 c[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) c[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 8; ++kb)
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
            c[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv[kt][kb], qv[kb], c[kt], 0, 0, 0);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
        *reinterpret_cast<f32x4 *>(&tile[col][wave * kPfWaveKeys + 16 * kt + 4 * grp]) = c[kt];
}

// Stores of a staged tile: each wave writes four whole rows (one 1 KiB row
// segment per store instruction).  n: key limit of this lane's query of that
// tile (lane rr holds query rr's).
__device__ __forceinline__ void store_tile(const PrefillArgs &a, const float (*tile)[kTileStride],
                                           int n, int b, int qt, int jg, int wave, int lane) {
    const int j0 = jg + 4 * lane;  // this lane's 4 keys of every row
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rr = wave * 4 + i;
        const int nr = __builtin_amdgcn_readlane(n, rr);
        if (j0 >= nr) continue;
        const f32x4 v = *reinterpret_cast<const f32x4 *>(&tile[rr][4 * lane]);
        float *dst = a.scores + ((size_t)b * a.n_q + qt * 16 + rr) * a.row_stride + j0;
        if (a.vec_store && j0 + 4 <= nr) {
            __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(dst));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (j0 + r < nr) dst[r] = v[r];
        }
    }
}

// Scores of one query tile against the wave's 64 keys, left in registers:
// c[kt][r] is key jw + 16 kt + 4 grp + r of query col.
__device__ __forceinline__ void score_regs(const bf16x8 (&kv)[4][8], const bf16x8 (&qv)[8],
                                           f32x4 (&c)[4]) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) c[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 8; ++kb)
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
            c[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv[kt][kb], qv[kb], c[kt], 0, 0, 0);
}

// Workgroup: 256 keys of one sequence against all of its query tiles.  Per
// tile qt, in this order: (a) wait for every global access issued so far --
// the tile's queries (loaded one tile ahead) and the stores of tile qt-2,
// issued a whole tile earlier; (b) store tile qt-1 from LDS; (c) load tile
// qt+1's key limits and queries; (d) products of tile qt into LDS; (e) LDS-only
// barrier.  Stores and loads both count in vmcnt and need not complete in
// order with each other, so a wait for a load also waits for every store
// before it; issuing a tile's stores only after the next tile's queries have
// arrived keeps the stores' completion out of the wait.  Tiles whose rows all
// end before the workgroup's first key (causal) compute and store nothing.
// With key_stride S > 1 (the first pass of the chunked-prefill top-k) the
// block's keys are every S-th position and the scores go to a [rows,
// row_stride] sample matrix.  Workgroups of one key block split the query
// tiles into qsplit ranges.
template <bool PAGED, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void index_prefill_kernel(PrefillArgs a) {
    const int per_seq = a.kblocks * a.qsplit;
    const int b = blockIdx.x / per_seq;
    const int kblk = (blockIdx.x - b * per_seq) / a.qsplit;
    const int qs = blockIdx.x - b * per_seq - kblk * a.qsplit;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int col = lane & 15, grp = lane >> 4;
    if (a.attn_tickets)
        for (int x = blockIdx.x * 256 + threadIdx.x; x < a.n_tickets; x += gridDim.x * 256)
            a.attn_tickets[x] = 0u;
    const int stride = a.key_stride;
    const int len_pos = clamp_len(a.seq_lens[b], a.max_len);  // positions
    const int len = strided_limit(len_pos, stride);           // keys (of this pass)
    const int jg = kblk * kPfKeys;                       // first key of this workgroup
    const int jw = jg + wave * kPfWaveKeys;              // first key of this wave
    if (jg >= len) return;                               // uniform over the workgroup
    __shared__ float tile[2][16][kTileStride];
    __shared__ __align__(16) uint16_t s_q[2][16][kQStride];  // query tiles (bf16)

    // the wave's 64 keys as A operands: key tile kt, row col = key jw + 16*kt + col
    bf16x8 kv[4][8];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        const int j = min(jw + 16 * kt + col, len - 1) * stride;  // clamped keys are never stored
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

    const int ntiles_all = div_up(a.n_q, 16);
    const int tpw = div_up(ntiles_all, a.qsplit);        // query tiles of each range
    const int qt0 = qs * tpw;
    const int qt_end = min(ntiles_all, qt0 + tpw);
    if (qt0 >= qt_end) return;                           // uniform
    const int32_t *qpos = CAUSAL ? a.q_pos + (size_t)b * a.n_q : nullptr;
    // Query tiles go through LDS, each loaded once per workgroup: wave w loads
    // queries 4w .. 4w+3 of a tile (lane: 32 bytes of query 4w + (lane >> 4)),
    // a tile ahead, and writes them to s_q after the next wait.
    const int sq_row = wave * 4 + (lane >> 4), sq_col = (lane & 15) * 16;
    u32x4 qs_v[2];
    auto load_quarter = [&](int qt) {
        const int t = min(qt * 16 + sq_row, a.n_q - 1);  // rows past n_q: never stored
        const uint16_t *p = a.q_idx + ((size_t)b * a.n_q + t) * kIdxDim + sq_col;
        qs_v[0] = *reinterpret_cast<const u32x4 *>(p);
        qs_v[1] = *reinterpret_cast<const u32x4 *>(p + 8);
    };
    auto stage_quarter = [&](int buf) {
        *reinterpret_cast<u32x4 *>(&s_q[buf][sq_row][sq_col]) = qs_v[0];
        *reinterpret_cast<u32x4 *>(&s_q[buf][sq_row][sq_col + 8]) = qs_v[1];
    };
    int p_cur = key_pos<CAUSAL>(qpos, a.n_q, qt0 * 16 + col);  // raw positions, a tile ahead
    load_quarter(qt0);
    __builtin_amdgcn_s_waitcnt(kPfWaitVm0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    stage_quarter(qt0 & 1);
    if (qt0 + 1 < qt_end) load_quarter(qt0 + 1);
    pf_lds_barrier();
    int n_prev = 0;       // key limits of the tile staged in LDS, not yet stored
    bool staged = false;
    for (int qt = qt0; qt < qt_end; ++qt) {
        int p_next = 0;
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(kPfWaitVm0);                         // (a)
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_sched_barrier(0);
        const int n_cur = strided_limit(key_limit<CAUSAL>(p_cur, len_pos, a.n_q, qt * 16 + col), stride);
        if (qt + 1 < qt_end) stage_quarter((qt + 1) & 1);               // tile qt+1's queries
        if (staged)                                                     // (b)
            store_tile(a, tile[(qt - 1) & 1], n_prev, b, qt - 1, jg, wave, lane);
        if (qt + 1 < qt_end) {                                          // (c)
            p_next = key_pos<CAUSAL>(qpos, a.n_q, (qt + 1) * 16 + col);
        }
        if (qt + 2 < qt_end) load_quarter(qt + 2);
        __builtin_amdgcn_sched_barrier(0);
        staged = tile_limit(n_cur) > jg;                                // uniform
        if (staged) {                                                   // (d)
            bf16x8 qv[8];
#pragma unroll
            for (int kb = 0; kb < 8; ++kb)
                qv[kb] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4 *>(&s_q[qt & 1][col][kb * 32 + grp * 8]));
            score_tile(kv, qv, wave, lane, tile[qt & 1]);
        }
        n_prev = n_cur;
        p_cur = p_next;
        pf_lds_barrier();                                               // (e)
    }
    if (staged) store_tile(a, tile[(qt_end - 1) & 1], n_prev, b, qt_end - 1, jg, wave, lane);
}

// The candidate pass (the second pass of the chunked-prefill top-k): the
// products of index_prefill_kernel, but instead of storing the scores each
// row's candidates (valid keys whose score is at least the row's threshold)
// go to its (row, key block) list.  Each lane decides its 16 keys of a tile in
// fp32 against the threshold turned back into a float, counts them into s_cnt,
// and after the tile's barrier takes its slots of the list: those of the
// (wave, lane group)s before it.  Each (row, key block) list is written by this
// workgroup alone, so no atomics are needed; its count is written in full (a
// count past the slots sends the row to the exact fallback of the top-k).  Two
// query tiles per step: the wait, the barrier and the candidate stores of a
// step cover 32 queries (one tile per step measured 4% slower).  Per step P (tiles qt, qt + 1): (a) wait
// for every global access so far (pair P + 1's queries, loaded a step ahead,
// and the candidate stores of step P - 2); stage pair P + 1's queries in LDS;
// (b) store pair P - 1's candidates; (c) load pair P + 1's key limits and
// thresholds and pair P + 2's queries; (d) products and candidate masks of
// pair P; (e) LDS-only barrier.  The scores of a pair wait in LDS (each lane
// reads back only its own) until its candidates are stored a step later
// (picking them out of the registers by a select chain on the slot number
// measured slower).
template <bool PAGED, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void index_emit_kernel(PrefillArgs a) {
    const int per_seq = a.kblocks * a.qsplit;
    const int b = blockIdx.x / per_seq;
    const int kblk = (blockIdx.x - b * per_seq) / a.qsplit;
    const int qs = blockIdx.x - b * per_seq - kblk * a.qsplit;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int col = lane & 15, grp = lane >> 4;
    if (a.attn_tickets)
        for (int x = blockIdx.x * 256 + threadIdx.x; x < a.n_tickets; x += gridDim.x * 256)
            a.attn_tickets[x] = 0u;
    const int len = clamp_len(a.seq_lens[b], a.max_len);
    const int jg = kblk * kPfKeys;
    const int jw = jg + wave * kPfWaveKeys;
    if (jg >= len) return;  // uniform
    __shared__ __align__(16) uint16_t s_q[2][2][16][kQStride];  // [stage][tile of the pair]
    __shared__ __align__(16) uint32_t s_cnt[2][2][16][16];      // [step parity][tile][query][wave, lane group]
    __shared__ uint32_t s_ek[2][4][16][64];                      // [tile][wave][key slot][lane]

    bf16x8 kv[4][8];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        const int j = min(jw + 16 * kt + col, len - 1);  // clamped keys are never candidates
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

    const int ntiles_all = div_up(a.n_q, 16);
    const int tpw = div_up(ntiles_all, a.qsplit);
    const int qt0 = qs * tpw;
    const int qt_end = min(ntiles_all, qt0 + tpw);
    if (qt0 >= qt_end) return;  // uniform
    const int32_t *qpos = CAUSAL ? a.q_pos + (size_t)b * a.n_q : nullptr;
    const int sq_row = wave * 4 + (lane >> 4), sq_col = (lane & 15) * 16;
    u32x4 qs_v[2][2];
    auto load_pair = [&](int qt) {  // wave w: queries 4w .. 4w+3 of tiles qt and qt + 1
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int r = min((qt + t) * 16 + sq_row, a.n_q - 1);  // past the end: never used
            const uint16_t *p = a.q_idx + ((size_t)b * a.n_q + r) * kIdxDim + sq_col;
            qs_v[t][0] = *reinterpret_cast<const u32x4 *>(p);
            qs_v[t][1] = *reinterpret_cast<const u32x4 *>(p + 8);
        }
    };
    auto stage_pair = [&](int st) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            *reinterpret_cast<u32x4 *>(&s_q[st][t][sq_row][sq_col]) = qs_v[t][0];
            *reinterpret_cast<u32x4 *>(&s_q[st][t][sq_row][sq_col + 8]) = qs_v[t][1];
        }
    };
    auto row_of = [&](int qt, int t) { return min((qt + t) * 16 + col, a.n_q - 1); };
    int p_cur[2], p_next[2] = {0, 0};
    uint32_t th_cur[2], th_next[2] = {0u, 0u};
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        p_cur[t] = key_pos<CAUSAL>(qpos, a.n_q, qt0 * 16 + 16 * t + col);
        th_cur[t] = a.thresh[(size_t)b * a.n_q + row_of(qt0, t)];
    }
    load_pair(qt0);
    __builtin_amdgcn_s_waitcnt(kPfWaitVm0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    stage_pair(0);
    if (qt0 + 2 < qt_end) load_pair(qt0 + 2);
    pf_lds_barrier();

    f32x4 e_c[2][4];
    uint32_t e_mask[2] = {0u, 0u};
    int e_qt[2] = {-1, -1};  // tiles whose candidates are still to be stored
    int e_par = 0;           // their step's parity (s_cnt buffer)
    auto emit_store = [&](auto tile) {  // tile: std::integral_constant (keeps e_c indices static)
        constexpr int t = decltype(tile)::value;
        if (e_qt[t] < 0) return;
        const uint32_t *cs = &s_cnt[e_par][t][col][0];
        const u32x4 c0 = *reinterpret_cast<const u32x4 *>(cs);
        const u32x4 c1 = *reinterpret_cast<const u32x4 *>(cs + 4);
        const u32x4 c2 = *reinterpret_cast<const u32x4 *>(cs + 8);
        const u32x4 c3 = *reinterpret_cast<const u32x4 *>(cs + 12);
        const uint32_t cnt[16] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w,
                                  c2.x, c2.y, c2.z, c2.w, c3.x, c3.y, c3.z, c3.w};
        const int me = wave * 4 + grp;
        uint32_t before = 0, total = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            before += i < me ? cnt[i] : 0u;
            total += cnt[i];
        }
        const int r = e_qt[t] * 16 + col;
        if (r < a.n_q) {
            const size_t blk = (size_t)(b * a.n_q + r) * a.kblocks + kblk;
            uint2 *dst = a.cands + blk * kTopkBlockSlots;
            uint32_t slot = before, m = e_mask[t];
            while (m) {
                const int j = __builtin_ctz(m);
                m &= m - 1u;
                if (slot < (uint32_t)kTopkBlockSlots)
                    dst[slot] = make_uint2(score_key(__uint_as_float(s_ek[t][wave][j][lane])),
                                           (uint32_t)(jw + 16 * (j >> 2) + 4 * grp + (j & 3)));
                ++slot;
            }
            if (me == 0) a.cand_count[blk] = total;
        }
        e_qt[t] = -1;
    };
    for (int qt = qt0, par = 0; qt < qt_end; qt += 2, par ^= 1) {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(kPfWaitVm0);                          // (a)
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_sched_barrier(0);
        int n_cur[2];
#pragma unroll
        for (int t = 0; t < 2; ++t)
            n_cur[t] = qt + t < qt_end ? key_limit<CAUSAL>(p_cur[t], len, a.n_q, (qt + t) * 16 + col) : 0;
        if (qt + 2 < qt_end) stage_pair(par ^ 1);                        // pair P + 1's queries
        emit_store(std::integral_constant<int, 0>{});                     // (b)
        emit_store(std::integral_constant<int, 1>{});
        if (qt + 2 < qt_end) {                                           // (c)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                p_next[t] = key_pos<CAUSAL>(qpos, a.n_q, (qt + 2 + t) * 16 + col);
                th_next[t] = a.thresh[(size_t)b * a.n_q + row_of(qt + 2, t)];
            }
        }
        if (qt + 4 < qt_end) load_pair(qt + 4);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < 2; ++t) {                                    // (d)
            if (tile_limit(n_cur[t]) <= jg) continue;  // uniform: no query of the tile sees this block
            bf16x8 qv[8];
#pragma unroll
            for (int kb = 0; kb < 8; ++kb)
                qv[kb] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4 *>(&s_q[par][t][col][kb * 32 + grp * 8]));
            score_regs(kv, qv, e_c[t]);
            const float thf = thresh_float(th_cur[t]);
            uint32_t m = 0u;
            if (tile_limit_min(n_cur[t]) >= jw + kPfWaveKeys) {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        m |= (e_c[t][kt][r] >= thf ? 1u : 0u) << (4 * kt + r);
                        s_ek[t][wave][4 * kt + r][lane] = __float_as_uint(e_c[t][kt][r]);
                    }
            } else {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const bool cand = jw + 16 * kt + 4 * grp + r < n_cur[t] && e_c[t][kt][r] >= thf;
                        m |= (cand ? 1u : 0u) << (4 * kt + r);
                        s_ek[t][wave][4 * kt + r][lane] = __float_as_uint(e_c[t][kt][r]);
                    }
            }
            e_mask[t] = m;
            s_cnt[par][t][col][wave * 4 + grp] = (uint32_t)__popc(m);
            e_qt[t] = qt + t;
        }
        e_par = par;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            p_cur[t] = p_next[t];
            th_cur[t] = th_next[t];
        }
        pf_lds_barrier();                                                // (e)
    }
    emit_store(std::integral_constant<int, 0>{});
    emit_store(std::integral_constant<int, 1>{});
}

bool index_uses_mfma(const Geometry &g) { return g.n_q >= kPrefillMinRows; }

static PrefillArgs prefill_args(const Geometry &g, const void *q_idx, const void *k_idx,
                                const int32_t *page_table, const int32_t *seq_lens,
                                const int32_t *q_pos) {
    PrefillArgs a{};
    a.q_idx = static_cast<const uint16_t *>(q_idx);
    a.k_idx = static_cast<const uint16_t *>(k_idx);
    a.page_table = page_table;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.causal = g.causal;
    a.key_stride = 1;
    a.qsplit = 1;
    a.attn_tickets = nullptr;
    a.n_tickets = g.rows * g.kv_heads;
    return a;
}

static hipError_t launch_prefill(const Geometry &g, const PrefillArgs &a, hipStream_t stream) {
    const size_t blocks = (size_t)g.batch * a.kblocks * a.qsplit;
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

hipError_t launch_index_prefill(const Geometry &g, const void *q_idx, const void *k_idx,
                                const int32_t *page_table, const int32_t *seq_lens,
                                const int32_t *q_pos, float *scores, uint32_t *attn_tickets,
                                hipStream_t stream) {
    PrefillArgs a = prefill_args(g, q_idx, k_idx, page_table, seq_lens, q_pos);
    a.attn_tickets = attn_tickets;
    a.scores = scores;
    a.row_stride = g.max_len;
    a.kblocks = div_up(g.max_len, kPfKeys);
    a.vec_store = (g.max_len % 4) == 0;
    return launch_prefill(g, a, stream);
}

// Enough workgroups for the chip when a pass has few key blocks: split the
// query tiles of each key block over ranges.
static int prefill_qsplit(const Geometry &g, int kblocks) {
    const int ntiles = div_up(g.n_q, 16);
    int qsplit = 1;
    while ((long)g.batch * kblocks * qsplit < 1024 && qsplit * 4 <= ntiles) qsplit *= 2;
    return qsplit;
}

hipError_t launch_index_prefill_sample(const Geometry &g, const void *q_idx, const void *k_idx,
                                       const int32_t *page_table, const int32_t *seq_lens,
                                       const int32_t *q_pos, float *samples, uint32_t *attn_tickets,
                                       hipStream_t stream) {
    PrefillArgs a = prefill_args(g, q_idx, k_idx, page_table, seq_lens, q_pos);
    a.attn_tickets = attn_tickets;
    a.scores = samples;
    a.key_stride = kTopkSampleStride;
    a.row_stride = topk_sample_cols(g);
    a.kblocks = div_up(a.row_stride, kPfKeys);
    a.vec_store = (a.row_stride % 4) == 0;
    a.qsplit = prefill_qsplit(g, a.kblocks);
    return launch_prefill(g, a, stream);
}

hipError_t launch_index_prefill_emit(const Geometry &g, const void *q_idx, const void *k_idx,
                                     const int32_t *page_table, const int32_t *seq_lens,
                                     const int32_t *q_pos, const uint32_t *thresh,
                                     uint32_t *cand_count, uint32_t *cands, hipStream_t stream) {
    PrefillArgs a = prefill_args(g, q_idx, k_idx, page_table, seq_lens, q_pos);
    a.thresh = thresh;
    a.cand_count = cand_count;
    a.cands = reinterpret_cast<uint2 *>(cands);
    a.row_stride = g.max_len;
    a.kblocks = div_up(g.max_len, kPfKeys);
    a.qsplit = prefill_qsplit(g, a.kblocks);
    const size_t blocks = (size_t)g.batch * a.kblocks * a.qsplit;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)blocks), block(256);
    const bool paged = g.page_shift >= 0;
    if (paged && g.causal) index_emit_kernel<true, true><<<grid, block, 0, stream>>>(a);
    else if (paged) index_emit_kernel<true, false><<<grid, block, 0, stream>>>(a);
    else if (g.causal) index_emit_kernel<false, true><<<grid, block, 0, stream>>>(a);
    else index_emit_kernel<false, false><<<grid, block, 0, stream>>>(a);
    return hipGetLastError();
}

hipError_t take_device_error_index_prefill(uint32_t *bits) { return take_source_device_error(bits); }

}  // namespace clsa
