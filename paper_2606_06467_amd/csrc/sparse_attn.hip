// Sparse GQA attention over the shared index set (Section 2.1, Eq. 4:
// O_t = Attn(Q_t, K_{S_t}, V_{S_t}); softmax attention as in Eq. 1; no
// positional encoding on this path).
//
// One workgroup (NW waves: 4, or 1 in the chunked-prefill form) = one (query
// row, KV head g, split of S).  A split is a run of chunks of 16 NW tokens of
// the row's index list.  Per chunk:
//   * each 16-lane quarter-wave gathers one selected token's 256-byte K row and
//     256-byte V row of head g (16 bytes per lane); 4 rounds x NW waves x 4
//     quarters = 16 NW tokens.  Index loads, page-table loads and the K/V loads
//     are each issued as one unconditional batch (positions past the end are
//     clamped and masked afterwards), so a workgroup waits for memory about
//     three times instead of once per token;
//   * the G query heads of the GQA group share those rows.  Two forms:
//     - matrix-core form (MQK; contiguous caches, and chunked prefill with
//       thousands of units): each wave's 16 K rows go through its own LDS rows
//       into v_mfma_f32_16x16x32_bf16 against Q^T (heads padded to 16), and
//       each wave keeps its own online softmax per head (base-2 exponentials;
//       the four lanes of a head combine with permlane swaps) and its own
//       weighted-V accumulators: no workgroup barrier per chunk; the wave
//       states are merged by the log-sum-exp rule at the end.  The weighted V
//       is a v_mfma_f32_16x16x16_bf16 product whose operands are the lane's
//       own weights and V rows (the logits tile is ordered for that);
//     - vector form (paged decode grids): each lane dots its 8 key values with
//       the matching 8 values of every head (v_dot2_f32_bf16), a
//       transpose-reduction over the 16 lanes leaves one (head, token) logit
//       per lane, the logits go to LDS, and one wave per head takes the chunk
//       maximum and sum, updates the running max / denominator and rescales
//       (online softmax, shared by the workgroup);
//     so a split of any length needs one pass;
//   * in the vector form each lane accumulates weight x V for its 8 dimensions
//     and G heads (v_dot2_f32_bf16).
// The accumulators are then reduced over lanes and waves in LDS.  With one
// split the workgroup writes the bf16 output and lse itself.  Otherwise it
// writes fp32 partials (o, m, l), combined by the exact log-sum-exp rule: inside
// the kernel by the last split of each (row, KV head) to arrive (inside
// clsa_decode_step, whose first index launch clears the arrival counters; see
// split_merge: write-through partials and a relaxed ticket, since an agent-scope
// release fence writes back the whole L2 of the XCD from every workgroup on this
// chip), else by attn_merge_kernel as a second launch.
// The same kernels serve dense attention over every valid key (Eq. 1, the
// attention that Eq. 4 restricts), used as the reference point for the cost of
// sparse attention: token positions then come straight from the chunk, with no
// index list.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kHeadDim = 128;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxSplits = 128;  // splits per (row, KV head): the merge's largest shape
constexpr int kManyUnits = 4096; // (row, KV head) units from which splits go by key range
constexpr int kKtPitch = 17;     // 16-byte pieces per staged K row (one of padding)
constexpr int kManySplits = 8;   // splits per unit then (measured best of 1, 2, 4, 8, 16)
constexpr int kManyUnitWaves = 1;    // waves per workgroup of the many-unit form (measured 1, 2, 4)
constexpr int kRotationWaves = 4352; // many units: base of the chunk-order period, a little under
                                     // the 5120 waves resident (5 per SIMD); 3584..5632 measured

// The fields every workgroup reads first come first: the kernel's prologue
// then fetches them in one batch of scalar loads (a field pushed past them
// costs one more dependent round trip per workgroup, measurable in a kernel
// of a few microseconds).  The dense-only fields come last.
struct AttnArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    const int32_t *page_table;
    const int32_t *idx;      // sparse: [rows, top_k] selected positions
    const int32_t *n_sel;    // sparse: [rows] their count
    uint16_t *out;
    float *lse;          // may be null
    float *part_o;       // [rows, Hq, splits, 128]
    float *part_ml;      // [rows, Hq, splits, 2]
    int n_q, max_len, page_shift, max_pages, top_k, kv_heads, q_heads, splits, chunks_per_split;
    float scale_log2;    // softmax_scale * log2(e)
    const int32_t *seq_lens; // dense: [batch]
    const int32_t *q_pos;    // dense, causal: [rows]
    int causal;
    // inside a step: one arrival counter per (row, KV head), zero on entry; the
    // last split to arrive combines the splits (no merge launch).
    // NULL: attn_merge_kernel runs as a second launch.
    uint32_t *tickets;
};

__host__ __device__ constexpr int pow2_at_least(int x) {
    return x <= 1 ? 1 : 2 * pow2_at_least((x + 1) / 2);
}

// Keys of row `row`: the first n_sel entries of its index list, or (DENSE) every
// valid position 0 .. n-1 in order, n = its sequence length (causal: up to its
// own position).
template <bool DENSE>
__device__ __forceinline__ int row_keys(const AttnArgs &a, int row) {
    if (DENSE) return valid_keys(a.seq_lens, a.q_pos, a.causal, row / a.n_q, row, a.max_len);
    const int m = a.n_sel[row];
    if (m < 0 || m > a.top_k) {
        note_device_error(kDevErrNSel);
        return m < 0 ? 0 : a.top_k;
    }
    return m;
}

// Maximum / sum over the four rows (lanes l, l ^ 16, l ^ 32, l ^ 48) of a wave.
__device__ __forceinline__ float rows4_max(float x) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float rows4_sum(float x) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Index entry `pos` of a row's list: a 32-bit byte offset from the list's base
// (uniform over the workgroup), so that the load takes the scalar-base form.
__device__ __forceinline__ int sel_at(const int32_t *sel, int pos) {
    return *reinterpret_cast<const int32_t *>(reinterpret_cast<const char *>(sel) +
                                              (uint32_t)pos * 4u);
}

__device__ __forceinline__ uint64_t pack2f(float x, float y) {
    return (uint64_t)__float_as_uint(x) | ((uint64_t)__float_as_uint(y) << 32);
}

// In-kernel split merge.  Every split of a (row, KV head) stores its partials
// (o, m, l) with device-scope stores (written through the XCD's L2, so other
// XCDs can read them without a cache write-back), waits until they are
// complete, and takes a ticket from the unit's counter; the split that draws the
// last ticket resets the counter and combines every split by the log-sum-exp
// rule, reading the partials with device-scope loads (one wave per query head,
// lane l owning dimensions 2l and 2l + 1, all loads issued before the first
// wait).  The ticket is a relaxed atomic: ordering comes from the completed
// write-through stores, not from an agent-scope release, whose L2 write-back
// costs about a microsecond per workgroup.  At most kFusedMaxSplits splits.
constexpr int kFusedMaxSplits = 8;

template <int G, bool DENSE, int NW, typename Combine>
__device__ __forceinline__ void split_merge(const AttnArgs &a, int row, int g, int split,
                                            int nsplit, size_t base, Combine combine) {
    __shared__ uint32_t s_ticket;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    for (int e = 2 * tid; e < G * kHeadDim; e += 128 * NW) {
        const int h = e / kHeadDim, dim = e - h * kHeadDim;
        float m, l, s0, s1;
        combine(h, e, m, l, s0);
        combine(h, e + 1, m, l, s1);
        const size_t slot = base + (size_t)h * a.splits + split;
        __hip_atomic_store(reinterpret_cast<uint64_t *>(a.part_o + slot * kHeadDim + dim),
                           pack2f(s0, s1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (dim == 0)
            __hip_atomic_store(reinterpret_cast<uint64_t *>(a.part_ml + slot * 2), pack2f(m, l),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's partials are complete
    __syncthreads();                                   // ... and every wave's
    uint32_t *ticket = a.tickets + (size_t)row * a.kv_heads + g;
    if (tid == 0) s_ticket = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (s_ticket != (uint32_t)(nsplit - 1)) return;  // uniform
    if (tid == 0) __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int Hq = a.q_heads;
    for (int h = wave; h < G; h += NW) {
        const size_t hb = base + (size_t)h * a.splits;
        uint64_t o[kFusedMaxSplits], ml[kFusedMaxSplits];
#pragma unroll
        for (int s = 0; s < kFusedMaxSplits; ++s) {
            const size_t slot = hb + min(s, nsplit - 1);
            o[s] = __hip_atomic_load(reinterpret_cast<const uint64_t *>(a.part_o + slot * kHeadDim + 2 * lane),
                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ml[s] = __hip_atomic_load(reinterpret_cast<const uint64_t *>(a.part_ml + slot * 2),
                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        auto lo = [](uint64_t x) { return __uint_as_float((uint32_t)x); };
        auto hi = [](uint64_t x) { return __uint_as_float((uint32_t)(x >> 32)); };
        float M = lo(ml[0]);  // finite: split 0 holds tokens
#pragma unroll
        for (int s = 1; s < kFusedMaxSplits; ++s)
            if (s < nsplit) M = fmaxf(M, lo(ml[s]));
        float l = 0.0f, ox = 0.0f, oy = 0.0f;
#pragma unroll
        for (int s = 0; s < kFusedMaxSplits; ++s) {
            if (s < nsplit) {
                const float w = exp2f(lo(ml[s]) - M);
                l = fmaf(w, hi(ml[s]), l);
                ox = fmaf(w, lo(o[s]), ox);
                oy = fmaf(w, hi(o[s]), oy);
            }
        }
        const float inv = 1.0f / l;
        const size_t rh = (size_t)row * Hq + g * G + h;
        *reinterpret_cast<uint32_t *>(a.out + rh * kHeadDim + lane * 2) =
            f32_to_bf16_bits(ox * inv) | (f32_to_bf16_bits(oy * inv) << 16);
        if (a.lse && lane == 0) a.lse[rh] = (M + log2f(l)) * kLn2;
    }
}

// MQK: matrix-core logits and weighted V with per-wave softmax states.  NW:
// waves per workgroup (4; 1 in the many-unit form).
template <int G, bool PAGED, bool DENSE, bool MQK, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW < 4 && G <= 5 ? 5 : 1)))
void sparse_attn_kernel(AttnArgs a) {
    static_assert(NW == 4 || MQK, "fewer waves per workgroup: the matrix-core form only");
    constexpr int CH = 16 * NW;  // tokens per chunk: 16 per wave
    // Many-unit form (NW < 4): one wave per workgroup and five waves per
    // SIMD (G <= 5; G = 8 needs 97 registers and 10.6 KB of LDS, so four), so
    // that as many rows as possible are resident at once (see the chunk order
    // below); the query operands therefore wait in LDS instead of 16 registers:
    // the G query rows, which every wave writes in full (the same values) and
    // each lane reads back only where it wrote them itself, so no barrier is
    // needed.
    constexpr bool QLDS = NW < 4;
    __shared__ __align__(16) u32x4 s_qb[QLDS ? G : 1][QLDS ? 16 : 1];  // [head][16-byte piece]
    constexpr int NV = pow2_at_least(4 * G);   // logits per lane before the reduction
    constexpr int NO = pow2_at_least(8 * G);   // accumulators per lane before the reduction
    __shared__ float zs[G][64];                // logits -> weights of the current chunk
    __shared__ float s_scale[G];               // per-head rescale factor of this chunk
    __shared__ float s_ml[G][2];               // running max (log2 domain) and denominator
    __shared__ __align__(16) float red[NW][G * kHeadDim];  // cross-wave reduction of the accumulators
    // MQK: per wave, its 16 gathered K rows (16 x 16 pieces of 16 bytes, padded)
    __shared__ __align__(16) u32x4 s_kt[MQK ? NW : 1][MQK ? 16 : 1][MQK ? kKtPitch : 1];
    __shared__ float s_wml[MQK ? NW : 1][G][2];  // MQK: each wave's (max, sum) per head

    // flattened grid, few (row, KV head) units: (row * kv_heads + g) * splits + split;
    // many units (kManyUnits or more): split * units + (row * kv_heads + g), so that
    // every row's first stretch of its (ascending) index list is gathered before
    // any row's second: the rows' K/V working set at any time is a key range
    // that the 256 MB Infinity Cache can hold.
    const int units_all = gridDim.x / a.splits;
    const bool split_major = units_all >= kManyUnits;
    const int split = split_major ? blockIdx.x / units_all : blockIdx.x % a.splits;
    const int rg = split_major ? blockIdx.x % units_all : blockIdx.x / a.splits;
    const int g = rg % a.kv_heads, row = rg / a.kv_heads;
    const int b = row / a.n_q;
    const int Hq = a.q_heads;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int qq = lane >> 4, sub = lane & 15;
    const int span = a.chunks_per_split * 64;
    const int tok_begin = split * span;
    // Chunk order of the many-unit form (NW < 4): a workgroup starts at
    // chunk (blockIdx / P) mod cps of its cps chunks and wraps around, P being
    // about the resident workgroups (kRotationWaves / NW) over cps.  Workgroups
    // start in grid order, about P per chunk time once the chip is full, so
    // the resident ones tend to be on the same chunk of their stretch at the
    // same time; as the index lists are ascending and all rows' stretches span about
    // the same keys, the K/V rows gathered at any moment come from about one
    // chunk's share of the stretch instead of all of it, and each of them is
    // gathered by more of the resident rows while the L2 still holds it, the
    // more rows are resident.  The online softmax does not depend on the order
    // of the chunks (only the order of its fp32 roundings does).
    constexpr bool ROT = NW < 4;
    const int cps = span / CH;  // chunks per split
    const unsigned rot_period = max(1, kRotationWaves / NW / cps);
    const int rot = ROT && split_major ? (int)((blockIdx.x / rot_period) % (unsigned)cps) : 0;
    const int row_elems = a.kv_heads * kHeadDim;
    const char *kseq = reinterpret_cast<const char *>(
        a.k + ((size_t)b * a.max_len * a.kv_heads + g) * kHeadDim);
    const char *vseq = reinterpret_cast<const char *>(
        a.v + ((size_t)b * a.max_len * a.kv_heads + g) * kHeadDim);
    const int32_t *sel = DENSE ? nullptr : a.idx + (size_t)row * a.top_k;

    // Index loads of the first chunk do not wait for n_sel: the index list has
    // top_k entries (padding included), so any position below top_k is readable.
    int jpre[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        jpre[i] = DENSE ? tok_begin + rot * CH + i * 4 * NW + wave * 4 + qq
                        : sel_at(sel, min(tok_begin + rot * CH + i * 4 * NW + wave * 4 + qq, a.top_k - 1));
    const int n = row_keys<DENSE>(a, row);
    const int nsplit = div_up(n, span);  // splits that hold tokens

    if (n == 0) {  // empty index set: output 0, lse -inf
        if (split == 0) {
            for (int e = tid; e < G * kHeadDim; e += 64 * NW)
                a.out[((size_t)row * Hq + g * G) * kHeadDim + e] = 0;
            if (a.lse && tid < G) a.lse[(size_t)row * Hq + g * G + tid] = -INFINITY;
        }
        return;
    }
    if (split >= nsplit) return;  // uniform; the merge masks splits past the last one
    const int tok_end = min(n, tok_begin + span);
    const int nch = div_up(tok_end - tok_begin, CH);  // chunks of this split (>= 1)
    int cfirst = rot;
    if (ROT && cfirst >= nch) {  // a short split (the row's last): start from a chunk it has
        cfirst = rot % nch;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            jpre[i] = DENSE ? tok_begin + cfirst * CH + i * 4 * NW + wave * 4 + qq
                            : sel_at(sel, min(tok_begin + cfirst * CH + i * 4 * NW + wave * 4 + qq, a.top_k - 1));
    }

    uint4 qv[MQK ? 1 : G];
    bf16x8 qb[4];  // MQK: B operands, Q^T (32 dims x 16 head columns, heads >= G zero)
    if (!MQK) {
#pragma unroll
        for (int h = 0; h < G; ++h)
            qv[h] = *reinterpret_cast<const uint4 *>(
                a.q + ((size_t)row * Hq + g * G + h) * kHeadDim + sub * 8);
    } else {
        const int hq = min(sub, G - 1);
        const uint16_t *qp = a.q + ((size_t)row * Hq + g * G + hq) * kHeadDim + qq * 8;
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const u32x4 v = *reinterpret_cast<const u32x4 *>(qp + 32 * s4);
            if (QLDS) {
                if (sub < G) s_qb[sub][qq + 4 * s4] = v;
            } else {
                qb[s4] = __builtin_bit_cast(bf16x8, sub < G ? v : u32x4{0u, 0u, 0u, 0u});
            }
        }
    }
    if (tid < G) {
        s_ml[tid][0] = -INFINITY;
        s_ml[tid][1] = 0.0f;
    }
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int d = 0; d < 8; ++d) acc[h][d] = 0.0f;
    float m_run = -INFINITY, l_run = 0.0f;  // MQK: head sub's running max / sum (this wave)
    // MQK: weighted V per 16-dim block blk, lane (qq, sub): heads 4qq + r, dim 8sub + blk
    f32x4 pacc[MQK ? 8 : 1];
#pragma unroll
    for (int i = 0; i < (MQK ? 8 : 1); ++i) pacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int ci = 0, c = cfirst, c0 = tok_begin; ROT ? ci < nch : c0 < tok_end; ++ci, c0 += CH) {
        int c0_next = c0 + CH;
        if constexpr (ROT) {
            c0 = tok_begin + c * CH;
            c = c + 1 < nch ? c + 1 : 0;  // the next chunk in this workgroup's order
            c0_next = tok_begin + c * CH;
        }
        int jr[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)  // -1 padding -> row 0; dense positions past n -> row n-1
            jr[i] = DENSE ? min(jpre[i], n - 1) : min(max(jpre[i], 0), a.max_len - 1);
        uint32_t trow[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (PAGED) {
                const int page = a.page_table[(size_t)b * a.max_pages + (jr[i] >> a.page_shift)];
                trow[i] = ((uint32_t)page << a.page_shift) + (jr[i] & ((1 << a.page_shift) - 1));
            } else {
                trow[i] = 0;  // unused: contiguous caches use byte offsets from kseq / vseq
            }
        }
        uint4 kr[4], vr[4];
        if (PAGED) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const size_t off = (size_t)trow[i] * row_elems + (size_t)g * kHeadDim + sub * 8;
                kr[i] = *reinterpret_cast<const uint4 *>(a.k + off);
                vr[i] = *reinterpret_cast<const uint4 *>(a.v + off);
            }
        } else {
            // contiguous caches: a 32-bit byte offset inside the row's sequence
            // (one sequence's cache is below 4 GiB, checked at the boundary) from
            // a base that is the same for the whole workgroup
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t off = (uint32_t)jr[i] * (uint32_t)(row_elems * 2) + (uint32_t)(sub * 16);
                kr[i] = *reinterpret_cast<const uint4 *>(kseq + off);
                vr[i] = *reinterpret_cast<const uint4 *>(vseq + off);
            }
        }
        // prefetch the next chunk's indices (clamped, so always readable)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            jpre[i] = DENSE ? c0_next + i * 4 * NW + wave * 4 + qq
                            : sel_at(sel, min(c0_next + i * 4 * NW + wave * 4 + qq, a.top_k - 1));
        // All K and V gathers of the chunk are in flight before any math (without
        // this the scheduler sinks the V loads below the logits, which costs a
        // second memory round trip per chunk).
        __builtin_amdgcn_sched_barrier(0);
        // weight x V with the lane's tokens in pairs (rounds 0, 1 and 2, 3): bf16
        // weights and values into v_dot2_f32_bf16, fp32 accumulation.  weight(h, i):
        // the weight of head h for this lane's round-i token (0 past the end).
        auto weighted_v = [&](auto weight) {
#pragma unroll
            for (int pr = 0; pr < 2; ++pr) {
                bf16x2 wp[G];
#pragma unroll
                for (int h = 0; h < G; ++h)
                    wp[h] = bf16x2{(__bf16)weight(h, 2 * pr), (__bf16)weight(h, 2 * pr + 1)};
                const uint32_t va[4] = {vr[2 * pr].x, vr[2 * pr].y, vr[2 * pr].z, vr[2 * pr].w};
                const uint32_t vb[4] = {vr[2 * pr + 1].x, vr[2 * pr + 1].y, vr[2 * pr + 1].z,
                                        vr[2 * pr + 1].w};
#pragma unroll
                for (int c2 = 0; c2 < 4; ++c2) {
                    // dims 2c2 and 2c2+1 of both tokens: {va.lo, vb.lo} and {va.hi, vb.hi}
                    const bf16x2 lo = __builtin_bit_cast(
                        bf16x2, __builtin_amdgcn_perm(vb[c2], va[c2], 0x05040100u));
                    const bf16x2 hi = __builtin_bit_cast(
                        bf16x2, __builtin_amdgcn_perm(vb[c2], va[c2], 0x07060302u));
#pragma unroll
                    for (int h = 0; h < G; ++h) {
                        acc[h][2 * c2] =
                            __builtin_amdgcn_fdot2_f32_bf16(wp[h], lo, acc[h][2 * c2], false);
                        acc[h][2 * c2 + 1] =
                            __builtin_amdgcn_fdot2_f32_bf16(wp[h], hi, acc[h][2 * c2 + 1], false);
                    }
                }
            }
        };
        if (MQK) {
            // Logits on the matrix cores: C = K_w (16 tokens x 128) x Q^T (128 x 16
            // head columns).  The wave's 16 K rows (gathered as above: token slot
            // r = 4i + qq is chunk token 4 NW i + 4w + qq) go through this wave's LDS
            // rows to reach the operand layout: lane (qq, sub) supplies A row sub,
            // dims 8qq + 32s of step s, and receives C rows 4qq + r of head sub.
            // A row m holds slot 4(m & 3) + (m >> 2), so that
            // C row 4qq + r is slot 4r + qq: this lane's own gathered row of round r.
            u32x4 *sk = &s_kt[wave][0][0];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                sk[(i * 4 + qq) * kKtPitch + sub] = u32x4{kr[i].x, kr[i].y, kr[i].z, kr[i].w};
            f32x4 c = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int arow = 4 * (sub & 3) + (sub >> 2);
                const bf16x8 ka = __builtin_bit_cast(bf16x8, sk[arow * kKtPitch + qq + 4 * s4]);
                const bf16x8 qop = QLDS ? __builtin_bit_cast(bf16x8, sub < G ? s_qb[min(sub, G - 1)][qq + 4 * s4]
                                                                              : u32x4{0u, 0u, 0u, 0u})
                                        : qb[s4];
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qop, c, 0, 0, 0);
            }
            // Online softmax per wave over its own 16 slots (no workgroup barrier):
            // lane (qq, sub) keeps the running maximum and sum of head sub; the
            // four lanes of a head (one per row) combine with permlane swaps.
            float z[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tl = r * 4 * NW + wave * 4 + qq;  // slot 4r + qq
                z[r] = sub < G && c0 + tl < tok_end ? c[r] * a.scale_log2 : -INFINITY;
            }
            const float mx = rows4_max(fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3])));
            const float m_new = fmaxf(m_run, mx);
            const float base = m_new == -INFINITY ? 0.0f : m_new;  // no valid slot yet
            float w[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) w[r] = __builtin_amdgcn_exp2f(z[r] - base);  // -inf -> 0
            const float scl = __builtin_amdgcn_exp2f(m_run - base);  // m_run = -inf -> 0
            l_run = l_run * scl + rows4_sum((w[0] + w[1]) + (w[2] + w[3]));
            m_run = m_new;
            // Weighted V on the matrix cores with no data movement: contraction
            // index k = 4qq + j stands for slot 4j + qq, so the A operand (P,
            // heads x slots) is this lane's own weights w[0..3] (bf16) and the
            // B operand of 16-dim block blk (slots x dims 8n + blk) is element
            // blk of this lane's own four V rows.
            const s16x4 pa = __builtin_bit_cast(
                s16x4, u32x2{__builtin_bit_cast(uint32_t, bf16x2{(__bf16)w[0], (__bf16)w[1]}),
                             __builtin_bit_cast(uint32_t, bf16x2{(__bf16)w[2], (__bf16)w[3]})});
            // rescale: C row 4qq + r is head 4qq + r, whose factor every lane
            // (*, head) holds
            float f[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                f[r] = r < G ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                             __builtin_bit_cast(int, scl), r))
                             : 1.0f;
                if (4 + r < G)
                    f[r] = qq == 1 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                                   __builtin_bit_cast(int, scl), 4 + r))
                                   : f[r];
            }
#pragma unroll
            for (int blk = 0; blk < 8; ++blk)
#pragma unroll
                for (int r = 0; r < 4; ++r) pacc[blk][r] *= f[r];
            const uint32_t v0[4] = {vr[0].x, vr[0].y, vr[0].z, vr[0].w};
            const uint32_t v1[4] = {vr[1].x, vr[1].y, vr[1].z, vr[1].w};
            const uint32_t v2[4] = {vr[2].x, vr[2].y, vr[2].z, vr[2].w};
            const uint32_t v3[4] = {vr[3].x, vr[3].y, vr[3].z, vr[3].w};
#pragma unroll
            for (int c2 = 0; c2 < 4; ++c2) {
                // dims 2c2 (low halves) and 2c2 + 1 (high halves) of rounds 0..3
                const s16x4 blo = __builtin_bit_cast(
                    s16x4, u32x2{__builtin_amdgcn_perm(v1[c2], v0[c2], 0x05040100u),
                                 __builtin_amdgcn_perm(v3[c2], v2[c2], 0x05040100u)});
                const s16x4 bhi = __builtin_bit_cast(
                    s16x4, u32x2{__builtin_amdgcn_perm(v1[c2], v0[c2], 0x07060302u),
                                 __builtin_amdgcn_perm(v3[c2], v2[c2], 0x07060302u)});
                pacc[2 * c2] =
                    __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, blo, pacc[2 * c2], 0, 0, 0);
                pacc[2 * c2 + 1] =
                    __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, bhi, pacc[2 * c2 + 1], 0, 0, 0);
            }
        } else {
            // logits: value index i*G + h, transpose-reduced over the 16 lanes of the quarter
            float p[NV];
#pragma unroll
            for (int v = 0; v < NV; ++v) p[v] = 0.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int h = 0; h < G; ++h) p[i * G + h] = dot8_bf16(kr[i], qv[h], 0.0f);
            transpose_reduce<NV, 8, 1, NV>(p, sub);
            // lane `sub` now holds value indices [sub*NV/16, sub*NV/16 + NV/16) (NV >= 16)
            // or index sub / (16/NV) (NV < 16).
            constexpr int PER = NV >= 16 ? NV / 16 : 1;
#pragma unroll
            for (int v = 0; v < PER; ++v) {
                const int orig = NV >= 16 ? sub * PER + v : sub / (16 / NV);
                if (orig < 4 * G) {
                    const int i = orig / G, h = orig - i * G;
                    const int tl = i * 16 + wave * 4 + qq;
                    zs[h][tl] = c0 + tl < tok_end ? p[v] * a.scale_log2 : -INFINITY;
                }
            }
        }
        if (!MQK) {
        __syncthreads();
        // per-head chunk statistics and online-softmax update
        for (int h = wave; h < G; h += 4) {
            const float z = zs[h][lane];
            const float mx = wave_max(z);
            const float m_old = s_ml[h][0];
            const float m_new = fmaxf(m_old, mx);   // finite: the chunk has a valid token
            const float w = exp2f(z - m_new);        // z = -inf -> 0
            const float sum = wave_sum(w);
            zs[h][lane] = w;
            if (lane == 0) {
                const float sc = exp2f(m_old - m_new);  // m_old = -inf -> 0
                s_scale[h] = sc;
                s_ml[h][0] = m_new;
                s_ml[h][1] = s_ml[h][1] * sc + sum;
            }
        }
        __syncthreads();
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float sc = s_scale[h];
#pragma unroll
            for (int d = 0; d < 8; ++d) acc[h][d] *= sc;
        }
        weighted_v([&](int h, int i) { return zs[h][i * 16 + wave * 4 + qq]; });
        __syncthreads();  // zs / s_scale are rewritten by the next chunk
        }
    }

    if constexpr (MQK) {
        // the wave's weighted V is complete in the C tiles: head 4qq + r, dims 8sub..8sub+7
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (4 * qq + r < G) {
                float *dst = &red[wave][(4 * qq + r) * kHeadDim + sub * 8];
                *reinterpret_cast<float4 *>(dst) =
                    make_float4(pacc[0][r], pacc[1][r], pacc[2][r], pacc[3][r]);
                *reinterpret_cast<float4 *>(dst + 4) =
                    make_float4(pacc[4][r], pacc[5][r], pacc[6][r], pacc[7][r]);
            }
        }
    } else {
    // ---- reduce the accumulators over the 4 quarters of each wave (lanes ^16, ^32) ----
    float o[NO];
#pragma unroll
    for (int v = 0; v < NO; ++v) o[v] = 0.0f;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int d = 0; d < 8; ++d) o[h * 8 + d] = acc[h][d];
    transpose_reduce<NO, 32, 16, NO>(o, lane);
    // lane (qq, sub) holds value indices [qq*NO/4, qq*NO/4 + NO/4); index = h*8 + d
#pragma unroll
    for (int v = 0; v < NO / 4; ++v) {
        const int orig = qq * (NO / 4) + v;
        if (orig < 8 * G) {
            const int h = orig >> 3, d = orig & 7;
            red[wave][h * kHeadDim + sub * 8 + d] = o[v];
        }
    }
    }
    if (MQK && qq == 0 && sub < G) {  // this wave's (max, sum) of head sub
        s_wml[wave][sub][0] = m_run;
        s_wml[wave][sub][1] = l_run;
    }
    __syncthreads();
    // (max, sum, weighted V) of head h over the workgroup: with per-wave softmax
    // states (MQK) the NW waves combine by the log-sum-exp rule
    auto combine = [&](int h, int e, float &m, float &l, float &sum) {
        if constexpr (MQK) {
            if constexpr (NW == 4) {
                m = fmaxf(fmaxf(s_wml[0][h][0], s_wml[1][h][0]), fmaxf(s_wml[2][h][0], s_wml[3][h][0]));
            } else {
                m = s_wml[0][h][0];
#pragma unroll
                for (int w4 = 1; w4 < NW; ++w4) m = fmaxf(m, s_wml[w4][h][0]);
            }
            l = 0.0f;
            sum = 0.0f;
#pragma unroll
            for (int w4 = 0; w4 < NW; ++w4) {
                const float mw = s_wml[w4][h][0];
                const float f = mw == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mw - m);
                l = fmaf(f, s_wml[w4][h][1], l);
                sum = fmaf(f, red[w4][e], sum);
            }
        } else {
            m = s_ml[h][0];
            l = s_ml[h][1];
            sum = red[0][e] + red[1][e] + red[2][e] + red[3][e];
        }
    };
    // one split, or (with the in-kernel merge) the only split that holds tokens
    if (a.splits == 1 || (a.tickets && nsplit == 1)) {
        for (int e = tid; e < G * kHeadDim; e += 64 * NW) {
            const int h = e / kHeadDim, dim = e - h * kHeadDim;
            float m, l, sum;
            combine(h, e, m, l, sum);
            const int hq = g * G + h;
            a.out[((size_t)row * Hq + hq) * kHeadDim + dim] =
                (uint16_t)f32_to_bf16_bits(sum / l);
            if (a.lse && dim == 0) a.lse[(size_t)row * Hq + hq] = (m + log2f(l)) * kLn2;
        }
        return;
    }
    const size_t base = ((size_t)row * Hq + g * G) * a.splits;  // slot of (head g*G, split 0)
    if (a.tickets) {
        split_merge<G, DENSE, NW>(a, row, g, split, nsplit, base, combine);
        return;
    }
    for (int e = tid; e < G * kHeadDim; e += 64 * NW) {
        const int h = e / kHeadDim, dim = e - h * kHeadDim;
        float m, l, sum;
        combine(h, e, m, l, sum);
        const size_t slot = base + (size_t)h * a.splits + split;
        a.part_o[slot * kHeadDim + dim] = sum;
        if (dim == 0) {
            a.part_ml[slot * 2] = m;
            a.part_ml[slot * 2 + 1] = l;
        }
    }
}

// Up to 4 splits: one wave per (row, query head), lane l owning dimensions 2l
// and 2l + 1 and holding every split's (m, l) and o slice in registers, so the
// log-sum-exp rule below needs no cross-lane step, no LDS and no barrier.  The
// loads are issued in one batch (splits past the row's last one read the last
// slot and are masked afterwards).
template <int SPW, bool DENSE>  // SPW: splits held per lane (SPW >= splits)
__global__ __launch_bounds__(64) void attn_merge_wave_kernel(AttnArgs a) {
    const int rh = blockIdx.x;  // row * Hq + head
    const int row = rh / a.q_heads;
    const int lane = threadIdx.x;
    const size_t base = (size_t)rh * a.splits;
    float2 o[SPW], ml[SPW];
#pragma unroll
    for (int s = 0; s < SPW; ++s) {
        const size_t slot = base + min(s, a.splits - 1);
        o[s] = *reinterpret_cast<const float2 *>(a.part_o + slot * kHeadDim + lane * 2);
        ml[s] = *reinterpret_cast<const float2 *>(a.part_ml + slot * 2);
    }
    const int n = row_keys<DENSE>(a, row);
    const int nsplit = div_up(n, a.chunks_per_split * 64);  // splits that hold tokens
    if (nsplit == 0) return;  // the attention kernel wrote the empty-set result
    float M = ml[0].x;        // finite: split 0 holds tokens
#pragma unroll
    for (int s = 1; s < SPW; ++s)
        if (s < nsplit) M = fmaxf(M, ml[s].x);
    float l = 0.0f, ox = 0.0f, oy = 0.0f;
#pragma unroll
    for (int s = 0; s < SPW; ++s) {
        if (s < nsplit) {
            const float w = exp2f(ml[s].x - M);
            l = fmaf(w, ml[s].y, l);
            ox = fmaf(w, o[s].x, ox);
            oy = fmaf(w, o[s].y, oy);
        }
    }
    const float inv = 1.0f / l;
    *reinterpret_cast<uint32_t *>(a.out + (size_t)rh * kHeadDim + lane * 2) =
        f32_to_bf16_bits(ox * inv) | (f32_to_bf16_bits(oy * inv) << 16);
    if (a.lse && lane == 0) a.lse[rh] = (M + log2f(l)) * kLn2;
}

// Combine the splits of one (row, query head) with the exact log-sum-exp rule:
// o = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s, M = max_s m_s.
// More than 4 splits: 256 threads = 8 split groups x 32 four-dimension slices.  Every load the
// workgroup needs (the row's selection count and all of its splits' (m, l) and
// o) is issued in one batch before the first wait: splits past the row's last
// one are read anyway (the buffer holds `splits` slots) and masked afterwards,
// so the kernel costs one memory round trip.
template <int SPT, bool DENSE>  // SPT: splits per thread (8 * SPT >= splits)
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
    __shared__ float s_max[8], s_l[8];
    __shared__ float4 s_o[8][32];
    const int rh = blockIdx.x;  // row * Hq + head
    const int row = rh / a.q_heads;
    const int tid = threadIdx.x, dq = tid & 31, sg = tid >> 5;
    const size_t base = (size_t)rh * a.splits;
    float4 o[SPT];
    float2 ml[SPT];
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int s = min(sg + 8 * j, a.splits - 1);
        o[j] = *reinterpret_cast<const float4 *>(a.part_o + (base + s) * kHeadDim + dq * 4);
        ml[j] = *reinterpret_cast<const float2 *>(a.part_ml + (base + s) * 2);
    }
    const int n = row_keys<DENSE>(a, row);
    const int nsplit = div_up(n, a.chunks_per_split * 64);  // splits that hold tokens
    if (nsplit == 0) return;  // the attention kernel wrote the empty-set result
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
        if (sg + 8 * j < nsplit) mx = fmaxf(mx, ml[j].x);
    if (dq == 0) s_max[sg] = mx;
    __syncthreads();
    float M = s_max[0];
#pragma unroll
    for (int x = 1; x < 8; ++x) M = fmaxf(M, s_max[x]);  // finite: split 0 holds tokens
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float l = 0.0f;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        if (sg + 8 * j < nsplit) {
            const float w = exp2f(ml[j].x - M);
            l = fmaf(w, ml[j].y, l);
            acc.x = fmaf(w, o[j].x, acc.x);
            acc.y = fmaf(w, o[j].y, acc.y);
            acc.z = fmaf(w, o[j].z, acc.z);
            acc.w = fmaf(w, o[j].w, acc.w);
        }
    }
    s_o[sg][dq] = acc;
    if (dq == 0) s_l[sg] = l;
    __syncthreads();
    if (tid < 32) {
        float4 r = s_o[0][dq];
        float L = s_l[0];
#pragma unroll
        for (int x = 1; x < 8; ++x) {
            const float4 t = s_o[x][dq];
            r.x += t.x; r.y += t.y; r.z += t.z; r.w += t.w;
            L += s_l[x];
        }
        const float inv = 1.0f / L;
        const uint32_t lo = f32_to_bf16_bits(r.x * inv) | (f32_to_bf16_bits(r.y * inv) << 16);
        const uint32_t hi = f32_to_bf16_bits(r.z * inv) | (f32_to_bf16_bits(r.w * inv) << 16);
        *reinterpret_cast<uint2 *>(a.out + (size_t)rh * kHeadDim + dq * 4) = make_uint2(lo, hi);
        if (a.lse && tid == 0) a.lse[rh] = (M + log2f(L)) * kLn2;
    }
}

// Splits per (row, KV head).  Sparse attention on contiguous caches (the
// matrix-core form) aims at about 256 workgroups (one per CU) with at most 8
// chunks of 64 tokens per split; everything else at about 1024 (four per CU).
// Either way a split keeps at least four chunks while that still leaves 256
// workgroups, so that the per-workgroup prologue and final merge are spread
// over more chunks.  Measured with the matrix-core form: 128K, 8 splits of 4
// chunks against 16 of 2 and 32 of 1; 32K, 4 splits of 8 chunks against 8 of 4.
// The paged 32-sequence ragged batch keeps 4 splits of 8 chunks (1 split is
// far slower there) and the 4K single-sequence step one chunk per split.  With
// many units (chunked prefill: thousands of rows) the grid is far wider than
// the chip anyway; there each list is cut into kManySplits stretches, issued
// stretch by stretch over all rows, so that the K/V rows gathered at any time
// come from one key range (the lists are ascending) and stay in the Infinity
// Cache (8192 rows x 2048 of 131072 keys: 8.8 -> 7.2 ms per layer); within a
// stretch the kernel rotates each workgroup's chunk order so that the resident
// workgroups gather from about one chunk's share of it, with one wave per
// workgroup so that many rows are resident.  keys: the
// most keys a row can have (top_k, or max_len for dense attention).
static void plan_splits(const Geometry &g, int keys, bool dense, int &splits,
                        int &chunks_per_split) {
    const int chunks = div_up(keys, 64);
    const long units = (long)g.rows * g.kv_heads;
    const bool wide = !dense && g.page_shift < 0;  // matrix-core form: fewer, longer workgroups
    long want = units > 0 ? ((wide ? 256 : 1024) + units - 1) / units : 1;
    if (wide && want < (chunks + 7) / 8) want = (chunks + 7) / 8;  // at most 8 chunks per split
    if (units >= kManyUnits && want < kManySplits) want = kManySplits;
    const long cap = units * (chunks / 4) >= 256 ? chunks / 4 : chunks;
    if (want > cap) want = cap;
    if (want > kMaxSplits) want = kMaxSplits;
    if (want < 1) want = 1;
    chunks_per_split = div_up(chunks, (int)want);
    splits = div_up(chunks, chunks_per_split);
}

size_t attn_partial_floats(const Geometry &g, bool dense) {
    int splits, cps;
    plan_splits(g, dense ? g.max_len : g.top_k, dense, splits, cps);
    if (splits == 1) return 0;
    return (size_t)g.rows * g.q_heads * splits * (kHeadDim + 2);
}

template <int G, bool DENSE>
static hipError_t launch_attn_g(const AttnArgs &a, bool paged, dim3 grid, int units,
                                hipStream_t stream, hipEvent_t split_done) {
    // Logits on the matrix cores with per-wave softmax states for contiguous
    // caches and for many units (chunked prefill); paged decode grids keep the
    // vector-unit logits and the shared softmax, which measured faster there.
    const bool many = grid.x / a.splits >= (unsigned)kManyUnits;
    constexpr int NWM = kManyUnitWaves;
    if (paged && many) sparse_attn_kernel<G, true, DENSE, true, NWM><<<grid, dim3(64 * NWM), 0, stream>>>(a);
    else if (paged) sparse_attn_kernel<G, true, DENSE, false, 4><<<grid, dim3(256), 0, stream>>>(a);
    else if (many) sparse_attn_kernel<G, false, DENSE, true, NWM><<<grid, dim3(64 * NWM), 0, stream>>>(a);
    else sparse_attn_kernel<G, false, DENSE, true, 4><<<grid, dim3(256), 0, stream>>>(a);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && split_done) e = hipEventRecord(split_done, stream);
    if (e != hipSuccess || a.splits == 1 || a.tickets) return e;
    const dim3 mgrid(units), mblock(256), wblock(64);
    // up to 4 splits: one wave per (row, query head) (32K step layers -1.7 us,
    // 32-sequence ragged batch -6.5 us); 8 splits measured faster on the
    // 256-thread form (128K layers 158.1 against 162.5 us)
    if (a.splits <= 4) attn_merge_wave_kernel<4, DENSE><<<mgrid, wblock, 0, stream>>>(a);
    else if (a.splits <= 8) attn_merge_kernel<1, DENSE><<<mgrid, mblock, 0, stream>>>(a);
    else if (a.splits <= 16) attn_merge_kernel<2, DENSE><<<mgrid, mblock, 0, stream>>>(a);
    else if (a.splits <= 32) attn_merge_kernel<4, DENSE><<<mgrid, mblock, 0, stream>>>(a);
    else if (a.splits <= 64) attn_merge_kernel<8, DENSE><<<mgrid, mblock, 0, stream>>>(a);
    else attn_merge_kernel<16, DENSE><<<mgrid, mblock, 0, stream>>>(a);
    return hipGetLastError();
}

template <bool DENSE>
static hipError_t launch_attn(const Geometry &g, const AttnArgs &a, bool paged, dim3 grid,
                              int units, hipStream_t stream, hipEvent_t split_done) {
    switch (g.group) {
        case 1: return launch_attn_g<1, DENSE>(a, paged, grid, units, stream, split_done);
        case 2: return launch_attn_g<2, DENSE>(a, paged, grid, units, stream, split_done);
        case 4: return launch_attn_g<4, DENSE>(a, paged, grid, units, stream, split_done);
        case 5: return launch_attn_g<5, DENSE>(a, paged, grid, units, stream, split_done);
        case 8: return launch_attn_g<8, DENSE>(a, paged, grid, units, stream, split_done);
        default: return hipErrorInvalidValue;
    }
}

static AttnArgs attn_args(const Geometry &g, const void *q, const void *k_cache,
                          const void *v_cache, const int32_t *page_table, void *out, float *lse,
                          float *partials, bool dense) {
    const int keys = dense ? g.max_len : g.top_k;
    AttnArgs a;
    a.q = static_cast<const uint16_t *>(q);
    a.k = static_cast<const uint16_t *>(k_cache);
    a.v = static_cast<const uint16_t *>(v_cache);
    a.page_table = page_table;
    a.idx = nullptr;
    a.n_sel = nullptr;
    a.seq_lens = nullptr;
    a.q_pos = nullptr;
    a.out = static_cast<uint16_t *>(out);
    a.lse = lse;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.top_k = g.top_k;
    a.kv_heads = g.kv_heads;
    a.q_heads = g.q_heads;
    a.causal = g.causal;
    a.tickets = nullptr;
    plan_splits(g, keys, dense, a.splits, a.chunks_per_split);
    a.scale_log2 = g.softmax_scale * kLog2e;
    const size_t part_o = (size_t)g.rows * g.q_heads * a.splits * kHeadDim;
    a.part_o = a.splits > 1 ? partials : nullptr;
    a.part_ml = a.splits > 1 ? partials + part_o : nullptr;
    return a;
}

hipError_t launch_sparse_attn(const Geometry &g, const void *q, const void *k_cache,
                              const void *v_cache, const int32_t *page_table,
                              const int32_t *idx, const int32_t *n_sel, void *out, float *lse,
                              float *partials, uint32_t *tickets, hipStream_t stream,
                              hipEvent_t split_done) {
    AttnArgs a = attn_args(g, q, k_cache, v_cache, page_table, out, lse, partials, false);
    a.idx = idx;
    a.n_sel = n_sel;
    if (g.rows == 0) return hipSuccess;
    const size_t blocks = (size_t)g.rows * g.kv_heads * a.splits;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    if (tickets && a.splits > 1 && a.splits <= kFusedMaxSplits) a.tickets = tickets;
    const int units = g.rows * g.q_heads;  // merge workgroups: one per (row, query head)
    return launch_attn<false>(g, a, g.page_shift >= 0, dim3((unsigned)blocks), units, stream,
                              split_done);
}

hipError_t launch_dense_attn(const Geometry &g, const void *q, const void *k_cache,
                             const void *v_cache, const int32_t *page_table,
                             const int32_t *seq_lens, const int32_t *q_pos, void *out, float *lse,
                             float *partials, hipStream_t stream) {
    AttnArgs a = attn_args(g, q, k_cache, v_cache, page_table, out, lse, partials, true);
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    if (g.rows == 0) return hipSuccess;
    const size_t blocks = (size_t)g.rows * g.kv_heads * a.splits;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    const int units = g.rows * g.q_heads;
    return launch_attn<true>(g, a, g.page_shift >= 0, dim3((unsigned)blocks), units, stream,
                             nullptr);
}

hipError_t take_device_error_sparse_attn(uint32_t *bits) { return take_source_device_error(bits); }

}  // namespace clsa
