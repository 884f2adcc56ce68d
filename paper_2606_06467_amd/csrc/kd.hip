// Training side of the shared indexer (Section 2.2): the distillation target
// of Eq. 5 and the KL loss of Eq. 6 with its gradient.
//
// Eq. 5: abar[b,t,j] = (1 / (L * Hq)) * sum over layers l and query heads h of
// softmax_j(scale * q_l[b,t,h] . K[b,j,g(h)]) over the valid keys of row (b,t),
// one shared key cache for every layer.  Logits on the matrix cores
// (v_mfma_f32_16x16x32_bf16: A = 16 query rows x 32 dims, B = 32 dims x 16
// keys; lane l supplies row / key (l & 15) for dims (l >> 4) * 8 .. +8 and
// receives rows 4 * (l >> 4) + r of key (l & 15), so the 16 keys of one row
// sit in one DPP row of 16 lanes):
//   * kd_lse_kernel: per (64-row tile, layer, up to 4 heads of one KV head), an
//     online softmax over the row's keys gives each row's log-sum-exp (log2
//     units, in the workspace); each lane keeps statistics over its own keys
//     and the 16 lanes of a row are combined once at the end.  When the caller
//     already has these log-sum-exps (the dense forward pass of every layer
//     makes them), kd_lse_import_kernel copies them in instead;
//   * kd_target_kernel: per (16-row, 64-key) tile, every (layer, head) adds
//     exp(logit - lse) into the tile held in registers; the key operands of a
//     KV head are loaded once for all layers and heads of its group, the four
//     waves of a workgroup share their rows' query operands, and abar is
//     written once, with no atomics.
// Eq. 6: P = abar (a constant), Q = softmax(I_t) over the valid keys, I the
// unscaled index scores of Eq. 3 (computed by the indexer kernels); the loss
// is the mean over rows with at least one key of KL(P || Q), and
// dL/dI = (Q - P) / n_rows:
//   * kd_rows_kernel: per row, the log-sum-exp of I, the row's KL term and
//     Q - P, written over the scores;
//   * kd_loss_kernel: n_rows and the mean of the row terms (summed in double
//     in a fixed order);
//   * kd_dq_kernel / kd_dk_kernel: dq = dL/dI K_idx and dk = dL/dI^T Q_idx,
//     fp32 matrix-core products tiled through LDS (64 x 64 outputs per
//     workgroup, 32-deep steps).
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kKdLog2e = 1.4426950408889634f;
constexpr float kKdLn2 = 0.6931471805599453f;
constexpr int kKdDim = 128;  // attention head dimension
constexpr int kKdTile = 64;  // rows and keys per target tile
constexpr int kIdxDim = 256; // index vector width

struct KdArgs {
    const uint16_t *q_layers;  // [L, rows, Hq, 128]
    const uint16_t *k_cache;   // [B, max_len, Hkv, 128] | paged
    const int32_t *page_table, *seq_lens, *q_pos;
    float *lse2;               // [L, Hq, rows_pad], log2 units (rows_pad = rows + 16)
    float *abar;               // [rows, max_len]
    int n_layers, batch, n_q, rows, max_len, page_shift, max_pages, causal;
    int q_heads, kv_heads, group, row_tiles, key_tiles, rows_pad;
    float scale_log2, inv_lh;  // softmax_scale * log2(e), 1 / (L * Hq)
};

// 2^x by the hardware instruction alone: results below 2^-126 may flush to
// zero, which is far below every tolerance here (exp2f adds a rescaling for
// such results, five more VALU operations per call).
__device__ __forceinline__ float kd_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 kd_ld8(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// Key limits of the lane's four rows t0 + 4 * grp + r (0 for rows past n_q).
__device__ __forceinline__ void kd_row_limits(const KdArgs &a, int b, int t0, int grp,
                                              int (&n)[4]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int t = t0 + 4 * grp + r;
        n[r] = t < a.n_q ? valid_keys(a.seq_lens, a.q_pos, a.causal, b, b * a.n_q + t, a.max_len)
                         : 0;
    }
}

// A operands: query row t0 + col of layer l, head h (rows past n_q clamped).
__device__ __forceinline__ void kd_load_query(const KdArgs &a, int b, int t0, int l, int h,
                                              int col, int grp, bf16x8 (&qa)[4]) {
    const int t = min(t0 + col, a.n_q - 1);
    const uint16_t *p = a.q_layers +
                        (((size_t)l * a.rows + (size_t)b * a.n_q + t) * a.q_heads + h) * kKdDim +
                        grp * 8;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qa[kb] = kd_ld8(p + kb * 32);
}

// B operands of keys j0 + 16 * ct + col of KV head g (keys past len clamped to
// the last one; their logits are masked by the caller).  Paged caches: the four
// page-table reads are issued together, before the key reads.
template <bool PAGED>
__device__ __forceinline__ void kd_load_keys(const KdArgs &a, int b, int j0, int len, int g,
                                             int col, int grp, bf16x8 (&kv)[4][4]) {
    size_t tok[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
        const int j = min(j0 + 16 * ct + col, len - 1);
        if (PAGED) {
            const int page = a.page_table[(size_t)b * a.max_pages + (j >> a.page_shift)];
            tok[ct] = ((size_t)page << a.page_shift) + (j & ((1 << a.page_shift) - 1));
        } else {
            tok[ct] = (size_t)b * a.max_len + j;
        }
    }
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
        const uint16_t *p = a.k_cache + (tok[ct] * a.kv_heads + g) * kKdDim + grp * 8;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) kv[ct][kb] = kd_ld8(p + kb * 32);
    }
}

// Unscaled logits of the lane's 4 rows x 4 keys: c[ct][r] = row 4 * grp + r,
// key 16 * ct + col.
__device__ __forceinline__ void kd_logits(const bf16x8 (&qa)[4], const bf16x8 (&kv)[4][4],
                                          f32x4 (&c)[4]) {
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
        c[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
            c[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kb], kv[ct][kb], c[ct], 0, 0, 0);
    }
}

// Largest / smallest of a per-lane-group value over the four groups of a wave.
__device__ __forceinline__ int kd_groups_max(int v) {
    v = max(v, __shfl_xor(v, 16));
    return max(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ int kd_groups_min(int v) {
    v = min(v, __shfl_xor(v, 16));
    return min(v, __shfl_xor(v, 32));
}

// The log-sum-exps of every (layer, row, query head) supplied by the caller
// (natural log, [L, rows, Hq], as the dense attention returns them) into the
// statistics layout [L, Hq, rows_pad] in log2 units.  grid-stride over L*rows*Hq.
__global__ __launch_bounds__(256) void kd_lse_import_kernel(KdArgs a, const float *lse_in) {
    const size_t total = (size_t)a.n_layers * a.rows * a.q_heads;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (size_t)gridDim.x * 256) {
        const int h = (int)(i % a.q_heads);
        const size_t lr = i / a.q_heads;
        const int r = (int)(lr % a.rows), l = (int)(lr / a.rows);
        a.lse2[((size_t)l * a.q_heads + h) * a.rows_pad + r] = lse_in[i] * kKdLog2e;
    }
}

// IEEE maximum (gfx950 v_maximum3_f32; no operand canonicalisation).
__device__ __forceinline__ float kd_max(float x, float y) {
    return __builtin_elementwise_maximum(x, y);
}

// Online softmax statistics of the lane's four rows over the lane's own four
// keys of a tile, in log2 units: s is the sum of 2^(sl * z - base).  The base
// follows the running maximum lazily: it moves only when a logit exceeds it by
// more than 2^16 (then every row of the lane is rebased, on a branch the whole
// wave takes), so that the steady state needs no rescaling exponential.  Terms
// up to 2^16 keep the sums far from the fp32 range, and the relative precision
// of the sum does not depend on the base.
constexpr float kLazyMargin = 16.0f;

template <bool FULL>
__device__ __forceinline__ void kd_stats_update(const f32x4 (&c)[4], float sl, int j0, int col,
                                                const int (&n)[4], float (&base)[4],
                                                float (&s)[4]) {
    float v[4][4], tm[4];
    bool over = false;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
            v[r][ct] = FULL || j0 + 16 * ct + col < n[r] ? c[ct][r] : -INFINITY;
        tm[r] = kd_max(kd_max(v[r][0], v[r][1]), kd_max(v[r][2], v[r][3])) * sl;
        over |= tm[r] > base[r] + kLazyMargin;
    }
    if (__builtin_amdgcn_ballot_w64(over)) {  // rare: rebase every row of the wave
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float nb = kd_max(base[r], tm[r]);
            if (nb != -INFINITY) {
                s[r] *= kd_exp2(base[r] - nb);  // base = -inf: s is 0 anyway
                base[r] = nb;
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float b = base[r] == -INFINITY ? 0.0f : base[r];  // no key of the lane yet
        s[r] += (kd_exp2(fmaf(v[r][0], sl, -b)) + kd_exp2(fmaf(v[r][1], sl, -b))) +
                (kd_exp2(fmaf(v[r][2], sl, -b)) + kd_exp2(fmaf(v[r][3], sl, -b)));
    }
}

constexpr int kStagePitch = kKdDim + 8;  // bf16 per staged row (272 bytes): the 16 rows read
                                         // by one 16-lane group fall on distinct banks

// Log-sum-exp (log2 units) of every (layer, query head, row): a workgroup holds
// 64 rows (16 per wave) and HP heads of one KV head, the query operands in
// registers.  The key tiles of that KV head stream through LDS, double-buffered
// and shared by the four waves (one barrier per tile); each key tile serves HP
// heads.  grid: (((b * row_tiles + tile) * L + l) * (group / HP) + head block)
// * kv_heads + g, so that the workgroups of one KV head land on the same XCD
// when kv_heads divides 8.
template <int HP, bool PAGED>
__global__ __launch_bounds__(256) void kd_lse_kernel(KdArgs a) {
    __shared__ __align__(16) uint16_t s_k[2][kKdTile][kStagePitch];
    __shared__ int s_nmax[4];
    int x = blockIdx.x;
    const int g = x % a.kv_heads;
    x /= a.kv_heads;
    const int hsplit = a.group / HP;
    const int hs = x % hsplit;
    x /= hsplit;
    const int l = x % a.n_layers;
    x /= a.n_layers;
    const int tile = x % a.row_tiles, b = x / a.row_tiles;
    const int h0 = g * a.group + hs * HP;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int t0 = tile * kKdTile + wave * 16;
    const int len = clamp_len(a.seq_lens[b], a.max_len);
    int n[4];
    kd_row_limits(a, b, t0, grp, n);  // 0 for rows past n_q
    const int nmax = kd_groups_max(max(max(n[0], n[1]), max(n[2], n[3])));
    const int nmin = kd_groups_min(min(min(n[0], n[1]), min(n[2], n[3])));
    if (lane == 0) s_nmax[wave] = nmax;
    bf16x8 q[HP][4];
    if (t0 < a.n_q) {
#pragma unroll
        for (int hh = 0; hh < HP; ++hh) kd_load_query(a, b, t0, l, h0 + hh, col, grp, q[hh]);
    }
    float m[HP][4], s[HP][4];  // per head and row: base (log2 units) and sum
#pragma unroll
    for (int hh = 0; hh < HP; ++hh)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            m[hh][r] = -INFINITY;
            s[hh][r] = 0.0f;
        }
    __syncthreads();
    const int wg_max = max(max(s_nmax[0], s_nmax[1]), max(s_nmax[2], s_nmax[3]));
    const int tiles = div_up(wg_max, kKdTile);

    // staging: thread -> key row kr of the tile, 16-byte pieces 4 * kq .. 4 * kq + 3
    const int kr = tid >> 2, kq = tid & 3;
    auto fetch = [&](int u, u32x4 (&v)[4]) {
        const int j = min(u * kKdTile + kr, len - 1);
        size_t tok;
        if (PAGED) {
            const int page = a.page_table[(size_t)b * a.max_pages + (j >> a.page_shift)];
            tok = ((size_t)page << a.page_shift) + (j & ((1 << a.page_shift) - 1));
        } else {
            tok = (size_t)b * a.max_len + j;
        }
        const uint16_t *p = a.k_cache + (tok * a.kv_heads + g) * kKdDim + kq * 32;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = *reinterpret_cast<const u32x4 *>(p + i * 8);
    };
    auto stage = [&](int buf, const u32x4 (&v)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            *reinterpret_cast<u32x4 *>(&s_k[buf][kr][kq * 32 + i * 8]) = v[i];
    };
    u32x4 v[4];
    if (tiles > 0) {
        fetch(0, v);
        stage(0, v);
    }
    __syncthreads();
    for (int u = 0; u < tiles; ++u) {
        if (u + 1 < tiles) fetch(u + 1, v);
        const int j0 = u * kKdTile;
        if (j0 < nmax) {  // uniform per wave
            const int buf = u & 1;
            bf16x8 kv[4][4];
#pragma unroll
            for (int ct = 0; ct < 4; ++ct)
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
                    kv[ct][kb] = *reinterpret_cast<const bf16x8 *>(
                        &s_k[buf][16 * ct + col][kb * 32 + grp * 8]);
            const bool full = j0 + kKdTile <= nmin;
#pragma unroll
            for (int hh = 0; hh < HP; ++hh) {
                f32x4 c[4];
                kd_logits(q[hh], kv, c);
                if (full) kd_stats_update<true>(c, a.scale_log2, j0, col, n, m[hh], s[hh]);
                else kd_stats_update<false>(c, a.scale_log2, j0, col, n, m[hh], s[hh]);
            }
        }
        if (u + 1 < tiles) stage((u + 1) & 1, v);
        __syncthreads();
    }
    if (t0 >= a.n_q) return;
#pragma unroll
    for (int hh = 0; hh < HP; ++hh)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float mr = row16_max(m[hh][r]);
            const float part = m[hh][r] == -INFINITY ? 0.0f : s[hh][r] * exp2f(m[hh][r] - mr);
            const float sr = row16_sum(part);
            const int t = t0 + 4 * grp + r;
            if (col == 0 && t < a.n_q)
                a.lse2[((size_t)l * a.q_heads + h0 + hh) * a.rows_pad + (size_t)b * a.n_q + t] =
                    n[r] > 0 ? mr + log2f(sr) : -INFINITY;
        }
}

constexpr int kTgtChunk = 4;              // (layer, head) combinations per LDS stage
constexpr int kTgtWaveTiles = 1;          // 64-key tiles per wave in the target pass

template <bool FULL>
__device__ __forceinline__ void kd_accumulate(float sl, const bf16x8 (&qa)[4],
                                              const float4 &lse, const bf16x8 (&kv)[4][4],
                                              int j0, int col, const int (&n)[4],
                                              f32x4 (&acc)[4]) {
    f32x4 c[4];
    kd_logits(qa, kv, c);
    const float lr[4] = {lse.x, lse.y, lse.z, lse.w};
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float e = kd_exp2(fmaf(c[ct][r], sl, -lr[r]));
            if (FULL) acc[ct][r] += e;
            else acc[ct][r] += j0 + 16 * ct + col < n[r] ? e : 0.0f;
        }
}

// A workgroup covers 16 rows x (4 * kTgtWaveTiles * 64) keys: each of its four
// waves holds the key operands of kTgtWaveTiles 64-key tiles of the current KV
// head in registers, and the query operands and log-sum-exps of the 16 rows
// are staged through LDS, kTgtChunk (layer, head) combinations at a time,
// double-buffered: the next stage's global reads are in flight while the
// current one is on the matrix cores, one barrier per stage.  Each staged query
// tile serves every key tile of the workgroup, so the query traffic per output
// falls with the keys a workgroup covers.  Workgroups are dealt to the 8 XCDs
// in turn; the mapping gives every key block of a row block to the same XCD,
// one after another, so the 2 MB of query operands of a row block (16 rows x
// every layer and head) are read from that XCD's L2 as far as it holds them.
// grid: ((row block group * key_blocks + key block) * 8 + xcd); row block
// index over all sequences = row block group * 8 + xcd.
template <int G, bool PAGED>  // G: query heads per KV head
__global__ __launch_bounds__(256) void kd_target_kernel(KdArgs a) {
    constexpr int KT = kTgtWaveTiles;
    __shared__ __align__(16) uint16_t s_q[2][kTgtChunk][16][kStagePitch];
    __shared__ __align__(16) float s_l[2][kTgtChunk][16];
    const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
    const int kblk = local % a.key_tiles;
    const int rb_all = (local / a.key_tiles) * 8 + xcd;
    if (rb_all >= a.batch * a.row_tiles) return;  // padding of the last group (uniform)
    const int rblk = rb_all % a.row_tiles, b = rb_all / a.row_tiles;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int t0 = rblk * 16;
    const int jw = (kblk * 4 + wave) * KT * kKdTile;  // this wave's first key
    int n[4];
    kd_row_limits(a, b, t0, grp, n);
    const int nmax = kd_groups_max(max(max(n[0], n[1]), max(n[2], n[3])));
    const int nmin = kd_groups_min(min(min(n[0], n[1]), min(n[2], n[3])));
    if (kblk * 4 * KT * kKdTile >= nmax) return;  // no valid key in the block (uniform)
    const bool active = jw < nmax;                 // this wave's tiles hold valid keys
    const bool full = jw + KT * kKdTile <= nmin;
    const int len = clamp_len(a.seq_lens[b], a.max_len);

    // staging: thread -> (row sr, 16-byte piece sd) of every combination of a stage
    const int sr = tid >> 4, sd = tid & 15;
    const size_t layer_q = (size_t)a.rows * a.q_heads * kKdDim;
    const uint16_t *qsrc = a.q_layers +
                           ((size_t)b * a.n_q + min(t0 + sr, a.n_q - 1)) * a.q_heads * kKdDim +
                           sd * 8;
    // Combination ci = l * G + hh of KV head g is (layer l, query head g * G + hh);
    // a stage holds kTgtChunk consecutive combinations of one KV head.  G is a
    // compile-time constant, so the index arithmetic has no division.
    const int combos = a.n_layers * G;
    const int nchunk = div_up(combos, kTgtChunk);
    auto fetch = [&](int g, int c0, u32x4 (&v)[kTgtChunk], float &lv) {
#pragma unroll
        for (int c = 0; c < kTgtChunk; ++c) {
            const int ci = min(c0 + c, combos - 1);
            const int l = ci / G, h = g * G + ci % G;
            v[c] = *reinterpret_cast<const u32x4 *>(qsrc + l * layer_q + (size_t)h * kKdDim);
        }
        if (tid < kTgtChunk * 16) {
            const int ci = min(c0 + (tid >> 4), combos - 1);
            const int l = ci / G, h = g * G + ci % G;
            lv = a.lse2[((size_t)l * a.q_heads + h) * a.rows_pad + (size_t)b * a.n_q + t0 +
                        (tid & 15)];
        }
    };
    auto stage = [&](int buf, const u32x4 (&v)[kTgtChunk], float lv) {
#pragma unroll
        for (int c = 0; c < kTgtChunk; ++c)
            *reinterpret_cast<u32x4 *>(&s_q[buf][c][sr][sd * 8]) = v[c];
        if (tid < kTgtChunk * 16) s_l[buf][tid >> 4][tid & 15] = lv;
    };

    f32x4 acc[KT][4];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) acc[kt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    u32x4 v[kTgtChunk];
    float lv = 0.0f;
    fetch(0, 0, v, lv);
    stage(0, v, lv);
    __syncthreads();
    bf16x8 kv[KT][4][4];
    // stage u = (KV head g, block k of kTgtChunk combinations), walked in order
    int g = 0, k = 0, buf = 0;
    for (;;) {
        if (k == 0 && active) {
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
                kd_load_keys<PAGED>(a, b, jw + kt * kKdTile, len, g, col, grp, kv[kt]);
        }
        const int k1 = k + 1 == nchunk ? 0 : k + 1, g1 = k + 1 == nchunk ? g + 1 : g;
        const bool more = g1 < a.kv_heads;
        if (more) fetch(g1, k1 * kTgtChunk, v, lv);
        if (active) {
#pragma unroll
            for (int c = 0; c < kTgtChunk; ++c) {
                if (k * kTgtChunk + c >= combos) break;  // uniform: short last stage
                bf16x8 qa[4];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
                    qa[kb] = *reinterpret_cast<const bf16x8 *>(&s_q[buf][c][col][kb * 32 + grp * 8]);
                const float4 lse = *reinterpret_cast<const float4 *>(&s_l[buf][c][4 * grp]);
#pragma unroll
                for (int kt = 0; kt < KT; ++kt) {
                    if (full)
                        kd_accumulate<true>(a.scale_log2, qa, lse, kv[kt], jw + kt * kKdTile, col,
                                            n, acc[kt]);
                    else
                        kd_accumulate<false>(a.scale_log2, qa, lse, kv[kt], jw + kt * kKdTile,
                                             col, n, acc[kt]);
                }
            }
        }
        if (more) stage(buf ^ 1, v, lv);
        __syncthreads();
        if (!more) break;
        g = g1;
        k = k1;
        buf ^= 1;
    }
    if (!active) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int t = t0 + 4 * grp + r;
        float *row = a.abar + ((size_t)b * a.n_q + t) * a.max_len;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int ct = 0; ct < 4; ++ct) {
                const int j = jw + kt * kKdTile + 16 * ct + col;
                if (j < n[r]) row[j] = acc[kt][ct][r] * a.inv_lh;
            }
    }
}

struct KdLossArgs {
    const float *abar;         // [rows, max_len]
    float *dI;                 // [rows, max_len]: index scores in, Q - P out
    float *row_kl;             // [rows]
    float *stats;              // [0] = 1 / n_rows (0 when none), [1] = n_rows
    int32_t *step_max;         // [B, ceil(n_q / 32)]: most keys of any row of each 32-row step
    float *loss;
    const uint16_t *q_idx;     // [rows, 256]
    const uint16_t *k_idx;     // index-key cache
    float *dq, *dk;
    const int32_t *page_table, *seq_lens, *q_pos;
    int n_q, rows, max_len, page_shift, max_pages, causal, row_tiles, key_tiles;
};

// One workgroup of 256 threads per row.
__global__ __launch_bounds__(256) void kd_rows_kernel(KdLossArgs a) {
    __shared__ float red_m[4], red_s[4];
    const int row = blockIdx.x, b = row / a.n_q;
    const int tid = threadIdx.x, wave = tid >> 6;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    if (n == 0) {  // uniform: no keys, no loss term
        if (tid == 0) a.row_kl[row] = 0.0f;
        return;
    }
    float *s = a.dI + (size_t)row * a.max_len;
    const float *p = a.abar + (size_t)row * a.max_len;
    float m = -INFINITY, sum = 0.0f;  // log2 units
    for (int j = tid; j < n; j += 256) {
        const float x = s[j] * kKdLog2e;
        if (x > m) {
            sum = sum * exp2f(m - x) + 1.0f;
            m = x;
        } else {
            sum += exp2f(x - m);
        }
    }
    const float wm = wave_max(m);
    const float ws = wave_sum(sum > 0.0f ? sum * exp2f(m - wm) : 0.0f);
    if ((tid & 63) == 0) {
        red_m[wave] = wm;
        red_s[wave] = ws;
    }
    __syncthreads();
    const float bm = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
    float bs = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) bs += red_s[w] > 0.0f ? red_s[w] * exp2f(red_m[w] - bm) : 0.0f;
    const float lse2 = bm + log2f(bs);
    float kl = 0.0f;  // log2 units
    for (int j = tid; j < n; j += 256) {
        const float z = fmaf(s[j], kKdLog2e, -lse2);
        const float pj = p[j];
        if (pj > 0.0f) kl += pj * (log2f(pj) - z);
        s[j] = exp2f(z) - pj;
    }
    kl = wave_sum(kl);
    __syncthreads();  // red_s reads above are done
    if ((tid & 63) == 0) red_s[wave] = kl;
    __syncthreads();
    if (tid == 0) a.row_kl[row] = (red_s[0] + red_s[1] + red_s[2] + red_s[3]) * kKdLn2;
}

// One workgroup: n_rows, 1 / n_rows and the mean row term.
__global__ __launch_bounds__(256) void kd_loss_kernel(KdLossArgs a) {
    __shared__ double red_t[256];
    __shared__ int red_c[256];
    const int tid = threadIdx.x;
    double tot = 0.0;
    int cnt = 0;
    for (int r = tid; r < a.rows; r += 256) {
        tot += (double)a.row_kl[r];
        cnt += valid_keys(a.seq_lens, a.q_pos, a.causal, r / a.n_q, r, a.max_len) > 0;
    }
    red_t[tid] = tot;
    red_c[tid] = cnt;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (tid < w) {
            red_t[tid] += red_t[tid + w];
            red_c[tid] += red_c[tid + w];
        }
        __syncthreads();
    }
    if (tid == 0) {
        const int nr = red_c[0];
        a.loss[0] = nr > 0 ? (float)(red_t[0] / nr) : 0.0f;
        a.stats[0] = nr > 0 ? 1.0f / (float)nr : 0.0f;
        a.stats[1] = (float)nr;
    }
}

constexpr int kGemmDepth = 32;  // contraction steps per LDS stage
constexpr int kRowPitch = 36;   // [row][key] staging: the MFMA reads (16 rows x 4 keys) and the
                                // row-contiguous stores both fall on distinct banks
constexpr int kColPitch = 80;   // [k][column] staging: the MFMA reads (4 k x 16 columns) fall
                                // on distinct banks

// 8 bf16 -> 8 floats stored at dst (16-byte aligned).
__device__ __forceinline__ void kd_store8(float *dst, u32x4 v) {
    float4 lo = make_float4(bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y));
    float4 hi = make_float4(bf16_lo(v.z), bf16_hi(v.z), bf16_lo(v.w), bf16_hi(v.w));
    *reinterpret_cast<float4 *>(dst) = lo;
    *reinterpret_cast<float4 *>(dst + 4) = hi;
}

// The gradient products run on v_mfma_f32_16x16x4_f32 (fp32 operands, so the
// bf16 keys and queries enter exactly and dL/dI keeps its fp32 bits): lane l
// supplies A[l & 15][l >> 4] and B[l >> 4][l & 15] and receives C rows
// 4 * (l >> 4) + r of column l & 15.  A workgroup computes 64 x 64 outputs,
// each wave 16 rows x 64 columns (four column tiles), 32 contraction steps per
// LDS stage.

// step_max[b, s] = the most valid keys of any row of rows 32 s .. 32 s + 31 of
// sequence b.  One thread per (sequence, step).
__global__ __launch_bounds__(256) void kd_step_max_kernel(KdLossArgs a, int total) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int nsteps = div_up(a.n_q, kGemmDepth);
    const int b = i / nsteps, r0 = (i % nsteps) * kGemmDepth;
    int m = 0;
    for (int k = 0; k < kGemmDepth && r0 + k < a.n_q; ++k)
        m = max(m, valid_keys(a.seq_lens, a.q_pos, a.causal, b, b * a.n_q + r0 + k, a.max_len));
    a.step_max[i] = m;
}

// dq[b,t,c] = (1 / n_rows) sum_{j < n(b,t)} dI[b,t,j] k_idx[b,j,c].
// grid: ((b * row_tiles + tile) * 4 + column tile), 64 rows x 64 columns each.
__global__ __launch_bounds__(256) void kd_dq_kernel(KdLossArgs a) {
    __shared__ __align__(16) float As[64][kRowPitch];           // [row][key]
    __shared__ __align__(16) float Bs[kGemmDepth][kColPitch];   // [key][column]
    __shared__ int s_n[64];
    int x = blockIdx.x;
    const int c0 = (x & 3) * 64;
    x >>= 2;
    const int tile = x % a.row_tiles, b = x / a.row_tiles;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 15, kq = lane >> 4;
    const int t0 = tile * 64;
    if (tid < 64) {
        const int t = t0 + tid;
        s_n[tid] = t < a.n_q ? valid_keys(a.seq_lens, a.q_pos, a.causal, b, b * a.n_q + t, a.max_len)
                             : 0;
    }
    __syncthreads();
    int nmax = 0;
    for (int i = 0; i < 64; ++i) nmax = max(nmax, s_n[i]);
    f32x4 acc[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ak = tid & 31, ai = tid >> 5;        // A loads: key ak, rows ai + 8 * step
    const int bk = tid >> 3, bc = (tid & 7) * 8;   // B loads: key bk, columns bc .. bc + 7
    int nrow[8];
#pragma unroll
    for (int st = 0; st < 8; ++st) nrow[st] = s_n[ai + 8 * st];
    // one stage's operands, read into registers a stage ahead of their use
    float av_n[8];
    u32x4 kv_n;
    auto fetch = [&](int j0) {
        const int j = j0 + ak;
#pragma unroll
        for (int st = 0; st < 8; ++st)
            av_n[st] = j < nrow[st]
                           ? a.dI[((size_t)b * a.n_q + t0 + ai + 8 * st) * a.max_len + j]
                           : 0.0f;
        const int jb = j0 + bk;
        kv_n = u32x4{0u, 0u, 0u, 0u};
        if (jb < nmax)
            kv_n = *reinterpret_cast<const u32x4 *>(
                a.k_idx + token_offset(a.page_table, a.page_shift, a.max_pages, a.max_len, b, jb,
                                       kIdxDim) +
                c0 + bc);
    };
    if (nmax > 0) fetch(0);
    for (int j0 = 0; j0 < nmax; j0 += kGemmDepth) {
#pragma unroll
        for (int st = 0; st < 8; ++st) As[ai + 8 * st][ak] = av_n[st];
        kd_store8(&Bs[bk][bc], kv_n);
        __syncthreads();
        if (j0 + kGemmDepth < nmax) fetch(j0 + kGemmDepth);
#pragma unroll
        for (int kk = 0; kk < kGemmDepth; kk += 4) {
            const float av = As[wave * 16 + col][kk + kq];
#pragma unroll
            for (int ct = 0; ct < 4; ++ct)
                acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, Bs[kk + kq][ct * 16 + col],
                                                               acc[ct], 0, 0, 0);
        }
        __syncthreads();
    }
    const float inv_n = a.stats[0];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int t = t0 + wave * 16 + 4 * kq + r;
        if (t < a.n_q) {
            float *dst = a.dq + ((size_t)b * a.n_q + t) * kIdxDim + c0 + col;
#pragma unroll
            for (int ct = 0; ct < 4; ++ct) dst[ct * 16] = acc[ct][r] * inv_n;
        }
    }
}

// dk[b,j,c] = (1 / n_rows) sum_{t : j < n(b,t)} dI[b,t,j] q_idx[b,t,c], for j < seq_lens[b].
// grid: ((b * key_tiles + tile) * 4 + column tile), 64 keys x 64 columns each.
__global__ __launch_bounds__(256) void kd_dk_kernel(KdLossArgs a) {
    __shared__ __align__(16) float As[kGemmDepth][kColPitch];  // [row][key]
    __shared__ __align__(16) float Bs[kGemmDepth][kColPitch];  // [row][column]
    int x = blockIdx.x;
    const int c0 = (x & 3) * 64;
    x >>= 2;
    const int tile = x % a.key_tiles, b = x / a.key_tiles;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 15, kq = lane >> 4;
    const int j0 = tile * 64;
    const int len = clamp_len(a.seq_lens[b], a.max_len);
    if (j0 >= len) return;  // uniform: no token of this tile is written
    f32x4 acc[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ai = tid & 63, ak = tid >> 6;        // A loads: key ai, rows ak + 4 * step
    const int bk = tid >> 3, bc = (tid & 7) * 8;   // B loads: row bk, columns bc .. bc + 7
    // one step's operands (32 rows from r0), read into registers a step ahead
    float av_n[8];
    u32x4 qv_n;
    auto fetch = [&](int r0) {
#pragma unroll
        for (int st = 0; st < 8; ++st) {
            const int t = r0 + ak + 4 * st;
            const int nk = t < a.n_q ? valid_keys(a.seq_lens, a.q_pos, a.causal, b, b * a.n_q + t,
                                                  a.max_len)
                                     : 0;
            av_n[st] = j0 + ai < nk ? a.dI[((size_t)b * a.n_q + t) * a.max_len + j0 + ai] : 0.0f;
        }
        const int t = r0 + bk;
        qv_n = u32x4{0u, 0u, 0u, 0u};
        if (t < a.n_q)
            qv_n = *reinterpret_cast<const u32x4 *>(a.q_idx + ((size_t)b * a.n_q + t) * kIdxDim +
                                                    c0 + bc);
    };
    // Only the steps with a row that sees one of the tile's keys contribute
    // (in a causal sequence, those from the tile's own position on): 256 steps
    // at a time, their per-step key maxima give an ordered list of the useful
    // ones (wave ballots, so the summation order is fixed), and the loop runs
    // over that list with the next step's operands in flight.
    __shared__ int s_list[256];
    __shared__ int s_wcnt[4];
    const int nsteps = div_up(a.n_q, kGemmDepth);
    const int32_t *smax = a.step_max + (size_t)b * nsteps;
    for (int s0 = 0; s0 < nsteps; s0 += 256) {
        const int st_i = s0 + tid;
        const bool useful = st_i < nsteps && smax[st_i] > j0;
        const uint64_t m = __builtin_amdgcn_ballot_w64(useful);
        const int before = __builtin_popcountll(m & ((1ull << lane) - 1ull));
        if (lane == 0) s_wcnt[wave] = __builtin_popcountll(m);
        __syncthreads();
        int off = 0;
        for (int w = 0; w < wave; ++w) off += s_wcnt[w];
        const int cnt = s_wcnt[0] + s_wcnt[1] + s_wcnt[2] + s_wcnt[3];
        if (useful) s_list[off + before] = st_i;
        __syncthreads();
        if (cnt > 0) fetch(s_list[0] * kGemmDepth);
        for (int i = 0; i < cnt; ++i) {
#pragma unroll
            for (int st = 0; st < 8; ++st) As[ak + 4 * st][ai] = av_n[st];
            kd_store8(&Bs[bk][bc], qv_n);
            __syncthreads();
            if (i + 1 < cnt) fetch(s_list[i + 1] * kGemmDepth);
#pragma unroll
            for (int kk = 0; kk < kGemmDepth; kk += 4) {
                const float av = As[kk + kq][wave * 16 + col];
#pragma unroll
                for (int ct = 0; ct < 4; ++ct)
                    acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, Bs[kk + kq][ct * 16 + col],
                                                                   acc[ct], 0, 0, 0);
            }
            __syncthreads();  // As / Bs and s_list are rewritten next
        }
    }
    const float inv_n = a.stats[0];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int j = j0 + wave * 16 + 4 * kq + r;
        if (j < len) {
            float *dst = a.dk + token_offset(a.page_table, a.page_shift, a.max_pages, a.max_len, b,
                                             j, kIdxDim) +
                         c0 + col;
#pragma unroll
            for (int ct = 0; ct < 4; ++ct) dst[ct * 16] = acc[ct][r] * inv_n;
        }
    }
}

static bool grid_fits(long long n) { return n >= 1 && n <= 0x7fffffffLL; }

// Row blocks of 16 and key blocks of 256 for the target pass; the lane offsets
// into one layer's queries must fit 32 bits.
bool kd_target_supported(const Geometry &g, int n_layers) {
    const long long tiles = (long long)g.batch * div_up(g.n_q, kKdTile);
    const long long blocks = (long long)g.batch * div_up(g.n_q, 16);
    return n_layers >= 1 && grid_fits(tiles * n_layers * g.q_heads) &&
           grid_fits((blocks + 7) / 8 * 8 * div_up(g.max_len, 4 * kTgtWaveTiles * kKdTile)) &&
           (long long)g.rows * g.q_heads * kKdDim * 2 < (1LL << 31);
}

size_t kd_target_ws_floats(const Geometry &g, int n_layers) {
    return (size_t)n_layers * g.q_heads * ((size_t)g.rows + 16);
}

hipError_t launch_kd_target(const Geometry &g, int n_layers, const void *q_layers,
                            const void *k_cache, const int32_t *page_table,
                            const int32_t *seq_lens, const int32_t *q_pos, const float *lse_in,
                            float *abar, float *lse2, hipStream_t stream, hipEvent_t between) {
    if (!kd_target_supported(g, n_layers)) return hipErrorInvalidValue;
    KdArgs a;
    a.q_layers = static_cast<const uint16_t *>(q_layers);
    a.k_cache = static_cast<const uint16_t *>(k_cache);
    a.page_table = page_table;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.lse2 = lse2;
    a.abar = abar;
    a.n_layers = n_layers;
    a.batch = g.batch;
    a.n_q = g.n_q;
    a.rows = g.rows;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.causal = g.causal;
    a.q_heads = g.q_heads;
    a.kv_heads = g.kv_heads;
    a.group = g.group;
    a.row_tiles = div_up(g.n_q, kKdTile);
    a.key_tiles = div_up(g.max_len, kKdTile);
    a.rows_pad = g.rows + 16;
    a.scale_log2 = g.softmax_scale * kKdLog2e;
    a.inv_lh = 1.0f / ((float)n_layers * (float)g.q_heads);
    const long long tiles = (long long)g.batch * a.row_tiles;
    // heads per workgroup of the statistics pass (a divisor of the group)
    const int hp = g.group == 8 ? 4 : g.group;
    const dim3 lse_grid((unsigned)(tiles * n_layers * (g.group / hp) * g.kv_heads));
    const bool paged = g.page_shift >= 0;
    if (lse_in) {  // the caller's log-sum-exps: no statistics pass
        const size_t total = (size_t)n_layers * g.rows * g.q_heads;
        const size_t blocks = (total + 255) / 256;
        kd_lse_import_kernel<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                               stream>>>(a, lse_in);
    } else {
#define KD_LSE(HP)                                                              \
    (paged ? kd_lse_kernel<HP, true><<<lse_grid, dim3(256), 0, stream>>>(a)    \
           : kd_lse_kernel<HP, false><<<lse_grid, dim3(256), 0, stream>>>(a))
        switch (hp) {
            case 1: KD_LSE(1); break;
            case 2: KD_LSE(2); break;
            case 4: KD_LSE(4); break;
            case 5: KD_LSE(5); break;
            default: return hipErrorInvalidValue;
        }
#undef KD_LSE
    }
    if (between && hipEventRecord(between, stream) != hipSuccess) return hipErrorUnknown;
    // the target pass: 16-row blocks x (4 waves x kTgtWaveTiles x 64)-key blocks
    a.row_tiles = div_up(g.n_q, 16);
    a.key_tiles = div_up(g.max_len, 4 * kTgtWaveTiles * kKdTile);
    const long long groups = ((long long)g.batch * a.row_tiles + 7) / 8;
    const dim3 tgt_grid((unsigned)(groups * a.key_tiles * 8));
#define KD_TGT(G)                                                                  \
    (paged ? kd_target_kernel<G, true><<<tgt_grid, dim3(256), 0, stream>>>(a)     \
           : kd_target_kernel<G, false><<<tgt_grid, dim3(256), 0, stream>>>(a))
    switch (g.group) {
        case 1: KD_TGT(1); break;
        case 2: KD_TGT(2); break;
        case 4: KD_TGT(4); break;
        case 5: KD_TGT(5); break;
        case 8: KD_TGT(8); break;
        default: return hipErrorInvalidValue;
    }
#undef KD_TGT
    return hipGetLastError();
}

bool kd_loss_supported(const Geometry &g) {
    return grid_fits((long long)g.batch * div_up(g.n_q, 64) * 4) &&
           grid_fits((long long)g.batch * div_up(g.max_len, 64) * 4);
}

size_t kd_loss_ws_floats(const Geometry &g) {
    // scores / dL/dI, row terms, 2 statistics, per-step key maxima (int32)
    return (size_t)g.rows * g.max_len + g.rows + 2 + (size_t)g.batch * div_up(g.n_q, 32);
}

hipError_t launch_kd_loss(const Geometry &g, const float *abar, const void *q_idx,
                          const void *k_idx, const int32_t *page_table, const int32_t *seq_lens,
                          const int32_t *q_pos, float *loss, float *dq, float *dk, float *ws,
                          hipStream_t stream, hipEvent_t after_scores, hipEvent_t after_loss) {
    if (!kd_loss_supported(g)) return hipErrorInvalidValue;
    KdLossArgs a;
    a.abar = abar;
    a.dI = ws;
    a.row_kl = ws + (size_t)g.rows * g.max_len;
    a.stats = a.row_kl + g.rows;
    a.step_max = reinterpret_cast<int32_t *>(a.stats + 2);
    a.loss = loss;
    a.q_idx = static_cast<const uint16_t *>(q_idx);
    a.k_idx = static_cast<const uint16_t *>(k_idx);
    a.dq = dq;
    a.dk = dk;
    a.page_table = page_table;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.n_q = g.n_q;
    a.rows = g.rows;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.causal = g.causal;
    a.row_tiles = div_up(g.n_q, 64);
    a.key_tiles = div_up(g.max_len, 64);
    // The scores of Eq. 3 for every valid (row, key), then the row terms in place.
    hipError_t e = index_uses_mfma(g)
                       ? launch_index_prefill(g, q_idx, k_idx, page_table, seq_lens, q_pos, a.dI,
                                              nullptr, stream)
                       : launch_index_scores(g, q_idx, k_idx, page_table, seq_lens, q_pos, a.dI,
                                             nullptr, nullptr, stream);
    if (e != hipSuccess) return e;
    if (after_scores && hipEventRecord(after_scores, stream) != hipSuccess) return hipErrorUnknown;
    kd_rows_kernel<<<dim3(g.rows), dim3(256), 0, stream>>>(a);
    kd_loss_kernel<<<dim3(1), dim3(256), 0, stream>>>(a);
    if (after_loss && hipEventRecord(after_loss, stream) != hipSuccess) return hipErrorUnknown;
    const int steps_total = g.batch * div_up(g.n_q, kGemmDepth);
    kd_step_max_kernel<<<dim3(div_up(steps_total, 256)), dim3(256), 0, stream>>>(a, steps_total);
    kd_dq_kernel<<<dim3((unsigned)(g.batch * a.row_tiles * 4)), dim3(256), 0, stream>>>(a);
    kd_dk_kernel<<<dim3((unsigned)(g.batch * a.key_tiles * 4)), dim3(256), 0, stream>>>(a);
    return hipGetLastError();
}

hipError_t take_device_error_kd(uint32_t *bits) { return take_source_device_error(bits); }

}  // namespace clsa
