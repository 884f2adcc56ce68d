// Exact token-level top-k (Section 2.1, Eq. 3: S_t = TopK(I_t, k)).
//
// No sort.  The exact k-th largest key tau is found with a radix select on the
// order-preserving uint32 keys of the fp32 scores, then the selected positions
// are emitted in ascending order:
//
//   1. coarse histogram of the top 11 key bits (made by the indexer as it writes
//      the scores, or by coarse_hist_kernel) -> bin b1 holding the k-th key;
//   2. filter pass over the row: keys above b1 are certainly selected (bitmap
//      words built with wavefront ballots), keys in b1 go to a candidate list;
//   3. two radix passes (11 + 10 bits) over the candidates in LDS -> tau and
//      r, the number of keys equal to tau still to be taken;
//   4. candidates above tau are added to the "sure" bitmap, those equal to tau
//      to a "tie" bitmap;
//   5. a block-wide scan of the bitmaps' popcounts gives each word its output
//      offset; of the ties only the first r in position order are kept (ties
//      go to the lowest index).
//
// Two shapes of the same algorithm:
//   * topk_row_kernel: one 1024-thread workgroup per row, bitmaps and the
//     candidate list in LDS -- for many long rows (chunked prefill);
//   * for the few, long rows of decode, step 2 is spread over many 256-thread
//     workgroups (topk_filter_kernel, 4096 keys each, writing a global bitmap
//     and, per wave, its candidates into a region of its own) and a second
//     launch with one workgroup per row (topk_finish_kernel) does steps 3-5
//     with the bitmaps in LDS and the candidates in registers.  The hand-off
//     goes through the kernel boundary: the finish works with 1024 threads per
//     row, the filter with 256-thread workgroups, so a last-arriver finish (as
//     the attention kernel merges its splits) would run on a quarter of the
//     threads.
// If the per-row kernel's candidate list overflows (very flat score rows),
// steps 3-4 re-read the row instead: slower, same result.  The regions of the
// wide path hold every key of their wave, so they never overflow.
// Rows of at most kTopkRowMaxLen keys take a third form (topk_short_kernel):
// the row in registers, tau fixed 4 bits at a time by counting, no bitmaps.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

// Refinement digits below the coarse one: bits 20..10, then 9..0.
constexpr int kMidShift = 10;
constexpr int kMidBins = 1 << (kCoarseShift - kMidShift);  // 2048
constexpr int kLowBins = 1 << kMidShift;                   // 1024
constexpr int kHistWords = kCoarseBins > kMidBins ? kCoarseBins : kMidBins;
constexpr int kWideThreads = 256;
constexpr int kWideChunk = 4096;  // keys filtered by one wide workgroup (16 per thread)
constexpr int kRowThreads = 1024;

// Inclusive prefix sum over the 64 lanes of a wave (every lane active): DPP
// row shifts by 1, 2, 4 and 8 inside each row of 16 lanes (a lane whose source
// lies outside its row adds 0), then the totals of the rows below are read
// with v_readlane.  No LDS round trips.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 15);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 31);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 47);
    const int row = lane >> 4;
    return v + (row > 0 ? r0 : 0u) + (row > 1 ? r1 : 0u) + (row > 2 ? r2 : 0u);
}

// Exclusive prefix sums over the workgroup of two values per thread, and their
// totals.  s_wave: 2 * NT / 64 entries.  One barrier to publish the wave totals
// (each thread then adds those of the waves before its own) and one before
// s_wave may be reused.
template <int NT>
__device__ __forceinline__ void block_excl_scan2(uint32_t x, uint32_t y, uint32_t *s_wave,
                                                 uint32_t &x_before, uint32_t &y_before,
                                                 uint32_t &x_total, uint32_t &y_total) {
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t xi = wave_incl_scan(x, lane), yi = wave_incl_scan(y, lane);
    if (lane == 63) {
        s_wave[wave] = xi;
        s_wave[NW + wave] = yi;
    }
    __syncthreads();
    uint32_t xo = 0, yo = 0, xs = 0, ys = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const uint32_t u = s_wave[w], v = s_wave[NW + w];
        xs += u;
        ys += v;
        xo += w < wave ? u : 0u;
        yo += w < wave ? v : 0u;
    }
    x_before = xo + xi - x;
    y_before = yo + yi - y;
    x_total = xs;
    y_total = ys;
    __syncthreads();
}

// Given hist[NBINS] in LDS, find the bin b with suffix(b) >= need > suffix(b+1),
// suffix(x) = the keys in bins >= x, and write b and suffix(b+1) to out[0..1]
// ((0, 0) if no bin qualifies, which consistent counts never produce).  One
// wave searches in two levels: lane l sums the NBINS/64 bins just below
// NBINS - l * NBINS/64, so an inclusive prefix over lanes is a suffix over
// bins and the first lane whose prefix reaches `need` holds b; then lane i
// takes that lane's i-th bin from the top, and a second prefix and ballot
// locate b itself.  Every thread of the workgroup calls this (it ends with a
// barrier).
template <int NBINS>
__device__ __forceinline__ void find_threshold_bin(const uint32_t *hist, uint32_t need,
                                                   uint32_t *out) {
    constexpr int PER = NBINS / 64;
    static_assert(PER % 4 == 0 && PER <= 64, "bins are read four at a time, one per lane");
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        uint32_t sum = 0;
#pragma unroll
        for (int i = 0; i < PER; i += 4) {
            const uint4 v = *reinterpret_cast<const uint4 *>(hist + NBINS - (lane + 1) * PER + i);
            sum += (v.x + v.y) + (v.z + v.w);
        }
        const uint32_t inc = wave_incl_scan(sum, lane);
        const uint64_t reach = __ballot(inc >= need);
        if (reach == 0) {
            if (lane == 0) {
                out[0] = 0u;
                out[1] = 0u;
            }
        } else {
            const int owner = __builtin_ctzll(reach);
            const uint32_t above = (uint32_t)__builtin_amdgcn_readlane((int)(inc - sum), owner);
            const int top = NBINS - owner * PER - 1;  // the owner's highest bin
            const uint32_t c = lane < PER ? hist[top - lane] : 0u;
            const uint32_t sfx = above + wave_incl_scan(c, lane);  // suffix(top - lane)
            const int i = __builtin_ctzll(__ballot(sfx >= need));
            if (lane == i) {
                out[0] = (uint32_t)(top - i);
                out[1] = sfx - c;
            }
        }
    }
    __syncthreads();
}

// Steps 3 and 4 for the keys of coarse bin b1 (visited by `visit(fn)`, which
// calls fn(key, position) for every such key).  hist: LDS [kMidBins], low: LDS
// [kLowBins]; both are cleared here, together, so that the second digit's
// histogram needs no barrier of its own before it is filled.
template <int NT, class Visit>
__device__ void refine_and_mark(Visit visit, uint32_t b1, uint32_t need1, uint32_t *hist,
                                uint32_t *low, uint32_t *s_res, uint32_t *sure, uint32_t *tie,
                                uint32_t &r_ties) {
    for (int x = threadIdx.x; x < kMidBins; x += NT) hist[x] = 0u;
    for (int x = threadIdx.x; x < kLowBins; x += NT) low[x] = 0u;
    __syncthreads();
    visit([&](uint32_t key, uint32_t) {
        atomicAdd(&hist[(key >> kMidShift) & (kMidBins - 1)], 1u);
    });
    __syncthreads();
    find_threshold_bin<kMidBins>(hist, need1, s_res);
    const uint32_t b2 = s_res[0];
    const uint32_t need2 = need1 - s_res[1];
    const uint32_t pref = (b1 << (kCoarseShift - kMidShift)) | b2;  // key >> kMidShift
    visit([&](uint32_t key, uint32_t) {
        if ((key >> kMidShift) == pref) atomicAdd(&low[key & (kLowBins - 1)], 1u);
    });
    __syncthreads();  // also: every thread has read s_res before it is rewritten
    find_threshold_bin<kLowBins>(low, need2, s_res);
    const uint32_t tau = (pref << kMidShift) | s_res[0];
    r_ties = need2 - s_res[1];  // keys equal to tau that are taken (>= 1)
    visit([&](uint32_t key, uint32_t j) {
        if (key > tau) atomicOr(&sure[j >> 5], 1u << (j & 31));
        else if (key == tau) atomicOr(&tie[j >> 5], 1u << (j & 31));
    });
}

// Step 5: ordered output from the bitmaps (words [0, words), a multiple of 4).
// Per slice of 4 * NT words, each thread owns 4 consecutive words (one 16-byte
// LDS read per bitmap); a workgroup-wide prefix of the sure and tie counts
// gives each thread its first output slot, and of the ties only the first
// r_ties in position order are kept (ties go to the lowest index).  A thread
// then emits its positions in one loop over the set bits of its 128 positions.
template <int NT>
__device__ void compact_bitmaps(const uint32_t *sure, const uint32_t *tie, int words,
                                uint32_t r_ties, int k, int32_t *out, uint32_t *s_wave) {
    uint32_t sure_done = 0, tie_done = 0;  // counts of the slices before
    for (int s0 = 0; s0 < words; s0 += 4 * NT) {  // uniform
        const int w0 = s0 + 4 * (int)threadIdx.x;
        uint4 sv = make_uint4(0u, 0u, 0u, 0u), tv = make_uint4(0u, 0u, 0u, 0u);
        if (w0 < words) {
            sv = *reinterpret_cast<const uint4 *>(sure + w0);
            tv = *reinterpret_cast<const uint4 *>(tie + w0);
        }
        uint64_t a = sv.x | ((uint64_t)sv.y << 32), b = sv.z | ((uint64_t)sv.w << 32);
        uint64_t ta = tv.x | ((uint64_t)tv.y << 32), tb = tv.z | ((uint64_t)tv.w << 32);
        const uint32_t cs = __popcll(a) + __popcll(b), ct = __popcll(ta) + __popcll(tb);
        uint32_t sure_before, tie_before, sure_total, tie_total;
        block_excl_scan2<NT>(cs, ct, s_wave, sure_before, tie_before, sure_total, tie_total);
        sure_before += sure_done;
        tie_before += tie_done;
        sure_done += sure_total;
        tie_done += tie_total;
        uint32_t take = tie_before < r_ties ? r_ties - tie_before : 0u;  // ties kept here
        if (take >= ct) {
            a |= ta;
            b |= tb;
        } else {
            for (; take; --take) {  // the one thread that keeps only part of its ties
                if (ta) {
                    a |= ta & (0ull - ta);
                    ta &= ta - 1;
                } else {
                    b |= tb & (0ull - tb);
                    tb &= tb - 1;
                }
            }
        }
        uint32_t pos = sure_before + min(tie_before, r_ties);
        const int p0 = w0 * 32;
        while (a | b) {
            const bool lo = a != 0;
            const uint64_t m = lo ? a : b;
            const int bit = __builtin_ctzll(m) + (lo ? 0 : 64);
            if (lo) a &= a - 1;
            else b &= b - 1;
            if (pos < (uint32_t)k) out[pos] = p0 + bit;
            ++pos;
        }
    }
}

// One wave's share of the filter pass: 1024 keys starting at `base`, lane-strided
// so that each ballot is exactly two bitmap words.  filter_load_1024 reads them
// (positions clamped to `last`, which must be readable); filter_classify_1024
// marks the keys above bin b1 in the bitmap words and returns, per 64 keys, the
// ballot of those in it; filter_append_1024 hands those candidates, in position
// order, to `append` from slot `slot` on.  Keys past n are neither selected nor
// candidates.
__device__ __forceinline__ void filter_load_1024(const float *srow, int base, int last,
                                                 uint32_t (&key)[16]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int u = 0; u < 16; ++u)
        key[u] = score_key(__builtin_nontemporal_load(srow + min(base + u * 64 + lane, last)));
}

// Returns the wave's candidate count.
__device__ __forceinline__ uint32_t filter_classify_1024(const uint32_t (&key)[16], int base,
                                                         int n, uint32_t b1,
                                                         uint32_t *sure_words,
                                                         uint32_t *tie_words,
                                                         uint64_t (&cmask)[16]) {
    const int lane = threadIdx.x & 63;
    uint32_t ccount = 0;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const bool ok = base + u * 64 + lane < n;
        const uint32_t d = key[u] >> kCoarseShift;
        const uint64_t sm = __ballot(ok && d > b1);
        cmask[u] = __ballot(ok && d == b1);
        ccount += __popcll(cmask[u]);
        if (lane < 2) {
            sure_words[2 * u + lane] = lane ? (uint32_t)(sm >> 32) : (uint32_t)sm;
            if (tie_words) tie_words[2 * u + lane] = 0u;
        }
    }
    return ccount;
}

template <class AppendFn>
__device__ __forceinline__ void filter_append_1024(const uint32_t (&key)[16], int base,
                                                   const uint64_t (&cmask)[16], uint32_t slot,
                                                   AppendFn append) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const uint64_t lower = lane ? (cmask[u] << (64 - lane)) : 0ull;
        if ((cmask[u] >> lane) & 1ull) append(slot + (uint32_t)__popcll(lower), key[u],
                                              (uint32_t)(base + u * 64 + lane));
        slot += (uint32_t)__popcll(cmask[u]);
    }
}

// ------------------------------------------------------------------------------------
// Per-row kernel (many rows).

struct TopkRowArgs {
    const float *scores;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    const uint32_t *hist;  // [rows, 256] or null
    int32_t *idx;
    int32_t *n_sel;
    int n_q, max_len, causal, top_k;
    int words_max;  // bitmap words reserved in LDS per bitmap
    int cand_cap;
};

// Steps 1-5 for one row of scores srow[0 .. n-1] (n > k) by one workgroup of
// kRowThreads, writing k ascending positions to out.  ghist: the row's coarse
// histogram from the indexer, or null (made here from the scores).  lds:
// dynamic LDS of row_kernel_lds() bytes.
__device__ void row_topk(const float *srow, const uint32_t *ghist, int n, int k, int words_max,
                         int cand_cap, int32_t *out, uint32_t *lds, uint32_t *s_wave,
                         uint32_t *s_res, uint32_t *s_cand_count) {
    constexpr int NW = kRowThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    uint32_t *hist = lds;                // kHistWords
    uint32_t *low = hist + kHistWords;   // kLowBins
    uint32_t *sure = low + kLowBins;     // words_max
    uint32_t *tie = sure + words_max;    // words_max
    uint32_t *ckey = tie + words_max;    // cand_cap
    uint32_t *cidx = ckey + cand_cap;    // cand_cap
    const int nchunks = div_up(n, 1024);

    for (int x = tid; x < kCoarseBins; x += kRowThreads) hist[x] = ghist ? ghist[x] : 0u;
    if (tid == 0) *s_cand_count = 0u;
    __syncthreads();
    if (!ghist) {
        for (int c = wave; c < nchunks; c += NW) {
            uint32_t key[16];
#pragma unroll
            for (int u = 0; u < 16; ++u)
                key[u] = score_key(srow[min(c * 1024 + u * 64 + lane, n - 1)]);
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (c * 1024 + u * 64 + lane < n) atomicAdd(&hist[key[u] >> kCoarseShift], 1u);
        }
        __syncthreads();
    }
    find_threshold_bin<kCoarseBins>(hist, (uint32_t)k, s_res);
    const uint32_t b1 = s_res[0];
    const uint32_t need1 = (uint32_t)k - s_res[1];

    const uint32_t cap = (uint32_t)cand_cap;
    for (int c = wave; c < nchunks; c += NW) {
        uint32_t key[16];
        filter_load_1024(srow, c * 1024, n - 1, key);
        uint64_t cmask[16];
        const uint32_t cnt =
            filter_classify_1024(key, c * 1024, n, b1, sure + c * 32, tie + c * 32, cmask);
        uint32_t slot = 0;
        if (lane == 0 && cnt) slot = atomicAdd(s_cand_count, cnt);
        filter_append_1024(key, c * 1024, cmask, __builtin_amdgcn_readfirstlane(slot),
                           [&](uint32_t at, uint32_t kv, uint32_t j) {
                               if (at < cap) {
                                   ckey[at] = kv;
                                   cidx[at] = j;
                               }
                           });
    }
    __syncthreads();
    const uint32_t ncand = *s_cand_count;
    auto visit = [&](auto &&fn) {
        if (ncand <= cap) {
            for (uint32_t i = tid; i < ncand; i += kRowThreads) fn(ckey[i], cidx[i]);
        } else {
            for (int j = tid; j < n; j += kRowThreads) {
                const uint32_t key = score_key(srow[j]);
                if ((key >> kCoarseShift) == b1) fn(key, (uint32_t)j);
            }
        }
    };
    uint32_t r_ties;
    refine_and_mark<kRowThreads>(visit, b1, need1, hist, low, s_res, sure, tie, r_ties);
    __syncthreads();
    compact_bitmaps<kRowThreads>(sure, tie, nchunks * 32, r_ties, k, out, s_wave);
}

template <bool HAVE_HIST>
__global__ __launch_bounds__(kRowThreads) void topk_row_kernel(TopkRowArgs a) {
    constexpr int NW = kRowThreads / 64;
    extern __shared__ __align__(16) uint32_t lds[];
    __shared__ uint32_t s_wave[2 * NW];
    __shared__ uint32_t s_res[2];
    __shared__ uint32_t s_cand_count;

    const int row = blockIdx.x;
    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int k = a.top_k;
    const int tid = threadIdx.x;
    int32_t *out = a.idx + (size_t)row * k;
    if (n <= k) {  // every valid key is selected
        for (int i = tid; i < k; i += kRowThreads) out[i] = i < n ? i : -1;
        if (tid == 0) a.n_sel[row] = n;
        return;
    }
    row_topk(a.scores + (size_t)row * a.max_len,
             HAVE_HIST ? a.hist + (size_t)row * kCoarseBins : nullptr, n, k, a.words_max,
             a.cand_cap, out, lds, s_wave, s_res, &s_cand_count);
    if (tid == 0) a.n_sel[row] = k;
}

// ------------------------------------------------------------------------------------
// Short rows (up to kTopkRowMaxLen keys): one workgroup per row holds the whole
// row in registers, kShortKeys consecutive positions per thread, read once.
// tau is fixed four bits at a time from the top (up to 8 rounds): every thread
// counts the digits of its keys that still match the digits fixed so far in 16
// nibble counters (a 64-bit word per 8 keys); the counters are widened to 16
// bits, summed over the wave by a transpose-reduction and over the waves
// through LDS (one barrier per round, the buffer alternating between rounds),
// and every wave takes the same digit from the totals.  Each round is a chain
// of dependent latencies (about half a microsecond), so once at most
// kShortFinish keys still match, they are packed into one wave, which ranks
// them against each other directly and so fixes tau in one step.  There are no
// LDS atomics (the scores crowd into a few bins of the leading digits, where
// same-address atomics serialise) and no second pass over memory.  The
// ordered output is one workgroup prefix of each thread's counts of keys above
// tau and equal to tau; of the latter the first r in position order are kept.
constexpr int kShortKeys = 16;
static_assert(1024 * kShortKeys >= kTopkRowMaxLen, "one 1024-thread workgroup holds a short row");

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xf, 0xf, false);
}

// AND and OR over the 64 lanes of a wave (every lane active): a butterfly
// inside each 16-lane row with DPP (lane ^ 1, lane ^ 2, half-row and row
// mirrors), then across rows with the permlane16 / permlane32 swaps; VALU
// steps only, no LDS permutes.
__device__ __forceinline__ void wave_and_or(uint32_t &a, uint32_t &o) {
    a &= dpp_u32<0xB1>(a);  o |= dpp_u32<0xB1>(o);
    a &= dpp_u32<0x4E>(a);  o |= dpp_u32<0x4E>(o);
    a &= dpp_u32<0x141>(a); o |= dpp_u32<0x141>(o);
    a &= dpp_u32<0x140>(a); o |= dpp_u32<0x140>(o);
    auto ra = __builtin_amdgcn_permlane16_swap(a, a, false, false);
    auto ro = __builtin_amdgcn_permlane16_swap(o, o, false, false);
    a = ra[0] & ra[1];
    o = ro[0] | ro[1];
    ra = __builtin_amdgcn_permlane32_swap(a, a, false, false);
    ro = __builtin_amdgcn_permlane32_swap(o, o, false, false);
    a = ra[0] & ra[1];
    o = ro[0] | ro[1];
}

// Each of 8 values summed over the 64 lanes; lane L ends with the total of
// value L >> 3.  Halving exchanges across the row pairs (permlane32 / 16
// swaps) and inside rows (row mirror), then plain sums with the half mirror
// and the quad permutes (lanes reached: every lane of the wave exactly once).
__device__ __forceinline__ uint32_t wave_reduce8(const uint32_t (&w)[8], int lane) {
    uint32_t p[4], q[2];
#pragma unroll
    for (int v = 0; v < 4; ++v) {  // lanes 0-31 keep values 0-3, lanes 32-63 values 4-7
        const auto r = __builtin_amdgcn_permlane32_swap(w[v], w[v + 4], false, false);
        p[v] = r[0] + r[1];
    }
#pragma unroll
    for (int v = 0; v < 2; ++v) {  // then by lane bit 4
        const auto r = __builtin_amdgcn_permlane16_swap(p[v], p[v + 2], false, false);
        q[v] = r[0] + r[1];
    }
    const bool up = (lane & 8) != 0;  // then by lane bit 3, with the row-mirror partner
    uint32_t x = (up ? q[1] : q[0]) + dpp_u32<0x140>(up ? q[0] : q[1]);
    x += dpp_u32<0x141>(x);
    x += dpp_u32<0x4E>(x);
    return x + dpp_u32<0xB1>(x);
}

// The 16 digit counts of the keys of this wave selected by `sel` (keys past
// `cnt` are not counted), 16-bit halves two to a word, summed over the wave;
// lanes with (lane & 7) == 0 write word lane >> 3 to out.
template <int CNT>
__device__ __forceinline__ void wave_digit_counts(const uint32_t (&key)[CNT], uint32_t sel,
                                                  int shift, uint32_t prefix, uint32_t pmask,
                                                  int lane, uint32_t *out) {
    uint64_t acc[2] = {0ull, 0ull};  // nibble d of acc[h]: keys 8h .. 8h+7 with digit d
#pragma unroll
    for (int j = 0; j < CNT; ++j) {
        const uint32_t d = (key[j] >> shift) & 15u;
        const uint32_t m = ((key[j] ^ prefix) & pmask) == 0u ? (sel >> j) & 1u : 0u;
        acc[j >> 3] += (uint64_t)m << (4 * d);
    }
    // bytes of ev: digits 0, 2, .., 14; of od: 1, 3, .., 15 (each at most 16)
    constexpr uint64_t kLowNibbles = 0x0F0F0F0F0F0F0F0Full;
    const uint64_t ev = (acc[0] & kLowNibbles) + (acc[1] & kLowNibbles);
    const uint64_t od = ((acc[0] >> 4) & kLowNibbles) + ((acc[1] >> 4) & kLowNibbles);
    // 16-bit halves, two digits per word (the lookup is in topk_short_kernel)
    const uint32_t w[8] = {(uint32_t)ev & 0x00FF00FFu,          (uint32_t)(ev >> 8) & 0x00FF00FFu,
                           (uint32_t)(ev >> 32) & 0x00FF00FFu,  (uint32_t)(ev >> 40) & 0x00FF00FFu,
                           (uint32_t)od & 0x00FF00FFu,          (uint32_t)(od >> 8) & 0x00FF00FFu,
                           (uint32_t)(od >> 32) & 0x00FF00FFu,  (uint32_t)(od >> 40) & 0x00FF00FFu};
    const uint32_t t = wave_reduce8(w, lane);  // at most 64 * 16 per half
    if ((lane & 7) == 0) out[lane >> 3] = t;
}

// Inclusive prefix sum over the 16 lanes of each row (DPP row shifts).
__device__ __forceinline__ uint32_t row16_incl_scan(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
    return v + (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);
}

constexpr int kShortFinish = 64;  // candidates left when one wave ranks them directly

// LDS of short_select<NT>.
template <int NT>
struct ShortSelectLds {
    uint32_t cnt[2][NT / 64][8];  // per round: each wave's 16 digit counts, two per word
    uint32_t wave[2 * (NT / 64)];
    uint32_t pack[kShortFinish];
    uint32_t tau[2];
};

// tau, the k-th largest of the keys key[j] (j with bit j of vmask set) held by
// the NT threads of the workgroup (k at most their number), and r, the number
// of keys equal to tau among the k largest.  Every thread calls it; every
// thread gets the same tau and r.  first_round > 0: every valid key shares the
// digits of prefix0 above bit 32 - 4 first_round (the caller found them), and
// those rounds are skipped.
template <int NT>
__device__ void short_select(const uint32_t (&key)[kShortKeys], uint32_t vmask, uint32_t k,
                             ShortSelectLds<NT> &sm, uint32_t &tau, uint32_t &r,
                             int first_round = 0, uint32_t prefix0 = 0u) {
    constexpr int NW = NT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Lane l < 16 follows digit d = 15 - l (an inclusive prefix over lanes is
    // then a suffix over digits); digit d is half (d >> 2) & 1 of word
    // 4 (d & 1) + 2 (d >> 3) + ((d >> 1) & 1) of the counts.
    const int dg = 15 - (lane & 15);
    const int dword = 4 * (dg & 1) + 2 * (dg >> 3) + ((dg >> 1) & 1);
    const int dhalf = 16 * ((dg >> 2) & 1);

    // prefix: the digits of tau fixed so far; need: keys matching it still to be taken
    uint32_t pmask = first_round ? ~0u << (32 - 4 * first_round) : 0u;
    uint32_t prefix = prefix0 & pmask, need = k;
    tau = prefix;
    r = need;
#pragma unroll 1
    for (int round = first_round; round < 8; ++round) {
        const int shift = 28 - 4 * round;
        uint32_t(*buf)[8] = sm.cnt[round & 1];
        wave_digit_counts<kShortKeys>(key, vmask, shift, prefix, pmask, lane, buf[wave]);
        __syncthreads();
        uint32_t c = 0u;  // lanes 0..15: keys of digit dg summed over the waves
        if (lane < 16) {
#pragma unroll
            for (int x = 0; x < NW; ++x) c += (buf[x][dword] >> dhalf) & 0xFFFFu;
        }
        const uint32_t incl = row16_incl_scan(c);  // lanes 0..15: keys with digit >= dg
        const uint64_t reach = __ballot(lane < 16 && incl >= need);
        const int ls = reach ? __builtin_ctzll(reach) : 15;  // consistent counts always reach
        const uint32_t above = (uint32_t)__builtin_amdgcn_readlane((int)(incl - c), ls);
        const uint32_t left = (uint32_t)__builtin_amdgcn_readlane((int)c, ls);  // keys still matching
        need -= above;
        prefix |= (15u - (uint32_t)ls) << shift;
        pmask |= 15u << shift;
        if (round == 7) {
            tau = prefix;
            r = need;
        } else if (left <= (uint32_t)kShortFinish) {
            // Few keys still match: pack them (in thread order) into one wave,
            // which ranks them directly.  tau is the need-th largest of them.
            uint32_t mb = 0u;
#pragma unroll
            for (int j = 0; j < kShortKeys; ++j)
                mb |= (((key[j] ^ prefix) & pmask) == 0u ? 1u : 0u) << j;
            mb &= vmask;
            uint32_t before, unused0, total, unused1;
            block_excl_scan2<NT>((uint32_t)__popc(mb), 0u, sm.wave, before, unused0, total, unused1);
#pragma unroll
            for (int j = 0; j < kShortKeys; ++j)
                if ((mb >> j) & 1u) sm.pack[before++] = key[j];
            __syncthreads();
            if (wave == 0) {
                const uint32_t cv = lane < (int)left ? sm.pack[lane] : 0u;
                uint32_t gt = 0u, eq = 0u;
                for (uint32_t i = 0; i < left; ++i) {
                    const uint32_t ci = (uint32_t)__builtin_amdgcn_readlane((int)cv, (int)i);
                    gt += ci > cv ? 1u : 0u;
                    eq += ci == cv ? 1u : 0u;
                }
                const uint64_t hit = __ballot(lane < (int)left && gt < need && need <= gt + eq);
                if (lane == (hit ? __builtin_ctzll(hit) : 0)) {
                    sm.tau[0] = cv;
                    sm.tau[1] = need - gt;
                }
            }
            __syncthreads();
            tau = sm.tau[0];
            r = sm.tau[1];
            break;
        }
    }
}

template <int NT>  // NT * kShortKeys >= max_len
__global__ __launch_bounds__(NT) void topk_short_kernel(TopkRowArgs a) {
    __shared__ ShortSelectLds<NT> sm;

    const int row = blockIdx.x;
    const int tid = threadIdx.x;
    const float *srow = a.scores + (size_t)row * a.max_len;
    const int p0 = tid * kShortKeys;
    // loads issued before the row's length is known (clamped to its capacity)
    uint32_t key[kShortKeys];
#pragma unroll
    for (int j = 0; j < kShortKeys; ++j) key[j] = score_key(srow[min(p0 + j, a.max_len - 1)]);
    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int k = a.top_k;
    int32_t *out = a.idx + (size_t)row * k;
    if (n <= k) {  // every valid key is selected
        for (int i = tid; i < k; i += NT) out[i] = i < n ? i : -1;
        if (tid == 0) a.n_sel[row] = n;
        return;
    }
    const int nv = min(max(n - p0, 0), kShortKeys);  // this thread's valid keys: key[0 .. nv)
    const uint32_t vmask = (1u << nv) - 1u;              // as a bit mask (nv <= 16)
    uint32_t tau, r;
    short_select<NT>(key, vmask, (uint32_t)k, sm, tau, r);

    // this thread's keys above tau and equal to tau, as bit masks over j
    uint32_t sbits = 0u, tbits = 0u;
#pragma unroll
    for (int j = 0; j < kShortKeys; ++j) {
        sbits |= (key[j] > tau ? 1u : 0u) << j;
        tbits |= (key[j] == tau ? 1u : 0u) << j;
    }
    sbits &= vmask;
    tbits &= vmask;
    uint32_t sure_before, tie_before, sure_total, tie_total;
    block_excl_scan2<NT>((uint32_t)__popc(sbits), (uint32_t)__popc(tbits), sm.wave, sure_before,
                         tie_before, sure_total, tie_total);
    uint32_t take = tie_before < r ? r - tie_before : 0u;  // ties this thread may still keep
    uint32_t keep = sbits;
    for (; take && tbits; --take) {  // the first `take` ties in position order
        keep |= tbits & (0u - tbits);
        tbits &= tbits - 1u;
    }
    uint32_t pos = sure_before + min(tie_before, r);
    while (keep) {
        const int j = __builtin_ctz(keep);
        keep &= keep - 1u;
        if (pos < (uint32_t)k) out[pos] = p0 + j;
        ++pos;
    }
    if (tid == 0) a.n_sel[row] = k;
}

// ------------------------------------------------------------------------------------
// Chunked prefill without the score block (many causal rows, k <= 2048).
//
//   pass 1: the indexer scores every kTopkSampleStride-th key of every row;
//           topk_sample_thresh_kernel takes, per row, the order-preserving key
//           tau' of the R-th largest sampled score (topk_sample_rank);
//   pass 2: the indexer recomputes every score with the same arithmetic and
//           writes the keys at or above tau' (key, position) to the row's
//           slots of each 256-key block (kTopkBlockSlots kept, all counted);
//   finish: topk_cand_kernel selects exactly from the candidates.
// If a row has at least k candidates, every key at or above its k-th largest
// score is among them (that score is >= tau'), so the selection, ties
// included, is the one the full row would give.  A row with fewer than k
// candidates, or more than the list holds (very flat rows), is finished by its
// workgroup the slow way: it recomputes the row's scores on the vector units
// and runs the per-row selection on them.

struct SampleArgs {
    const float *samples;    // [rows, cols] sampled scores
    const int32_t *seq_lens;
    const int32_t *q_pos;
    uint32_t *thresh;        // [rows]
    uint32_t *slow;          // [1 + rows]: its count is cleared here for the selection pass
    int n_q, max_len, causal, top_k, cols, rank;
};

// One workgroup per row: the rank-th largest of the row's valid sampled keys,
// found by short_select over 16 keys per thread in registers (NT = 256 for up
// to 4096 samples, 512 for up to 8192; which thread holds which key does not
// matter, so the loads are strided and coalesced).  Rows with no more than k
// valid keys select them all and get the largest threshold (no candidates);
// rows with no more than `rank` valid samples get 0 (every key a candidate).
static_assert(kMaxLen / kTopkSampleStride <= 512 * kShortKeys, "samples of a row fit 512 threads");

template <int NT>
__global__ __launch_bounds__(NT) void topk_sample_thresh_kernel(SampleArgs a) {
    __shared__ ShortSelectLds<NT> sm;
    const int row = blockIdx.x, b = row / a.n_q, tid = threadIdx.x;
    if (row == 0 && tid == 0) a.slow[0] = 0u;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int m = div_up(n, kTopkSampleStride);  // valid samples, at most a.cols <= NT * kShortKeys
    if (n <= a.top_k || m <= a.rank) {
        if (tid == 0) a.thresh[row] = n <= a.top_k ? 0xffffffffu : 0u;
        return;
    }
    const float *srow = a.samples + (size_t)row * a.cols;
    uint32_t key[kShortKeys], vmask = 0u;
#pragma unroll
    for (int j = 0; j < kShortKeys; ++j) {
        const int i = j * NT + tid;
        key[j] = score_key(srow[min(i, m - 1)]);
        vmask |= (i < m ? 1u : 0u) << j;
    }
    uint32_t tau, r;
    short_select<NT>(key, vmask, (uint32_t)a.rank, sm, tau, r);
    if (tid == 0) a.thresh[row] = tau;
}

struct CandArgs {
    const uint32_t *cand_count;  // [rows, kblocks]
    const uint2 *cands;          // [rows, kblocks, kTopkBlockSlots]
    const int32_t *seq_lens;
    const int32_t *q_pos;
    int32_t *idx;
    int32_t *n_sel;
    float *scores;               // [rows, max_len]: rows finished the slow way
    const uint16_t *q_idx;
    const uint16_t *k_idx;
    const int32_t *page_table;
    uint32_t *slow;              // [1 + rows]: count, then the rows left for the slow way
    int n_q, max_len, causal, top_k, words_max, cand_cap, page_shift, max_pages, kblocks;
};

// Selection from the candidates, one 512-thread workgroup per row: the row's
// kept candidates are copied to LDS in key-block order (thread t copies those
// of its BPT consecutive blocks, at its offset from a workgroup prefix of the
// block counts), each thread takes 16 consecutive ones into registers and
// short_select fixes tau and the number r of ties to keep; then each thread
// turns its own blocks' candidates into bitmap words of the keys above tau and
// of those equal to tau over the blocks' positions (8 words per 256-key block),
// so that one more workgroup prefix orders the output by position (the slots
// of a block are not in position order).  A row whose candidates do not decide
// its set (a block with more than the slots, fewer than k, more than kCandCap)
// is appended to the slow list for topk_cand_slow_kernel.
constexpr int kCandThreads = 512;
constexpr int kCandCap = kCandThreads * kShortKeys;  // candidates held in registers
static_assert(kMaxLen / kTopkKeyBlock <= 2 * kCandThreads, "at most two key blocks per thread");
static_assert(kTopkKeyBlock == 8 * 32, "a block's positions are 8 bitmap words");

template <int BPT>  // key blocks per thread
// one key block per thread: at most 80 registers, so that three workgroups
// (six waves per SIMD) fit a CU beside their LDS
__global__ __launch_bounds__(kCandThreads) __attribute__((amdgpu_waves_per_eu(BPT == 1 ? 6 : 1)))
void topk_cand_fast_kernel(CandArgs a) {
    constexpr int NT = kCandThreads;
    constexpr int NW = NT / 64;
    constexpr int NWD = 8 * BPT;  // bitmap words per thread
    constexpr int kFirst = 16;    // entries of a block loaded in the first batch (one 128-byte line; about 8 expected)
    // [kCandCap] keys, then [kCandCap] 16-bit positions relative to the first
    // key of the owning thread's blocks (48 KiB: three workgroups per CU)
    extern __shared__ __align__(16) uint32_t lds[];
    __shared__ ShortSelectLds<NT> sm;
    __shared__ uint32_t s_andor[2][NW];
    uint32_t *s_key = lds;
    uint16_t *s_pos = reinterpret_cast<uint16_t *>(lds + kCandCap);
    static_assert(BPT * kTopkKeyBlock <= 65536, "relative positions fit 16 bits");

    const int row = blockIdx.x, b = row / a.n_q, tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int k = a.top_k;
    int32_t *out = a.idx + (size_t)row * k;
    if (n <= k) {  // every valid key is selected
        for (int i = tid; i < k; i += NT) out[i] = i < n ? i : -1;
        if (tid == 0) a.n_sel[row] = n;
        return;
    }
    const int nblk = div_up(n, kTopkKeyBlock);
    // block counts and the first kFirst entries of each of this thread's
    // blocks in one batch (the slots exist whatever the count: entries past it
    // are read and never used), before the workgroup prefix that places them
    uint32_t cbr[BPT];
    uint2 e[BPT][kFirst];
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
        const int kb = min(BPT * tid + u, a.kblocks - 1);
        cbr[u] = a.cand_count[(size_t)row * a.kblocks + kb];
        const uint2 *src = a.cands + ((size_t)row * a.kblocks + kb) * kTopkBlockSlots;
#pragma unroll
        for (int v = 0; v < kFirst; ++v) e[u][v] = src[v];
    }
    uint32_t kept[BPT], mine = 0u, lost_mine = 0u;
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
        const uint32_t cb = BPT * tid + u < nblk ? cbr[u] : 0u;
        kept[u] = min(cb, (uint32_t)kTopkBlockSlots);
        mine += kept[u];
        lost_mine += cb - kept[u];
    }
    uint32_t before, unused0, cnt, lost;
    block_excl_scan2<NT>(mine, lost_mine, sm.wave, before, unused0, cnt, lost);
    if (lost != 0 || cnt < (uint32_t)k || cnt > (uint32_t)kCandCap) {  // uniform
        if (tid == 0) a.slow[1 + atomicAdd(&a.slow[0], 1u)] = (uint32_t)row;
        return;
    }
    const uint32_t p_first = (uint32_t)tid * BPT * kTopkKeyBlock;  // first key of this thread's blocks
    {
        uint32_t at = before;
#pragma unroll
        for (int u = 0; u < BPT; ++u) {
#pragma unroll
            for (int v = 0; v < kFirst; ++v)
                if ((uint32_t)v < kept[u]) {
                    s_key[at + v] = e[u][v].x;
                    s_pos[at + v] = (uint16_t)(e[u][v].y - p_first);
                }
            const uint2 *src = a.cands + ((size_t)row * a.kblocks + BPT * tid + u) * kTopkBlockSlots;
            for (uint32_t q0 = kFirst; q0 < kept[u]; q0 += 8) {  // rare: more than kFirst candidates
                uint2 x[8];
#pragma unroll
                for (int v = 0; v < 8; ++v)
                    if (q0 + v < kept[u]) x[v] = src[q0 + v];
#pragma unroll
                for (int v = 0; v < 8; ++v)
                    if (q0 + v < kept[u]) {
                        s_key[at + q0 + v] = x[v].x;
                        s_pos[at + q0 + v] = (uint16_t)(x[v].y - p_first);
                    }
            }
            at += kept[u];
        }
    }
    __syncthreads();
    uint32_t key[kShortKeys];
#pragma unroll
    for (int j = 0; j < kShortKeys; ++j) key[j] = s_key[tid * kShortKeys + j];
    const int nv = min(max((int)cnt - tid * kShortKeys, 0), kShortKeys);
    const uint32_t vmask = (1u << nv) - 1u;
    // The candidates crowd above the row's threshold, so their keys share their
    // leading digits: AND and OR of every valid key fix those digits at once.
    uint32_t kand = ~0u, kor = 0u;
#pragma unroll
    for (int j = 0; j < kShortKeys; ++j)
        if ((vmask >> j) & 1u) {
            kand &= key[j];
            kor |= key[j];
        }
    wave_and_or(kand, kor);
    if (lane == 0) {
        s_andor[0][wave] = kand;
        s_andor[1][wave] = kor;
    }
    __syncthreads();
    kand = ~0u;
    kor = 0u;
#pragma unroll
    for (int x = 0; x < NW; ++x) {
        kand &= s_andor[0][x];
        kor |= s_andor[1][x];
    }
    const uint32_t differ = kand ^ kor;  // bits in which some valid keys differ
    const int first_round = differ ? __builtin_clz(differ) / 4 : 8;
    uint32_t tau, r;
    if (first_round == 8) {  // every candidate equal: the first k of them
        tau = kand;
        r = (uint32_t)k;
    } else {
        short_select<NT>(key, vmask, (uint32_t)k, sm, tau, r, first_round, kand);
    }

    // this thread's blocks (positions 256 BPT tid ..): keys above / equal to tau
    uint32_t sw[NWD], tw[NWD];
#pragma unroll
    for (int i = 0; i < NWD; ++i) sw[i] = tw[i] = 0u;
    for (uint32_t q = 0; q < mine; ++q) {
        const uint32_t kk = s_key[before + q];
        const uint32_t p = s_pos[before + q];  // 0 .. 256 BPT - 1
        const uint32_t bit = 1u << (p & 31u), wi = p >> 5;
        const uint32_t sb = kk > tau ? bit : 0u, tb = kk == tau ? bit : 0u;
#pragma unroll
        for (int i = 0; i < NWD; ++i) {
            sw[i] |= wi == (uint32_t)i ? sb : 0u;
            tw[i] |= wi == (uint32_t)i ? tb : 0u;
        }
    }
    uint32_t cs = 0u, ct = 0u;
#pragma unroll
    for (int i = 0; i < NWD; ++i) {
        cs += (uint32_t)__popc(sw[i]);
        ct += (uint32_t)__popc(tw[i]);
    }
    uint32_t sure_before, tie_before, sure_total, tie_total;
    block_excl_scan2<NT>(cs, ct, sm.wave, sure_before, tie_before, sure_total, tie_total);
    uint32_t take = tie_before < r ? r - tie_before : 0u;  // ties this thread may still keep
#pragma unroll
    for (int i = 0; i < NWD; ++i) {
        for (; take && tw[i]; --take) {  // the first `take` ties in position order
            sw[i] |= tw[i] & (0u - tw[i]);
            tw[i] &= tw[i] - 1u;
        }
    }
    uint32_t pos = sure_before + min(tie_before, r);
#pragma unroll
    for (int i = 0; i < NWD; ++i) {
        uint32_t m = sw[i];
        while (m) {
            const int j = __builtin_ctz(m);
            m &= m - 1u;
            if (pos < (uint32_t)k) out[pos] = (int32_t)(p_first + 32 * i + j);
            ++pos;
        }
    }
    if (tid == 0) a.n_sel[row] = k;
}

// Rows whose candidates do not decide the set (the slow list), the slow way:
// the row's scores recomputed on the vector units into the score buffer, then
// the per-row selection over them.  Each workgroup takes list entries
// blockIdx.x, blockIdx.x + gridDim.x, ...
__global__ __launch_bounds__(kRowThreads) void topk_cand_slow_kernel(CandArgs a) {
    constexpr int NW = kRowThreads / 64;
    extern __shared__ __align__(16) uint32_t lds[];
    __shared__ uint32_t s_wave[2 * NW];
    __shared__ uint32_t s_res[2];
    __shared__ uint32_t s_cand_count;
    __shared__ __align__(16) uint32_t s_q[128];  // the row's index query
    const int tid = threadIdx.x;
    const uint32_t count = a.slow[0];
    for (uint32_t li = blockIdx.x; li < count; li += gridDim.x) {
        const int row = (int)a.slow[1 + li], b = row / a.n_q;
        const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
        const int k = a.top_k;
        int32_t *out = a.idx + (size_t)row * k;
        if (tid < 128) s_q[tid] = reinterpret_cast<const uint32_t *>(a.q_idx + (size_t)row * 256)[tid];
        __syncthreads();
        float *srow = a.scores + (size_t)row * a.max_len;
        for (int j = tid; j < n; j += kRowThreads) {
            const uint16_t *kr = a.k_idx + token_offset(a.page_table, a.page_shift, a.max_pages,
                                                        a.max_len, b, j, 256);
            float acc = 0.0f;
#pragma unroll 8
            for (int p = 0; p < 32; ++p) {
                const uint4 kv = *reinterpret_cast<const uint4 *>(kr + 8 * p);
                const uint4 qv = *reinterpret_cast<const uint4 *>(&s_q[4 * p]);
                acc = dot8_bf16(kv, qv, acc);
            }
            srow[j] = acc;
        }
        __syncthreads();
        row_topk(srow, nullptr, n, k, a.words_max, a.cand_cap, out, lds, s_wave, s_res,
                 &s_cand_count);
        if (tid == 0) a.n_sel[row] = k;
        __syncthreads();  // LDS reused by the next row
    }
}

// ------------------------------------------------------------------------------------
// Wide kernel (few long rows).

struct TopkWideArgs {
    const float *scores;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    const uint32_t *hist;   // [rows, kCoarseBins], complete
    uint32_t *sure;         // [rows, words_max]: keys above the coarse bin
    uint32_t *cands;        // [rows, regions, 1024]: candidate entries per region
    uint32_t *counts;       // [rows, regions]: their number
    int32_t *idx;
    int32_t *n_sel;
    int n_q, max_len, causal, top_k, chunks_per_row, words_max, regions;
};

// Candidate entries of the wide path.  Region r of a row holds the candidates
// among keys [1024 r, 1024 r + 1024) (one wave's share of the filter), in
// position order; an entry packs the key bits below the coarse digit (the
// coarse digit is b1 for every candidate) and the position inside the region.
constexpr uint32_t kCandLowMask = (1u << kCoarseShift) - 1u;
static_assert(kCoarseShift + 10 <= 32, "an entry holds the low key bits and 10 position bits");
__device__ __forceinline__ uint32_t cand_entry(uint32_t key, uint32_t j) {
    return ((key & kCandLowMask) << 10) | (j & 1023u);
}

// Step 2 for 4096 keys of one row.  The loads that do not depend on the row's
// length (its coarse histogram, 8 bins per thread, and the chunk's scores,
// clamped to the row's capacity) are issued before that length is known, so
// the workgroup waits for memory once before its threshold search.  Each wave
// writes its candidates to its own region and their number beside it: no
// atomics (one shared counter per row, taken by every wave or workgroup of the
// row, serialised at the memory side and cost up to 5 us at 128K keys).
__global__ __launch_bounds__(kWideThreads) void topk_filter_kernel(TopkWideArgs a) {
    constexpr int NW = kWideThreads / 64;
    constexpr int HPT = kCoarseBins / kWideThreads;
    static_assert(kWideChunk == NW * 1024, "one region per wave");
    __shared__ __align__(16) uint32_t hist[kCoarseBins];
    __shared__ uint32_t s_res[2];

    const int row = blockIdx.x / a.chunks_per_row;
    const int c = blockIdx.x - row * a.chunks_per_row;
    const int tid = threadIdx.x, wave = tid >> 6;
    const uint32_t *ghist = a.hist + (size_t)row * kCoarseBins;
    uint32_t hv[HPT];
#pragma unroll
    for (int u = 0; u < HPT; ++u) hv[u] = ghist[u * kWideThreads + tid];
    const float *srow = a.scores + (size_t)row * a.max_len;
    const int base = c * kWideChunk + wave * 1024;
    uint32_t key[16];
    filter_load_1024(srow, base, a.max_len - 1, key);

    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    if (n <= a.top_k || c * kWideChunk >= n) return;  // uniform
#pragma unroll
    for (int u = 0; u < HPT; ++u) hist[u * kWideThreads + tid] = hv[u];
    __syncthreads();
    find_threshold_bin<kCoarseBins>(hist, (uint32_t)a.top_k, s_res);
    const uint32_t b1 = s_res[0];
    uint64_t cmask[16];
    const uint32_t cnt = filter_classify_1024(
        key, base, n, b1, a.sure + (size_t)row * a.words_max + base / 32, nullptr, cmask);
    const size_t region = (size_t)row * a.regions + (size_t)(base >> 10);
    if ((tid & 63) == 0) a.counts[region] = cnt;
    uint32_t *rc = a.cands + region * 1024;
    filter_append_1024(key, base, cmask, 0u,
                       [&](uint32_t at, uint32_t kv, uint32_t j) { rc[at] = cand_entry(kv, j); });
}

constexpr int kFinishRegCands = 8;   // region entries per thread loaded in the first batch
constexpr int kFinishRegWords = 8;   // bitmap words per thread loaded in the first batch
static_assert(kFinishRegWords * kRowThreads * 32 >= kMaxLen, "one batch holds the whole bitmap");
static_assert(kRowThreads / (kMaxLen / 1024) >= 1, "every region has a thread");

// Steps 3-5 for one row.  The first batch of loads needs nothing but the row
// number: the coarse histogram (two bins per thread), the "sure" bitmap
// (kFinishRegWords words per thread: the whole bitmap of the longest supported
// row) and the candidate regions -- T = kRowThreads / regions threads per
// region, each loading its region's count and entries q, q + T, ... of the
// first kFinishRegCands.  The refinement visits the candidates in registers;
// only a region with more than T * kFinishRegCands candidates has the rest
// read from memory.  The bitmaps live in LDS (dynamic, 2 x words_max); the
// tie bitmap starts empty.
__global__ __launch_bounds__(kRowThreads) void topk_finish_kernel(TopkWideArgs a) {
    constexpr int NW = kRowThreads / 64;
    constexpr int HPT = kCoarseBins / kRowThreads;
    extern __shared__ __align__(16) uint32_t lds[];
    __shared__ __align__(16) uint32_t hist[kHistWords];
    __shared__ __align__(16) uint32_t low[kLowBins];
    __shared__ uint32_t s_wave[2 * NW];
    __shared__ uint32_t s_res[2];

    const int row = blockIdx.x;
    const int k = a.top_k;
    const int tid = threadIdx.x;
    const int nr = a.regions;
    const int tpr = kRowThreads / nr;  // threads per region
    const int r = min(tid / tpr, nr - 1), q = tid - (tid / tpr) * tpr;
    const bool owner = tid / tpr < nr;
    const uint32_t *ghist = a.hist + (size_t)row * kCoarseBins;
    const uint32_t *gs = a.sure + (size_t)row * a.words_max;
    const uint32_t *rc = a.cands + ((size_t)row * nr + r) * 1024;
    uint32_t hv[HPT], sv[kFinishRegWords], ent[kFinishRegCands];
#pragma unroll
    for (int u = 0; u < HPT; ++u) hv[u] = ghist[u * kRowThreads + tid];
    const uint32_t rcount = a.counts[(size_t)row * nr + r];
#pragma unroll
    for (int u = 0; u < kFinishRegWords; ++u)
        sv[u] = gs[min(u * kRowThreads + tid, a.words_max - 1)];
#pragma unroll
    for (int u = 0; u < kFinishRegCands; ++u) ent[u] = rc[min(q + u * tpr, 1023)];

    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    int32_t *out = a.idx + (size_t)row * k;
    if (n <= k) {  // every valid key is selected
        for (int i = tid; i < k; i += kRowThreads) out[i] = i < n ? i : -1;
        if (tid == 0) a.n_sel[row] = n;
        return;
    }
    const int words = div_up(n, kWideChunk) * (kWideChunk / 32);
    // regions the filter wrote (every wave of every chunk that holds keys)
    const uint32_t cnt = owner && r < words / 32 ? min(rcount, 1024u) : 0u;
    uint32_t *sure = lds;
    uint32_t *tie = lds + a.words_max;
#pragma unroll
    for (int u = 0; u < kFinishRegWords; ++u) {
        const int w = u * kRowThreads + tid;
        if (w < words) {
            sure[w] = sv[u];
            tie[w] = 0u;
        }
    }
#pragma unroll
    for (int u = 0; u < HPT; ++u) hist[u * kRowThreads + tid] = hv[u];
    __syncthreads();
    find_threshold_bin<kCoarseBins>(hist, (uint32_t)k, s_res);
    const uint32_t b1 = s_res[0];
    const uint32_t need1 = (uint32_t)k - s_res[1];
    const uint32_t key_hi = b1 << kCoarseShift;
    const uint32_t pos0 = (uint32_t)r * 1024u;
    auto visit = [&](auto &&fn) {
#pragma unroll
        for (int u = 0; u < kFinishRegCands; ++u)
            if ((uint32_t)(q + u * tpr) < cnt) fn(key_hi | (ent[u] >> 10), pos0 + (ent[u] & 1023u));
        for (uint32_t i = q + kFinishRegCands * tpr; i < cnt; i += tpr) {
            const uint32_t e = rc[i];
            fn(key_hi | (e >> 10), pos0 + (e & 1023u));
        }
    };
    uint32_t r_ties;
    refine_and_mark<kRowThreads>(visit, b1, need1, hist, low, s_res, sure, tie, r_ties);
    __syncthreads();
    compact_bitmaps<kRowThreads>(sure, tie, words, r_ties, k, out, s_wave);
    if (tid == 0) a.n_sel[row] = k;
}

// Coarse histogram of the top 11 key bits for the wide kernels when the scores
// did not come from the indexer.  hist must be zero on entry.
__global__ __launch_bounds__(kWideThreads) void coarse_hist_kernel(const float *scores,
                                                                   const int32_t *seq_lens,
                                                                   const int32_t *q_pos,
                                                                   uint32_t *hist, int n_q,
                                                                   int max_len, int causal,
                                                                   int chunks_per_row) {
    __shared__ uint32_t h[kCoarseBins];
    const int row = blockIdx.x / chunks_per_row;
    const int c = blockIdx.x - row * chunks_per_row;
    const int b = row / n_q;
    const int n = valid_keys(seq_lens, q_pos, causal, b, row, max_len);
    if (c * kWideChunk >= n) return;
    const int tid = threadIdx.x;
    for (int x = tid; x < kCoarseBins; x += kWideThreads) h[x] = 0u;
    __syncthreads();
    const float *srow = scores + (size_t)row * max_len;
    const int base = c * kWideChunk + tid;
    uint32_t key[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) key[u] = score_key(srow[min(base + u * kWideThreads, n - 1)]);
#pragma unroll
    for (int u = 0; u < 16; ++u)
        if (base + u * kWideThreads < n) atomicAdd(&h[key[u] >> kCoarseShift], 1u);
    __syncthreads();
    for (int x = tid; x < kCoarseBins; x += kWideThreads)
        if (h[x]) atomicAdd(&hist[(size_t)row * kCoarseBins + x], h[x]);
}

__global__ __launch_bounds__(256) void zero_u32_kernel(uint32_t *p, size_t n) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = 0u;
}

hipError_t launch_zero_u32(uint32_t *p, size_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    zero_u32_kernel<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream>>>(p, n);
    return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Host side.

static int row_words(int max_len) { return div_up(max_len, 1024) * 32; }
static int wide_words(int max_len) { return div_up(max_len, kWideChunk) * (kWideChunk / 32); }

// Rows of up to kTopkRowMaxLen keys are short enough for one workgroup each,
// which holds the row in registers (one launch, no histogram); the few long
// rows of decode are spread over many workgroups.
bool topk_small_rows(const Geometry &g) { return g.max_len <= kTopkRowMaxLen; }
bool topk_uses_wide(const Geometry &g) { return g.rows <= kTopkWideMaxRows && !topk_small_rows(g); }

static size_t row_kernel_lds(int max_len) {
    return sizeof(uint32_t) * ((size_t)kHistWords + kLowBins + 2 * (size_t)row_words(max_len) +
                               2 * (size_t)kTopkCandCap);
}

size_t topk_lds_bytes(const Geometry &g) {
    if (topk_small_rows(g))  // short-row kernel: static LDS only
        return sizeof(uint32_t) * (2 * 16 * 8 + 2 * 16);
    if (topk_uses_wide(g))  // finish kernel: static histograms + two bitmaps
        return sizeof(uint32_t) * ((size_t)kHistWords + kLowBins + 2 * (size_t)wide_words(g.max_len));
    return row_kernel_lds(g.max_len);
}

TopkWideLayout topk_wide_layout(const Geometry &g) {
    TopkWideLayout L;
    L.words_max = wide_words(g.max_len);
    L.regions = L.words_max / 32;
    const size_t rows = (size_t)g.rows;
    L.hist_u32 = rows * kCoarseBins;
    L.bitmap_u32 = rows * L.words_max;
    L.cand_u32 = rows * L.regions * 1024;
    L.count_u32 = rows * L.regions;
    return L;
}

// R = c + max(c, 16), c = ceil(k / stride): a full row has about stride * R
// keys at or above the R-th largest sample, against the k it needs; the
// sampled keys among a row's top k number about c (at most about c + 4 sqrt(c)
// in practice), so fewer than k candidates is a many-sigma event.
int topk_sample_rank(const Geometry &g) {
    const int c = div_up(g.top_k, kTopkSampleStride);
    return c + (c > 16 ? c : 16);
}

// Many causal rows, k <= 2048, and rows long enough that the candidates
// (about stride * R per row) leave at most kTopkBlockMean per key block.
bool topk_uses_two_pass(const Geometry &g) {
    return index_uses_mfma(g) && g.rows > kTopkWideMaxRows && g.top_k <= kTopkTwoPassMaxK &&
           (int64_t)kTopkKeyBlock * kTopkSampleStride * topk_sample_rank(g) <=
               (int64_t)kTopkBlockMean * g.max_len;
}

hipError_t launch_topk_sample_thresh(const Geometry &g, const float *samples,
                                     const int32_t *seq_lens, const int32_t *q_pos,
                                     uint32_t *thresh, uint32_t *slow, hipStream_t stream) {
    if (g.rows == 0) return hipSuccess;
    SampleArgs a;
    a.samples = samples;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.thresh = thresh;
    a.slow = slow;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.causal = g.causal;
    a.top_k = g.top_k;
    a.cols = topk_sample_cols(g);
    a.rank = topk_sample_rank(g);
    if (a.cols <= 256 * kShortKeys)
        topk_sample_thresh_kernel<256><<<dim3(g.rows), dim3(256), 0, stream>>>(a);
    else
        topk_sample_thresh_kernel<512><<<dim3(g.rows), dim3(512), 0, stream>>>(a);
    return hipGetLastError();
}

hipError_t launch_topk_cands(const Geometry &g, const uint32_t *cand_count, const uint32_t *cands,
                             const int32_t *seq_lens, const int32_t *q_pos, const void *q_idx,
                             const void *k_idx, const int32_t *page_table, float *scores,
                             uint32_t *slow, int32_t *idx, int32_t *n_sel, hipStream_t stream) {
    if (g.rows == 0) return hipSuccess;
    CandArgs a;
    a.cand_count = cand_count;
    a.cands = reinterpret_cast<const uint2 *>(cands);
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.idx = idx;
    a.n_sel = n_sel;
    a.scores = scores;
    a.q_idx = static_cast<const uint16_t *>(q_idx);
    a.k_idx = static_cast<const uint16_t *>(k_idx);
    a.page_table = page_table;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.causal = g.causal;
    a.top_k = g.top_k;
    a.words_max = row_words(g.max_len);
    a.cand_cap = kTopkCandCap;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.kblocks = topk_key_blocks(g);
    a.slow = slow;
    const size_t fast_lds = (sizeof(uint32_t) + sizeof(uint16_t)) * (size_t)kCandCap;
    const bool two = a.kblocks > kCandThreads;  // more key blocks than threads
    const void *fast = two ? reinterpret_cast<const void *>(&topk_cand_fast_kernel<2>)
                           : reinterpret_cast<const void *>(&topk_cand_fast_kernel<1>);
    hipError_t e = hipFuncSetAttribute(fast, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)fast_lds);
    if (e != hipSuccess) return e;
    if (two) topk_cand_fast_kernel<2><<<dim3(g.rows), dim3(kCandThreads), fast_lds, stream>>>(a);
    else topk_cand_fast_kernel<1><<<dim3(g.rows), dim3(kCandThreads), fast_lds, stream>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t lds = row_kernel_lds(g.max_len);
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_cand_slow_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    topk_cand_slow_kernel<<<dim3(g.rows < 1024 ? g.rows : 1024), dim3(kRowThreads), lds, stream>>>(a);
    return hipGetLastError();
}

hipError_t launch_topk(const Geometry &g, const float *scores, const int32_t *seq_lens,
                       const int32_t *q_pos, const TopkBuffers &buf, bool hist_ready,
                       int32_t *idx, int32_t *n_sel, hipStream_t stream) {
    if (g.rows == 0) return hipSuccess;
    if (topk_uses_wide(g)) {
        const int cpr = div_up(g.max_len, kWideChunk);
        const size_t blocks = (size_t)g.rows * cpr;
        if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
        if (!hist_ready) {
            coarse_hist_kernel<<<dim3((unsigned)blocks), dim3(kWideThreads), 0, stream>>>(
                scores, seq_lens, q_pos, buf.hist, g.n_q, g.max_len, g.causal, cpr);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        const TopkWideLayout L = topk_wide_layout(g);
        TopkWideArgs a;
        a.scores = scores;
        a.seq_lens = seq_lens;
        a.q_pos = q_pos;
        a.hist = buf.hist;
        a.sure = buf.bitmaps;
        a.cands = buf.cands;
        a.counts = buf.counts;
        a.idx = idx;
        a.n_sel = n_sel;
        a.n_q = g.n_q;
        a.max_len = g.max_len;
        a.causal = g.causal;
        a.top_k = g.top_k;
        a.chunks_per_row = cpr;
        a.words_max = L.words_max;
        a.regions = L.regions;
        topk_filter_kernel<<<dim3((unsigned)blocks), dim3(kWideThreads), 0, stream>>>(a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const size_t lds = sizeof(uint32_t) * 2 * (size_t)L.words_max;
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_finish_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        topk_finish_kernel<<<dim3(g.rows), dim3(kRowThreads), lds, stream>>>(a);
        return hipGetLastError();
    }
    TopkRowArgs a;
    a.scores = scores;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.hist = hist_ready ? buf.hist : nullptr;
    a.idx = idx;
    a.n_sel = n_sel;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.causal = g.causal;
    a.top_k = g.top_k;
    a.words_max = row_words(g.max_len);
    a.cand_cap = kTopkCandCap;
    if (topk_small_rows(g)) {  // the whole row in registers (a histogram is not needed)
        if (g.max_len <= 256 * kShortKeys)
            topk_short_kernel<256><<<dim3(g.rows), dim3(256), 0, stream>>>(a);
        else if (g.max_len <= 512 * kShortKeys)
            topk_short_kernel<512><<<dim3(g.rows), dim3(512), 0, stream>>>(a);
        else
            topk_short_kernel<1024><<<dim3(g.rows), dim3(1024), 0, stream>>>(a);
        return hipGetLastError();
    }
    const size_t lds = row_kernel_lds(g.max_len);
    hipError_t e;
    if (hist_ready) {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_row_kernel<true>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        topk_row_kernel<true><<<dim3(g.rows), dim3(kRowThreads), lds, stream>>>(a);
    } else {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_row_kernel<false>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        topk_row_kernel<false><<<dim3(g.rows), dim3(kRowThreads), lds, stream>>>(a);
    }
    return hipGetLastError();
}

hipError_t take_device_error_topk(uint32_t *bits) { return take_source_device_error(bits); }

}  // namespace clsa
