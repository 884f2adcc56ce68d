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
//     candidate list in LDS -- for many rows (chunked prefill);
//   * for the few, long rows of decode, step 2 is spread over many 256-thread
//     workgroups (topk_filter_kernel, 4096 keys each, global bitmaps and a
//     global candidate list) and a second launch with one workgroup per row
//     (topk_finish_kernel) does steps 3-5 with the bitmaps copied to LDS.  The
//     hand-off goes through the kernel boundary: a ticket taken by the last
//     filter workgroup would need an agent-scope release fence, which on this
//     chip writes back the whole L2 of the XCD from every workgroup.
// If a candidate list overflows (very flat score rows), steps 3-4 re-read the
// row instead: slower, same result.
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

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t t = __shfl_up(v, d);
        if (lane >= d) v += t;
    }
    return v;
}

// Exclusive prefix over the workgroup of one value per thread; also returns the total.
// s_wave needs 2 * NT/64 + 1 entries.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *s_wave, uint32_t &total) {
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t inc = wave_incl_scan(v, lane);
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    if (wave == 0) {
        const uint32_t w = lane < NW ? s_wave[lane] : 0u;
        const uint32_t wi = wave_incl_scan(w, lane);
        if (lane < NW) s_wave[NW + lane] = wi - w;
        if (lane == NW - 1) s_wave[2 * NW] = wi;
    }
    __syncthreads();
    const uint32_t r = s_wave[NW + wave] + inc - v;
    total = s_wave[2 * NW];
    __syncthreads();
    return r;
}

// Given hist[nbins] in LDS, find the bin b with suffix(b) >= need > suffix(b+1),
// suffix(x) = sum of the bins >= x.  Writes b and suffix(b+1) to out[0..1]
// (0, 0 if no bin qualifies, which consistent counts never produce).
template <int NT>
__device__ void find_threshold_bin(const uint32_t *hist, int nbins, uint32_t need,
                                   uint32_t *s_wave, uint32_t *out) {
    const int per = nbins / NT > 0 ? nbins / NT : 1;
    if (threadIdx.x == 0) {
        out[0] = 0u;
        out[1] = 0u;
    }
    // thread t owns bins [nbins - (t+1)*per, nbins - t*per): thread 0 owns the top
    // bins, so an exclusive prefix over threads is a suffix over bins.
    const int hi = nbins - (int)threadIdx.x * per;
    const int lo = hi - per;
    uint32_t s = 0;
    if (lo >= 0)
        for (int x = lo; x < hi; ++x) s += hist[x];
    uint32_t total;
    const uint32_t above = block_excl_scan<NT>(s, s_wave, total);  // keys in bins >= hi
    if (lo >= 0 && above < need && above + s >= need) {
        uint32_t acc = above;
        for (int x = hi - 1; x >= lo; --x) {
            const uint32_t c = hist[x];
            if (acc + c >= need) {
                out[0] = (uint32_t)x;
                out[1] = acc;
                break;
            }
            acc += c;
        }
    }
    __syncthreads();
}

// Steps 3 and 4 for the keys of coarse bin b1 (visited by `visit(fn)`, which
// calls fn(key, position) for every such key).  hist: LDS [kHistWords].
template <int NT, class Visit>
__device__ void refine_and_mark(Visit visit, uint32_t b1, uint32_t need1, uint32_t *hist,
                                uint32_t *s_wave, uint32_t *s_res, uint32_t *sure, uint32_t *tie,
                                uint32_t &r_ties) {
    for (int x = threadIdx.x; x < kMidBins; x += NT) hist[x] = 0u;
    __syncthreads();
    visit([&](uint32_t key, uint32_t) {
        atomicAdd(&hist[(key >> kMidShift) & (kMidBins - 1)], 1u);
    });
    __syncthreads();
    find_threshold_bin<NT>(hist, kMidBins, need1, s_wave, s_res);
    const uint32_t b2 = s_res[0];
    const uint32_t need2 = need1 - s_res[1];
    __syncthreads();
    const uint32_t pref = (b1 << (kCoarseShift - kMidShift)) | b2;  // key >> kMidShift
    for (int x = threadIdx.x; x < kLowBins; x += NT) hist[x] = 0u;
    __syncthreads();
    visit([&](uint32_t key, uint32_t) {
        if ((key >> kMidShift) == pref) atomicAdd(&hist[key & (kLowBins - 1)], 1u);
    });
    __syncthreads();
    find_threshold_bin<NT>(hist, kLowBins, need2, s_wave, s_res);
    const uint32_t tau = (pref << kMidShift) | s_res[0];
    r_ties = need2 - s_res[1];  // keys equal to tau that are taken (>= 1)
    __syncthreads();
    visit([&](uint32_t key, uint32_t j) {
        if (key > tau) atomicOr(&sure[j >> 5], 1u << (j & 31));
        else if (key == tau) atomicOr(&tie[j >> 5], 1u << (j & 31));
    });
}

// Step 5: ordered output from the bitmaps (words [0, words)).
template <int NT>
__device__ void compact_bitmaps(const uint32_t *sure, const uint32_t *tie, int words,
                                uint32_t r_ties, int k, int32_t *out, uint32_t *s_wave) {
    const int per = div_up(words, NT);
    const int w0 = threadIdx.x * per;
    const int w1 = min(words, w0 + per);
    uint32_t cs = 0, ct = 0;
    for (int w = w0; w < w1; ++w) {
        cs += __popc(sure[w]);
        ct += __popc(tie[w]);
    }
    uint32_t tot_s, tot_t;
    uint32_t sure_before = block_excl_scan<NT>(cs, s_wave, tot_s);
    uint32_t tie_before = block_excl_scan<NT>(ct, s_wave, tot_t);
    for (int w = w0; w < w1; ++w) {
        const uint32_t sw = sure[w];
        uint32_t sel = sw;
        uint32_t tw = tie[w];
        uint32_t pos = sure_before + min(tie_before, r_ties);
        uint32_t take = tie_before < r_ties ? r_ties - tie_before : 0u;
        tie_before += __popc(tw);
        sure_before += __popc(sw);
        while (tw && take) {  // the lowest-index ties are the ones kept
            const uint32_t low = tw & (0u - tw);
            sel |= low;
            tw ^= low;
            --take;
        }
        while (sel && pos < (uint32_t)k) {
            const int bit = __ffs(sel) - 1;
            sel &= sel - 1;
            out[pos++] = w * 32 + bit;
        }
    }
}

// One wave's share of the filter pass: 1024 keys starting at `base`, lane-strided
// so that each ballot is exactly two bitmap words.  Keys past n are neither
// selected nor candidates.  Candidate slots come from `*cand_count`.
template <class AppendFn>
__device__ __forceinline__ void filter_1024(const float *srow, int base, int n, uint32_t b1,
                                            uint32_t *sure_words, uint32_t *tie_words,
                                            uint32_t *cand_count, AppendFn append) {
    const int lane = threadIdx.x & 63;
    uint32_t key[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const int j = min(base + u * 64 + lane, n - 1);
        key[u] = score_key(__builtin_nontemporal_load(srow + j));
    }
    uint64_t cmask[16];
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
            tie_words[2 * u + lane] = 0u;
        }
    }
    uint32_t slot = 0;
    if (lane == 0 && ccount) slot = atomicAdd(cand_count, ccount);
    slot = __shfl(slot, 0);
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

template <bool HAVE_HIST>
__global__ __launch_bounds__(kRowThreads) void topk_row_kernel(TopkRowArgs a) {
    constexpr int NW = kRowThreads / 64;
    extern __shared__ uint32_t lds[];
    __shared__ uint32_t s_wave[2 * NW + 1];
    __shared__ uint32_t s_res[2];
    __shared__ uint32_t s_cand_count;

    const int row = blockIdx.x;
    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int k = a.top_k;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t *out = a.idx + (size_t)row * k;
    if (n <= k) {  // every valid key is selected
        for (int i = tid; i < k; i += kRowThreads) out[i] = i < n ? i : -1;
        if (tid == 0) a.n_sel[row] = n;
        return;
    }
    const float *srow = a.scores + (size_t)row * a.max_len;
    uint32_t *hist = lds;                // kHistWords
    uint32_t *sure = hist + kHistWords;  // words_max
    uint32_t *tie = sure + a.words_max;  // words_max
    uint32_t *ckey = tie + a.words_max;  // cand_cap
    uint32_t *cidx = ckey + a.cand_cap;  // cand_cap
    const int nchunks = div_up(n, 1024);

    for (int x = tid; x < kCoarseBins; x += kRowThreads)
        hist[x] = HAVE_HIST ? a.hist[(size_t)row * kCoarseBins + x] : 0u;
    if (tid == 0) s_cand_count = 0u;
    __syncthreads();
    if (!HAVE_HIST) {
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
    find_threshold_bin<kRowThreads>(hist, kCoarseBins, (uint32_t)k, s_wave, s_res);
    const uint32_t b1 = s_res[0];
    const uint32_t need1 = (uint32_t)k - s_res[1];
    __syncthreads();

    const uint32_t cap = (uint32_t)a.cand_cap;
    for (int c = wave; c < nchunks; c += NW)
        filter_1024(srow, c * 1024, n, b1, sure + c * 32, tie + c * 32, &s_cand_count,
                    [&](uint32_t at, uint32_t key, uint32_t j) {
                        if (at < cap) {
                            ckey[at] = key;
                            cidx[at] = j;
                        }
                    });
    __syncthreads();
    const uint32_t ncand = s_cand_count;
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
    refine_and_mark<kRowThreads>(visit, b1, need1, hist, s_wave, s_res, sure, tie, r_ties);
    __syncthreads();
    compact_bitmaps<kRowThreads>(sure, tie, nchunks * 32, r_ties, k, out, s_wave);
    if (tid == 0) a.n_sel[row] = k;
}

// ------------------------------------------------------------------------------------
// Wide kernel (few long rows).

struct TopkWideArgs {
    const float *scores;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    const uint32_t *hist;   // [rows, 256], complete
    uint32_t *counters;     // [rows, 2]: candidate count (zero on entry), spare
    uint32_t *sure;         // [rows, words_max]
    uint32_t *tie;          // [rows, words_max]
    uint32_t *ckey;         // [rows, cand_cap]
    uint32_t *cidx;         // [rows, cand_cap]
    int32_t *idx;
    int32_t *n_sel;
    int n_q, max_len, causal, top_k, chunks_per_row, words_max, cand_cap;
};

// b1 (the coarse bin of the k-th key) and k minus the keys above it, from the
// row's complete coarse histogram.  hist: LDS scratch of kCoarseBins words.
template <int NT>
__device__ __forceinline__ void coarse_threshold(const uint32_t *ghist, int k, uint32_t *hist,
                                                 uint32_t *s_wave, uint32_t *s_res,
                                                 uint32_t &b1, uint32_t &need1) {
    for (int x = threadIdx.x; x < kCoarseBins; x += NT) hist[x] = ghist[x];
    __syncthreads();
    find_threshold_bin<NT>(hist, kCoarseBins, (uint32_t)k, s_wave, s_res);
    b1 = s_res[0];
    need1 = (uint32_t)k - s_res[1];
    __syncthreads();
}

// Step 2 for 4096 keys of one row.
__global__ __launch_bounds__(kWideThreads) void topk_filter_kernel(TopkWideArgs a) {
    constexpr int NW = kWideThreads / 64;
    __shared__ uint32_t hist[kCoarseBins];
    __shared__ uint32_t s_wave[2 * NW + 1];
    __shared__ uint32_t s_res[2];

    const int row = blockIdx.x / a.chunks_per_row;
    const int c = blockIdx.x - row * a.chunks_per_row;
    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    if (n <= a.top_k || c * kWideChunk >= n) return;  // uniform
    const int wave = threadIdx.x >> 6;
    uint32_t b1, need1;
    coarse_threshold<kWideThreads>(a.hist + (size_t)row * kCoarseBins, a.top_k, hist, s_wave,
                                   s_res, b1, need1);
    const float *srow = a.scores + (size_t)row * a.max_len;
    uint32_t *ckey = a.ckey + (size_t)row * a.cand_cap;
    uint32_t *cidx = a.cidx + (size_t)row * a.cand_cap;
    const uint32_t cap = (uint32_t)a.cand_cap;
    const int base = c * kWideChunk + wave * 1024;
    filter_1024(srow, base, n, b1, a.sure + (size_t)row * a.words_max + base / 32,
                a.tie + (size_t)row * a.words_max + base / 32, a.counters + 2 * (size_t)row,
                [&](uint32_t at, uint32_t key, uint32_t j) {
                    if (at < cap) {
                        ckey[at] = key;
                        cidx[at] = j;
                    }
                });
}

// Steps 3-5 for one row; the bitmaps are copied to LDS (dynamic, 2 x words_max).
__global__ __launch_bounds__(kRowThreads) void topk_finish_kernel(TopkWideArgs a) {
    constexpr int NW = kRowThreads / 64;
    extern __shared__ uint32_t lds[];
    __shared__ uint32_t hist[kHistWords];
    __shared__ uint32_t s_wave[2 * NW + 1];
    __shared__ uint32_t s_res[2];

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
    const int words = div_up(n, kWideChunk) * (kWideChunk / 32);
    uint32_t *sure = lds;
    uint32_t *tie = lds + a.words_max;
    const uint32_t *gs = a.sure + (size_t)row * a.words_max;
    const uint32_t *gt = a.tie + (size_t)row * a.words_max;
    for (int w = tid; w < words; w += kRowThreads) {
        sure[w] = gs[w];
        tie[w] = gt[w];
    }
    uint32_t b1, need1;
    coarse_threshold<kRowThreads>(a.hist + (size_t)row * kCoarseBins, k, hist, s_wave, s_res, b1,
                                  need1);
    const float *srow = a.scores + (size_t)row * a.max_len;
    const uint32_t *ckey = a.ckey + (size_t)row * a.cand_cap;
    const uint32_t *cidx = a.cidx + (size_t)row * a.cand_cap;
    const uint32_t ncand = a.counters[2 * (size_t)row];
    const uint32_t cap = (uint32_t)a.cand_cap;
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
    refine_and_mark<kRowThreads>(visit, b1, need1, hist, s_wave, s_res, sure, tie, r_ties);
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

bool topk_uses_wide(const Geometry &g) { return g.rows <= kTopkWideMaxRows; }

static size_t row_kernel_lds(int max_len) {
    return sizeof(uint32_t) * ((size_t)kHistWords + 2 * (size_t)row_words(max_len) +
                               2 * (size_t)kTopkCandCap);
}

size_t topk_lds_bytes(const Geometry &g) {
    if (topk_uses_wide(g))  // finish kernel: static fine histogram + two bitmaps
        return sizeof(uint32_t) * ((size_t)kHistWords + 2 * (size_t)wide_words(g.max_len));
    return row_kernel_lds(g.max_len);
}

TopkWideLayout topk_wide_layout(const Geometry &g) {
    TopkWideLayout L;
    L.words_max = wide_words(g.max_len);
    L.cand_cap = kTopkWideCandCap;
    const size_t rows = (size_t)g.rows;
    L.hist_u32 = rows * kCoarseBins;
    L.counters_u32 = rows * 2;
    L.bitmap_u32 = rows * L.words_max;
    L.cand_u32 = rows * (size_t)L.cand_cap;
    return L;
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
        a.counters = buf.counters;
        a.sure = buf.bitmaps;
        a.tie = buf.bitmaps + L.bitmap_u32;
        a.ckey = buf.cands;
        a.cidx = buf.cands + L.cand_u32;
        a.idx = idx;
        a.n_sel = n_sel;
        a.n_q = g.n_q;
        a.max_len = g.max_len;
        a.causal = g.causal;
        a.top_k = g.top_k;
        a.chunks_per_row = cpr;
        a.words_max = L.words_max;
        a.cand_cap = L.cand_cap;
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

}  // namespace clsa
