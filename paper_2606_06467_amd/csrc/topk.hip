// Exact token-level top-k (Section 2.1, Eq. 3: S_t = TopK(I_t, k)).
//
// No sort.  One 1024-thread workgroup owns one query row and finds the exact
// k-th largest key tau with a radix select on the order-preserving uint32 keys
// of the fp32 scores, then emits the selected positions in ascending order:
//
//   1. coarse histogram of the top 8 key bits (taken from the indexer when it
//      made one, else one pass over the row) -> bin b1 that holds the k-th key;
//   2. one pass over the row: keys above b1 are certainly selected (bitmap
//      words built with wavefront ballots), keys in b1 are appended to an LDS
//      candidate list;
//   3. two LDS radix passes (12 + 12 bits) over the candidates -> tau and r,
//      the number of keys equal to tau that are still to be taken;
//   4. candidates above tau go into the "sure" bitmap, those equal to tau into
//      a "tie" bitmap;
//   5. a block-wide scan of the bitmaps' popcounts gives each word its output
//      offset; of the ties only the first r in position order are kept, which
//      is the lowest-index-wins rule.
// If the candidate list overflows its LDS capacity (very flat score rows), the
// passes of steps 3-4 re-read the row from memory instead: slower, same result.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kFineBins = 4096;  // 12-bit refinement digits

struct TopkArgs {
    const float *scores;
    const int32_t *seq_lens;
    const int32_t *q_pos;
    const uint32_t *hist;
    int32_t *idx;
    int32_t *n_sel;
    int n_q, max_len, causal, top_k;
    int words_max;  // bitmap words reserved in LDS per bitmap (even)
    int cand_cap;
};

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t t = __shfl_up(v, d);
        if (lane >= d) v += t;
    }
    return v;
}

// Exclusive prefix over the workgroup of one value per thread; also returns the total.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *s_wave, uint32_t &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t inc = wave_incl_scan(v, lane);
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    if (wave == 0) {
        uint32_t w = lane < kTopkWaves ? s_wave[lane] : 0u;
        const uint32_t wi = wave_incl_scan(w, lane);
        if (lane < kTopkWaves) s_wave[kTopkWaves + lane] = wi - w;
        if (lane == kTopkWaves - 1) s_wave[2 * kTopkWaves] = wi;
    }
    __syncthreads();
    const uint32_t r = s_wave[kTopkWaves + wave] + inc - v;
    total = s_wave[2 * kTopkWaves];
    __syncthreads();
    return r;
}

// Given hist[nbins] in LDS, find the bin b with suffix(b) >= need > suffix(b+1),
// where suffix(x) = sum of bins >= x.  Writes b and suffix(b+1) to out[0..1].
// nbins is a multiple of the thread count times the bins per thread.
__device__ void find_threshold_bin(const uint32_t *hist, int nbins, uint32_t need,
                                   uint32_t *s_wave, uint32_t *out) {
    const int per = nbins / kTopkThreads > 0 ? nbins / kTopkThreads : 1;
    // thread t owns bins [nbins - (t+1)*per, nbins - t*per): thread 0 owns the top bins,
    // so an exclusive prefix over threads is a suffix over bins.
    if (threadIdx.x == 0) {  // defined result even if the counts were inconsistent
        out[0] = 0u;
        out[1] = 0u;
    }
    const int hi = nbins - threadIdx.x * per;
    const int lo = hi - per;
    uint32_t s = 0;
    if (lo >= 0)
        for (int x = lo; x < hi; ++x) s += hist[x];
    uint32_t total;
    const uint32_t above = block_excl_scan(s, s_wave, total);  // keys in bins >= hi
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

template <bool HAVE_HIST>
__global__ __launch_bounds__(kTopkThreads) void topk_row_kernel(TopkArgs a) {
    extern __shared__ uint32_t lds[];
    __shared__ uint32_t s_wave[2 * kTopkWaves + 1];
    __shared__ uint32_t s_res[8];
    __shared__ uint32_t s_cand_count;

    const int row = blockIdx.x;
    const int b = row / a.n_q;
    const int n = valid_keys(a.seq_lens, a.q_pos, a.causal, b, row, a.max_len);
    const int k = a.top_k;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t *out = a.idx + (size_t)row * k;

    if (n <= k) {  // every valid key is selected
        for (int i = tid; i < k; i += kTopkThreads) out[i] = i < n ? i : -1;
        if (tid == 0) a.n_sel[row] = n;
        return;
    }
    const float *srow = a.scores + (size_t)row * a.max_len;
    uint32_t *hist = lds;                      // kFineBins
    uint32_t *sure = hist + kFineBins;         // words_max
    uint32_t *tie = sure + a.words_max;        // words_max
    uint32_t *ckey = tie + a.words_max;        // cand_cap
    uint32_t *cidx = ckey + a.cand_cap;        // cand_cap
    const int nchunks = div_up(n, 1024);       // 1024 keys per wave-chunk
    const int words = nchunks * 32;            // bitmap words touched

    // ---- 1. coarse histogram (top 8 key bits) -> b1 ----
    if (tid < kCoarseBins) hist[tid] = HAVE_HIST ? a.hist[(size_t)row * kCoarseBins + tid] : 0u;
    if (tid == 0) s_cand_count = 0u;
    __syncthreads();
    if (!HAVE_HIST) {
        for (int c = wave; c < nchunks; c += kTopkWaves) {
            const int base = c * 1024 + lane;
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int j = base + u * 64;
                if (j < n) atomicAdd(&hist[score_key(srow[j]) >> 24], 1u);
            }
        }
        __syncthreads();
    }
    find_threshold_bin(hist, kCoarseBins, (uint32_t)k, s_wave, s_res);
    const uint32_t b1 = s_res[0];
    const uint32_t above1 = s_res[1];
    __syncthreads();

    // ---- 2. sure bits for keys above b1, candidate list for keys in b1 ----
    for (int c = wave; c < nchunks; c += kTopkWaves) {
        const int base = c * 1024 + lane;
        uint32_t key[16];
        uint64_t cmask[16];
        uint32_t ccount = 0;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int j = base + u * 64;
            key[u] = j < n ? score_key(__builtin_nontemporal_load(srow + j)) : 0u;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int j = base + u * 64;
            const uint32_t d = key[u] >> 24;
            const uint64_t sm = __ballot(j < n && d > b1);
            cmask[u] = __ballot(j < n && d == b1);
            ccount += __popcll(cmask[u]);
            if (lane < 2) {
                const int w = c * 32 + 2 * u + lane;
                sure[w] = lane ? (uint32_t)(sm >> 32) : (uint32_t)sm;
                tie[w] = 0u;
            }
        }
        uint32_t slot = 0;
        if (lane == 0 && ccount) slot = atomicAdd(&s_cand_count, ccount);
        slot = __shfl(slot, 0);
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const uint64_t lower = lane ? (cmask[u] << (64 - lane)) : 0ull;
            if ((cmask[u] >> lane) & 1ull) {
                const uint32_t at = slot + (uint32_t)__popcll(lower);
                if (at < (uint32_t)a.cand_cap) {
                    ckey[at] = key[u];
                    cidx[at] = (uint32_t)(base + u * 64);
                }
            }
            slot += (uint32_t)__popcll(cmask[u]);
        }
    }
    __syncthreads();
    const uint32_t ncand = s_cand_count;
    const bool in_lds = ncand <= (uint32_t)a.cand_cap;

    // Visit every candidate (key in bin b1): from the LDS list or from the row.
    auto for_each_candidate = [&](auto &&fn) {
        if (in_lds) {
            for (uint32_t i = tid; i < ncand; i += kTopkThreads) fn(ckey[i], cidx[i]);
        } else {
            for (int j = tid; j < n; j += kTopkThreads) {
                const uint32_t key = score_key(srow[j]);
                if ((key >> 24) == b1) fn(key, (uint32_t)j);
            }
        }
    };

    // ---- 3. refine: bits 23..12 then 11..0 ----
    const uint32_t need1 = (uint32_t)k - above1;
    for (int x = tid; x < kFineBins; x += kTopkThreads) hist[x] = 0u;
    __syncthreads();
    for_each_candidate([&](uint32_t key, uint32_t) { atomicAdd(&hist[(key >> 12) & 0xfffu], 1u); });
    __syncthreads();
    find_threshold_bin(hist, kFineBins, need1, s_wave, s_res);
    const uint32_t b2 = s_res[0];
    const uint32_t need2 = need1 - s_res[1];
    __syncthreads();
    const uint32_t pref20 = (b1 << 12) | b2;
    for (int x = tid; x < kFineBins; x += kTopkThreads) hist[x] = 0u;
    __syncthreads();
    for_each_candidate([&](uint32_t key, uint32_t) {
        if ((key >> 12) == pref20) atomicAdd(&hist[key & 0xfffu], 1u);
    });
    __syncthreads();
    find_threshold_bin(hist, kFineBins, need2, s_wave, s_res);
    const uint32_t tau = (pref20 << 12) | s_res[0];
    const uint32_t r_ties = need2 - s_res[1];  // >= 1 keys equal to tau are taken
    __syncthreads();

    // ---- 4. mark candidates above / equal to tau ----
    for_each_candidate([&](uint32_t key, uint32_t j) {
        if (key > tau) atomicOr(&sure[j >> 5], 1u << (j & 31));
        else if (key == tau) atomicOr(&tie[j >> 5], 1u << (j & 31));
    });
    __syncthreads();

    // ---- 5. ordered compaction ----
    const int per = div_up(words, kTopkThreads);
    const int w0 = tid * per;
    const int w1 = min(words, w0 + per);
    uint32_t cs = 0, ct = 0;
    for (int w = w0; w < w1; ++w) {
        cs += __popc(sure[w]);
        ct += __popc(tie[w]);
    }
    uint32_t tot_s, tot_t;
    uint32_t sure_before = block_excl_scan(cs, s_wave, tot_s);
    uint32_t tie_before = block_excl_scan(ct, s_wave, tot_t);
    for (int w = w0; w < w1; ++w) {
        uint32_t sel = sure[w];
        uint32_t tw = tie[w];
        const uint32_t pos0 = sure_before + min(tie_before, r_ties);
        // keep only the ties whose rank (in position order) is below r_ties
        uint32_t take = tie_before < r_ties ? r_ties - tie_before : 0u;
        tie_before += __popc(tw);
        while (tw && take) {
            const uint32_t low = tw & (0u - tw);
            sel |= low;
            tw ^= low;
            --take;
        }
        sure_before += __popc(sure[w]);
        uint32_t pos = pos0;
        while (sel && pos < (uint32_t)k) {
            const int bit = __ffs(sel) - 1;
            sel &= sel - 1;
            out[pos++] = w * 32 + bit;
        }
    }
    if (tid == 0) a.n_sel[row] = k;
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

static int words_for(int max_len) { return div_up(max_len, 1024) * 32; }

size_t topk_lds_bytes(int max_len) {
    return sizeof(uint32_t) * ((size_t)kFineBins + 2 * (size_t)words_for(max_len) +
                               2 * (size_t)kTopkCandCap);
}

hipError_t launch_topk(const Geometry &g, const float *scores, const int32_t *seq_lens,
                       const int32_t *q_pos, const uint32_t *coarse_hist, int32_t *idx,
                       int32_t *n_sel, hipStream_t stream) {
    TopkArgs a;
    a.scores = scores;
    a.seq_lens = seq_lens;
    a.q_pos = q_pos;
    a.hist = coarse_hist;
    a.idx = idx;
    a.n_sel = n_sel;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.causal = g.causal;
    a.top_k = g.top_k;
    a.words_max = words_for(g.max_len);
    a.cand_cap = kTopkCandCap;
    const size_t lds = topk_lds_bytes(g.max_len);
    if (g.rows == 0) return hipSuccess;
    hipError_t e;
    if (coarse_hist) {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_row_kernel<true>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        topk_row_kernel<true><<<dim3(g.rows), dim3(kTopkThreads), lds, stream>>>(a);
    } else {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_row_kernel<false>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        topk_row_kernel<false><<<dim3(g.rows), dim3(kTopkThreads), lds, stream>>>(a);
    }
    return hipGetLastError();
}

}  // namespace clsa
