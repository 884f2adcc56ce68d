// C-ABI entry points of libclsa: host-side validation, workspace carving and
// kernel dispatch.  Nothing here allocates device memory, and only the debug
// call clsa_get_device_error synchronises.
#include "clsa.h"

#include <math.h>
#include <stdint.h>

#include <atomic>

#include "clsa_internal.h"

namespace {

using clsa::Geometry;

using clsa::kMaxTopK;
using clsa::kMaxLen;
constexpr size_t kAlign = 256;

constexpr int kHookLayers = 64;  // layers whose attention kernel the hook can bracket
struct PhaseHook {
    hipEvent_t ev[4 + 2 * kHookLayers];
    int layers = 0;                 // layers bracketed by ev[4 + 2l], ev[5 + 2l]
    bool on = false;
};
// The profiling hook belongs to the host thread that set it: calls made from
// other threads never see it, so concurrent callers do not share any state here.
thread_local PhaseHook t_hook;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

int log2i(int x) {
    int s = 0;
    while ((1 << s) < x) ++s;
    return s;
}

enum Needs : unsigned { kIndex = 1u, kTopk = 2u, kAttn = 4u, kDense = 8u };

// Checks the shape for the operations in `needs` and fills the kernel geometry.
clsa_status check_shape(const clsa_shape *s, unsigned needs, Geometry *g) {
    if (!s) return CLSA_ERR_INVALID_ARG;
    if (s->batch < 1 || s->n_q < 1 || s->max_len < 1 || s->top_k < 1) return CLSA_ERR_INVALID_ARG;
    if (s->idx_heads < 1 || s->idx_dim < 1 || s->q_heads < 1 || s->kv_heads < 1 || s->head_dim < 1)
        return CLSA_ERR_INVALID_ARG;
    if ((int64_t)s->batch * s->n_q > 0x7fffffff) return CLSA_ERR_INVALID_ARG;
    if (s->causal != 0 && s->causal != 1) return CLSA_ERR_INVALID_ARG;
    if (s->page_size != 0) {
        if (!is_pow2(s->page_size)) return CLSA_ERR_INVALID_ARG;
        if (s->max_len % s->page_size != 0) return CLSA_ERR_INVALID_ARG;
        if ((int64_t)s->max_pages * s->page_size < s->max_len) return CLSA_ERR_INVALID_ARG;
        if (s->page_size < 16 || s->page_size > 4096) return CLSA_ERR_UNSUPPORTED;
    }
    if ((needs & kAttn) && !isfinite(s->softmax_scale)) return CLSA_ERR_INVALID_ARG;
    if ((needs & kAttn) && s->q_heads % s->kv_heads != 0) return CLSA_ERR_INVALID_ARG;
    // contiguous caches: one sequence's K (or V) cache is addressed with 32-bit offsets
    if ((needs & kAttn) && s->page_size == 0 &&
        (int64_t)s->max_len * s->kv_heads * 256 >= ((int64_t)1 << 32))
        return CLSA_ERR_UNSUPPORTED;
    if ((needs & kIndex) && s->idx_heads * s->idx_dim != 256) return CLSA_ERR_UNSUPPORTED;
    if (needs & kAttn) {
        const int grp = s->q_heads / s->kv_heads;
        if (s->head_dim != 128) return CLSA_ERR_UNSUPPORTED;
        if (grp != 1 && grp != 2 && grp != 4 && grp != 5 && grp != 8) return CLSA_ERR_UNSUPPORTED;
    }
    if (s->top_k > kMaxTopK) return CLSA_ERR_UNSUPPORTED;
    if ((needs & (kIndex | kTopk | kDense)) && s->max_len > kMaxLen) return CLSA_ERR_UNSUPPORTED;
    g->batch = s->batch;
    g->n_q = s->n_q;
    g->rows = s->batch * s->n_q;
    g->max_len = s->max_len;
    g->page_shift = s->page_size ? log2i(s->page_size) : -1;
    g->max_pages = s->page_size ? s->max_pages : 0;
    g->top_k = s->top_k;
    g->causal = s->causal;
    g->q_heads = s->q_heads;
    g->kv_heads = s->kv_heads;
    g->group = s->q_heads / s->kv_heads;
    g->softmax_scale = s->softmax_scale;
    return CLSA_OK;
}

clsa_status check_ptr(const void *p, uintptr_t align) {
    if (!p || !aligned(p, align)) return CLSA_ERR_INVALID_ARG;
    return CLSA_OK;
}

#define CLSA_TRY(expr)                        \
    do {                                      \
        const clsa_status st_ = (expr);       \
        if (st_ != CLSA_OK) return st_;       \
    } while (0)

clsa_status check_common(const clsa_shape *s, const int32_t *page_table, const int32_t *q_pos,
                         bool uses_q_pos, bool uses_pages) {
    if (uses_pages && s->page_size) CLSA_TRY(check_ptr(page_table, 4));
    if (uses_q_pos && s->causal) CLSA_TRY(check_ptr(q_pos, 4));
    return CLSA_OK;
}

// Device limit on LDS per workgroup, one entry per device (0 = not read yet).
// Threads that race on an entry store the same value, so relaxed atomics suffice.
using clsa::kMaxDevices;
static_assert(CLSA_NOALLOC_SCRATCH_BYTES == clsa::kNoallocScratchBytes, "one scratch size");
std::atomic<int> g_lds_limit[kMaxDevices];

clsa_status check_topk_lds(const Geometry &g) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return CLSA_ERR_HIP;
    int lds = dev >= 0 && dev < kMaxDevices ? g_lds_limit[dev].load(std::memory_order_relaxed) : 0;
    if (lds == 0) {
        if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
            return CLSA_ERR_HIP;
        if (dev >= 0 && dev < kMaxDevices) g_lds_limit[dev].store(lds, std::memory_order_relaxed);
    }
    return clsa::topk_lds_bytes(g) + 1024 <= (size_t)lds ? CLSA_OK : CLSA_ERR_UNSUPPORTED;
}

// Carves 256-byte aligned sub-buffers out of a workspace; with base == nullptr
// it only adds up the sizes.
struct Carver {
    char *base;
    size_t off = 0;
    template <class T>
    T *take(size_t count) {
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += align_up(sizeof(T) * count);
        return count ? p : nullptr;
    }
};

struct TopkWs {
    clsa::TopkBuffers buf{};
    uint32_t *zero = nullptr;  // start of the region to clear before use
    size_t zero_count = 0;
};

// Multi-workgroup top-k state: the coarse histogram (cleared per call), the
// bitmap, the candidate regions and their counts.
void carve_topk(const Geometry &g, Carver &c, TopkWs &t) {
    if (!clsa::topk_uses_wide(g)) return;
    const clsa::TopkWideLayout L = clsa::topk_wide_layout(g);
    t.zero_count = L.hist_u32;
    t.zero = c.take<uint32_t>(t.zero_count);
    t.buf.hist = t.zero;
    t.buf.bitmaps = c.take<uint32_t>(L.bitmap_u32);
    t.buf.cands = c.take<uint32_t>(L.cand_u32);
    t.buf.counts = c.take<uint32_t>(L.count_u32);
}

struct AttnWs {
    float *partials = nullptr;
};

void carve_attn(const Geometry &g, Carver &c, AttnWs &w, bool dense = false) {
    w.partials = c.take<float>(clsa::attn_partial_floats(g, dense));  // none with one split
}

struct DecodeWs {
    float *scores = nullptr;
    uint32_t *zero = nullptr;  // coarse histogram, cleared per step
    size_t zero_count = 0;
    clsa::TopkBuffers topk{};
    float *partials = nullptr;
    // two-pass chunked-prefill top-k
    float *samples = nullptr;      // [rows, sample columns]
    uint32_t *thresh = nullptr;    // [rows]
    uint32_t *cand_count = nullptr;  // [rows, key blocks]
    uint32_t *cands = nullptr;     // [rows, key blocks, kTopkBlockSlots, 2]
    uint32_t *slow = nullptr;      // [1 + rows]: rows selected the slow way
    uint32_t *tickets = nullptr;   // [rows, kv_heads]: split arrivals of the in-kernel merge,
                                   // cleared by the first index launch of every index set
};

// Every layer gathers its K/V rows from the cache through the shared index set.
// (A once-per-step compact copy of the selected rows measured slower on the
// 128K step: the layers are bound by memory latency and kernel boundaries, not
// by the gather pattern, and the copy costs a full read and write of the rows.)
size_t carve_decode(const Geometry &g, void *base, DecodeWs &w) {
    Carver c{static_cast<char *>(base)};
    w.scores = c.take<float>((size_t)g.rows * g.max_len);
    w.zero_count = (size_t)g.rows * clsa::kCoarseBins;
    w.zero = c.take<uint32_t>(w.zero_count);
    w.topk.hist = w.zero;
    if (clsa::topk_uses_wide(g)) {
        const clsa::TopkWideLayout L = clsa::topk_wide_layout(g);
        w.topk.bitmaps = c.take<uint32_t>(L.bitmap_u32);
        w.topk.cands = c.take<uint32_t>(L.cand_u32);
        w.topk.counts = c.take<uint32_t>(L.count_u32);
    }
    w.partials = c.take<float>(clsa::attn_partial_floats(g));
    w.tickets = c.take<uint32_t>((size_t)g.rows * g.kv_heads);
    if (clsa::topk_uses_two_pass(g)) {
        w.samples = c.take<float>((size_t)g.rows * clsa::topk_sample_cols(g));
        w.thresh = c.take<uint32_t>(g.rows);
        const size_t blocks = (size_t)g.rows * clsa::topk_key_blocks(g);
        w.cand_count = c.take<uint32_t>(blocks);
        w.cands = c.take<uint32_t>(blocks * clsa::kTopkBlockSlots * 2);
        w.slow = c.take<uint32_t>((size_t)g.rows + 1);
    }
    return c.off;
}

size_t topk_ws_bytes(const Geometry &g) {
    Carver c{nullptr};
    TopkWs t;
    carve_topk(g, c, t);
    return c.off;
}

size_t attn_ws_bytes(const Geometry &g, bool dense = false) {
    Carver c{nullptr};
    AttnWs w;
    carve_attn(g, c, w, dense);
    return c.off;
}

clsa_status from_hip(hipError_t e) { return e == hipSuccess ? CLSA_OK : CLSA_ERR_HIP; }

}  // namespace

extern "C" {

size_t clsa_workspace_bytes(const clsa_shape *shape, int32_t op, int32_t n_layers) {
    Geometry g;
    switch (op) {
        case CLSA_OP_INDEX:
            return 0;
        case CLSA_OP_TOPK:
            if (check_shape(shape, kTopk, &g) != CLSA_OK) return 0;
            return topk_ws_bytes(g);
        case CLSA_OP_ATTN:
            if (check_shape(shape, kAttn, &g) != CLSA_OK) return 0;
            return attn_ws_bytes(g);
        case CLSA_OP_DENSE:
            if (check_shape(shape, kAttn | kDense, &g) != CLSA_OK) return 0;
            return attn_ws_bytes(g, true);
        case CLSA_OP_KD_TARGET:
            if (check_shape(shape, kAttn, &g) != CLSA_OK || n_layers < 1 ||
                !clsa::kd_target_supported(g, n_layers))
                return 0;
            return align_up(sizeof(float) * clsa::kd_target_ws_floats(g, n_layers));
        case CLSA_OP_KD_LOSS:
            if (check_shape(shape, kIndex | kDense, &g) != CLSA_OK || !clsa::kd_loss_supported(g))
                return 0;
            return align_up(sizeof(float) * clsa::kd_loss_ws_floats(g));
        case CLSA_OP_DECODE: {
            // layers run one after another and reuse the same buffers
            if (check_shape(shape, kIndex | kTopk | kAttn, &g) != CLSA_OK || n_layers < 0)
                return 0;
            DecodeWs w;
            return carve_decode(g, nullptr, w);
        }
        default:
            return 0;
    }
}

clsa_status clsa_index_scores(const clsa_shape *shape, const void *q_idx, const void *k_idx,
                              const int32_t *page_table, const int32_t *seq_lens,
                              const int32_t *q_pos, float *scores, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kIndex, &g));
    CLSA_TRY(check_ptr(q_idx, 16));
    CLSA_TRY(check_ptr(k_idx, 16));
    CLSA_TRY(check_ptr(seq_lens, 4));
    CLSA_TRY(check_ptr(scores, 4));
    CLSA_TRY(check_common(shape, page_table, q_pos, true, true));
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (clsa::index_uses_mfma(g))
        return from_hip(clsa::launch_index_prefill(g, q_idx, k_idx, page_table, seq_lens, q_pos,
                                                   scores, nullptr, st));
    return from_hip(clsa::launch_index_scores(g, q_idx, k_idx, page_table, seq_lens, q_pos, scores,
                                              nullptr, nullptr, st));
}

clsa_status clsa_topk(const clsa_shape *shape, const float *scores, const int32_t *seq_lens,
                      const int32_t *q_pos, int32_t *idx, int32_t *n_sel, void *ws,
                      size_t ws_bytes, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kTopk, &g));
    CLSA_TRY(check_ptr(scores, 4));
    CLSA_TRY(check_ptr(seq_lens, 4));
    CLSA_TRY(check_ptr(idx, 4));
    CLSA_TRY(check_ptr(n_sel, 4));
    CLSA_TRY(check_common(shape, nullptr, q_pos, true, false));
    const size_t need = topk_ws_bytes(g);
    if (need && (!ws || ws_bytes < need || !aligned(ws, kAlign))) return CLSA_ERR_WORKSPACE;
    CLSA_TRY(check_topk_lds(g));
    Carver c{static_cast<char *>(ws)};
    TopkWs t;
    carve_topk(g, c, t);
    hipStream_t st = static_cast<hipStream_t>(stream);
    CLSA_TRY(from_hip(clsa::launch_zero_u32(t.zero, t.zero_count, st)));
    return from_hip(clsa::launch_topk(g, scores, seq_lens, q_pos, t.buf, false, idx, n_sel, st));
}

clsa_status clsa_sparse_attn(const clsa_shape *shape, const void *q, const void *k_cache,
                             const void *v_cache, const int32_t *page_table, const int32_t *idx,
                             const int32_t *n_sel, void *out, float *lse, void *ws,
                             size_t ws_bytes, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kAttn, &g));
    CLSA_TRY(check_ptr(q, 16));
    CLSA_TRY(check_ptr(k_cache, 16));
    CLSA_TRY(check_ptr(v_cache, 16));
    CLSA_TRY(check_ptr(idx, 4));
    CLSA_TRY(check_ptr(n_sel, 4));
    CLSA_TRY(check_ptr(out, 16));
    if (lse) CLSA_TRY(check_ptr(lse, 4));
    CLSA_TRY(check_common(shape, page_table, nullptr, false, true));
    const size_t need = attn_ws_bytes(g);
    if (need && (!ws || ws_bytes < need || !aligned(ws, kAlign))) return CLSA_ERR_WORKSPACE;
    Carver c{static_cast<char *>(ws)};
    AttnWs w;
    carve_attn(g, c, w);
    return from_hip(clsa::launch_sparse_attn(g, q, k_cache, v_cache, page_table, idx, n_sel, out,
                                             lse, w.partials, nullptr,
                                             static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

// One index pass + one top-k per group of `group` layers, then the group's
// layer passes; group >= n_layers is the shared-routing step.
clsa_status decode_step_impl(const clsa_shape *shape, const void *q_idx, int64_t q_idx_stride,
                             const void *k_idx, int64_t k_idx_stride, const void *k_cache,
                             const void *v_cache, const int32_t *page_table,
                             const int32_t *seq_lens, const int32_t *q_pos, int32_t n_layers,
                             int32_t group, const void *q_layers, void *out_layers,
                             float *lse_layers, int32_t *idx, int32_t *n_sel, void *ws,
                             size_t ws_bytes, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kIndex | kTopk | kAttn, &g));
    if (n_layers < 0 || group < 1 || q_idx_stride < 0 || k_idx_stride < 0)
        return CLSA_ERR_INVALID_ARG;
    if (q_idx_stride % 8 || k_idx_stride % 8) return CLSA_ERR_INVALID_ARG;  // 16-byte aligned sets
    CLSA_TRY(check_ptr(q_idx, 16));
    CLSA_TRY(check_ptr(k_idx, 16));
    CLSA_TRY(check_ptr(seq_lens, 4));
    CLSA_TRY(check_ptr(idx, 4));
    CLSA_TRY(check_ptr(n_sel, 4));
    if (n_layers > 0) {
        CLSA_TRY(check_ptr(k_cache, 16));
        CLSA_TRY(check_ptr(v_cache, 16));
        CLSA_TRY(check_ptr(q_layers, 16));
        CLSA_TRY(check_ptr(out_layers, 16));
        if (lse_layers) CLSA_TRY(check_ptr(lse_layers, 4));
    }
    CLSA_TRY(check_common(shape, page_table, q_pos, true, true));
    DecodeWs w;
    const size_t need = carve_decode(g, nullptr, w);
    if (!ws || ws_bytes < need || !aligned(ws, kAlign)) return CLSA_ERR_WORKSPACE;
    CLSA_TRY(check_topk_lds(g));

    carve_decode(g, ws, w);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool hook = t_hook.on;
    // Many query rows per sequence (chunked prefill): scores on the matrix cores,
    // without the coarse histogram, which the top-k then makes itself.  The
    // histogram needs clearing unless that top-k is the per-row one.
    const bool mfma = clsa::index_uses_mfma(g);
    // Many causal rows with a moderate k: the scores are never written; a
    // sampled pass sets each row's candidate threshold and a second pass
    // emits the candidates (see topk.hip).
    const bool two_pass = clsa::topk_uses_two_pass(g);
    const size_t q_stride = (size_t)g.rows * g.q_heads * 128;  // bf16 elements per layer
    const size_t lse_stride = (size_t)g.rows * g.q_heads;
    const size_t set_stride = (size_t)g.rows * g.top_k;         // index entries per set
    const int n_sets = n_layers > 0 ? (n_layers + group - 1) / group : 1;
    for (int s = 0; s < n_sets; ++s) {
        const uint16_t *qi = static_cast<const uint16_t *>(q_idx) + (size_t)s * q_idx_stride;
        const uint16_t *ki = static_cast<const uint16_t *>(k_idx) + (size_t)s * k_idx_stride;
        int32_t *is = idx + (size_t)s * set_stride;
        int32_t *ns = n_sel + (size_t)s * g.rows;
        const bool first = s == 0;
        if (two_pass) {
            if (first && hook && hipEventRecord(t_hook.ev[0], st) != hipSuccess) return CLSA_ERR_HIP;
            CLSA_TRY(from_hip(clsa::launch_index_prefill_sample(g, qi, ki, page_table, seq_lens,
                                                                q_pos, w.samples, w.tickets, st)));
            CLSA_TRY(from_hip(clsa::launch_topk_sample_thresh(g, w.samples, seq_lens, q_pos,
                                                              w.thresh, w.slow, st)));
            CLSA_TRY(from_hip(clsa::launch_index_prefill_emit(g, qi, ki, page_table, seq_lens,
                                                              q_pos, w.thresh, w.cand_count,
                                                              w.cands, st)));
            if (first && hook && hipEventRecord(t_hook.ev[1], st) != hipSuccess) return CLSA_ERR_HIP;
            CLSA_TRY(from_hip(clsa::launch_topk_cands(g, w.cand_count, w.cands, seq_lens, q_pos,
                                                      qi, ki, page_table, w.scores, w.slow, is, ns,
                                                      st)));
        } else {
            // the decode indexer makes the coarse histogram except for short rows,
            // whose per-row top-k makes its own in LDS
            const bool idx_hist = !mfma && !clsa::topk_small_rows(g);
            if (idx_hist || clsa::topk_uses_wide(g))
                CLSA_TRY(from_hip(clsa::launch_zero_u32(w.zero, w.zero_count, st)));
            if (first && hook && hipEventRecord(t_hook.ev[0], st) != hipSuccess) return CLSA_ERR_HIP;
            if (mfma)
                CLSA_TRY(from_hip(clsa::launch_index_prefill(g, qi, ki, page_table, seq_lens,
                                                             q_pos, w.scores, w.tickets, st)));
            else
                CLSA_TRY(from_hip(clsa::launch_index_scores(g, qi, ki, page_table, seq_lens, q_pos,
                                                            w.scores, idx_hist ? w.topk.hist : nullptr,
                                                            w.tickets, st)));
            if (first && hook && hipEventRecord(t_hook.ev[1], st) != hipSuccess) return CLSA_ERR_HIP;
            CLSA_TRY(from_hip(clsa::launch_topk(g, w.scores, seq_lens, q_pos, w.topk, idx_hist, is,
                                                ns, st)));
        }
        if (first && hook && hipEventRecord(t_hook.ev[2], st) != hipSuccess) return CLSA_ERR_HIP;
        const int l_end = n_layers < (s + 1) * group ? n_layers : (s + 1) * group;
        for (int l = s * group; l < l_end; ++l) {
            const uint16_t *ql = static_cast<const uint16_t *>(q_layers) + l * q_stride;
            uint16_t *ol = static_cast<uint16_t *>(out_layers) + l * q_stride;
            float *lsel = lse_layers ? lse_layers + l * lse_stride : nullptr;
            const bool mark = hook && l < t_hook.layers;
            if (mark && hipEventRecord(t_hook.ev[4 + 2 * l], st) != hipSuccess)
                return CLSA_ERR_HIP;
            CLSA_TRY(from_hip(clsa::launch_sparse_attn(g, ql, k_cache, v_cache, page_table, is,
                                                       ns, ol, lsel, w.partials, w.tickets, st,
                                                       mark ? t_hook.ev[5 + 2 * l] : nullptr)));
        }
    }
    if (hook && hipEventRecord(t_hook.ev[3], st) != hipSuccess) return CLSA_ERR_HIP;
    return CLSA_OK;
}

}  // namespace

extern "C" {

clsa_status clsa_decode_step(const clsa_shape *shape, const void *q_idx, const void *k_idx,
                             const void *k_cache, const void *v_cache,
                             const int32_t *page_table, const int32_t *seq_lens,
                             const int32_t *q_pos, int32_t n_layers, const void *q_layers,
                             void *out_layers, float *lse_layers, int32_t *idx, int32_t *n_sel,
                             void *ws, size_t ws_bytes, void *stream) {
    const int32_t group = n_layers > 0 ? n_layers : 1;
    return decode_step_impl(shape, q_idx, 0, k_idx, 0, k_cache, v_cache, page_table, seq_lens,
                            q_pos, n_layers, group, q_layers, out_layers, lse_layers, idx, n_sel,
                            ws, ws_bytes, stream);
}

clsa_status clsa_decode_step_noalloc(const clsa_shape *shape, const void *q_idx,
                                     const void *k_idx, const void *k_cache, const void *v_cache,
                                     const int32_t *page_table, const int32_t *seq_lens,
                                     const int32_t *q_pos, int32_t n_layers, const void *q_layers,
                                     void *out_layers, float *lse_layers, int32_t *idx,
                                     int32_t *n_sel, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kIndex | kTopk | kAttn, &g));
    DecodeWs w;
    if (carve_decode(g, nullptr, w) > clsa::kNoallocScratchBytes) return CLSA_ERR_SCRATCH_LIMIT;
    void *scratch = nullptr;
    CLSA_TRY(from_hip(clsa::noalloc_scratch(&scratch)));
    const int32_t group = n_layers > 0 ? n_layers : 1;
    return decode_step_impl(shape, q_idx, 0, k_idx, 0, k_cache, v_cache, page_table, seq_lens,
                            q_pos, n_layers, group, q_layers, out_layers, lse_layers, idx, n_sel,
                            scratch, clsa::kNoallocScratchBytes, stream);
}

clsa_status clsa_decode_step_grouped(const clsa_shape *shape, const void *q_idx,
                                     int64_t q_idx_group_stride, const void *k_idx,
                                     int64_t k_idx_group_stride, const void *k_cache,
                                     const void *v_cache, const int32_t *page_table,
                                     const int32_t *seq_lens, const int32_t *q_pos,
                                     int32_t n_layers, int32_t group, const void *q_layers,
                                     void *out_layers, float *lse_layers, int32_t *idx,
                                     int32_t *n_sel, void *ws, size_t ws_bytes, void *stream) {
    return decode_step_impl(shape, q_idx, q_idx_group_stride, k_idx, k_idx_group_stride, k_cache,
                            v_cache, page_table, seq_lens, q_pos, n_layers, group, q_layers,
                            out_layers, lse_layers, idx, n_sel, ws, ws_bytes, stream);
}

clsa_status clsa_project_append(const clsa_shape *shape, int32_t d_model, const void *h,
                                const void *w, const int32_t *pos, const int32_t *page_table,
                                void *q_idx, void *k_idx, void *k_cache, void *v_cache,
                                void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kIndex | kAttn, &g));
    if (d_model < 1) return CLSA_ERR_INVALID_ARG;
    if (!clsa::project_supported(d_model)) return CLSA_ERR_UNSUPPORTED;
    CLSA_TRY(check_ptr(h, 16));
    CLSA_TRY(check_ptr(w, 16));
    CLSA_TRY(check_ptr(pos, 4));
    CLSA_TRY(check_ptr(q_idx, 16));
    CLSA_TRY(check_ptr(k_idx, 16));
    CLSA_TRY(check_ptr(k_cache, 16));
    CLSA_TRY(check_ptr(v_cache, 16));
    CLSA_TRY(check_common(shape, page_table, nullptr, false, true));
    return from_hip(clsa::launch_project(g, d_model, h, w, pos, page_table, q_idx, k_idx, k_cache,
                                         v_cache, static_cast<hipStream_t>(stream)));
}

clsa_status clsa_dense_attn(const clsa_shape *shape, const void *q, const void *k_cache,
                            const void *v_cache, const int32_t *page_table,
                            const int32_t *seq_lens, const int32_t *q_pos, void *out, float *lse,
                            void *ws, size_t ws_bytes, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kAttn | kDense, &g));
    CLSA_TRY(check_ptr(q, 16));
    CLSA_TRY(check_ptr(k_cache, 16));
    CLSA_TRY(check_ptr(v_cache, 16));
    CLSA_TRY(check_ptr(seq_lens, 4));
    CLSA_TRY(check_ptr(out, 16));
    if (lse) CLSA_TRY(check_ptr(lse, 4));
    CLSA_TRY(check_common(shape, page_table, q_pos, true, true));
    const size_t need = attn_ws_bytes(g, true);
    if (need && (!ws || ws_bytes < need || !aligned(ws, kAlign))) return CLSA_ERR_WORKSPACE;
    Carver c{static_cast<char *>(ws)};
    AttnWs w;
    carve_attn(g, c, w, true);
    return from_hip(clsa::launch_dense_attn(g, q, k_cache, v_cache, page_table, seq_lens, q_pos,
                                            out, lse, w.partials,
                                            static_cast<hipStream_t>(stream)));
}

clsa_status clsa_kd_target(const clsa_shape *shape, int32_t n_layers, const void *q_layers,
                           const void *k_cache, const int32_t *page_table,
                           const int32_t *seq_lens, const int32_t *q_pos,
                           const float *lse_layers, float *abar, void *ws, size_t ws_bytes,
                           void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kAttn, &g));
    if (n_layers < 1 || !(shape->softmax_scale > 0.0f)) return CLSA_ERR_INVALID_ARG;
    if (!clsa::kd_target_supported(g, n_layers)) return CLSA_ERR_UNSUPPORTED;
    CLSA_TRY(check_ptr(q_layers, 16));
    CLSA_TRY(check_ptr(k_cache, 16));
    CLSA_TRY(check_ptr(seq_lens, 4));
    CLSA_TRY(check_ptr(abar, 4));
    if (lse_layers) CLSA_TRY(check_ptr(lse_layers, 4));
    CLSA_TRY(check_common(shape, page_table, q_pos, true, true));
    const size_t need = align_up(sizeof(float) * clsa::kd_target_ws_floats(g, n_layers));
    if (!ws || ws_bytes < need || !aligned(ws, kAlign)) return CLSA_ERR_WORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool hook = t_hook.on;
    if (hook && hipEventRecord(t_hook.ev[0], st) != hipSuccess) return CLSA_ERR_HIP;
    CLSA_TRY(from_hip(clsa::launch_kd_target(g, n_layers, q_layers, k_cache, page_table,
                                             seq_lens, q_pos, lse_layers, abar,
                                             static_cast<float *>(ws), st,
                                             hook ? t_hook.ev[1] : nullptr)));
    if (hook && hipEventRecord(t_hook.ev[2], st) != hipSuccess) return CLSA_ERR_HIP;
    return CLSA_OK;
}

clsa_status clsa_kd_loss(const clsa_shape *shape, const float *abar, const void *q_idx,
                         const void *k_idx, const int32_t *page_table, const int32_t *seq_lens,
                         const int32_t *q_pos, float *loss, float *dq_idx, float *dk_idx,
                         void *ws, size_t ws_bytes, void *stream) {
    Geometry g;
    CLSA_TRY(check_shape(shape, kIndex | kDense, &g));
    if (!clsa::kd_loss_supported(g)) return CLSA_ERR_UNSUPPORTED;
    CLSA_TRY(check_ptr(abar, 4));
    CLSA_TRY(check_ptr(q_idx, 16));
    CLSA_TRY(check_ptr(k_idx, 16));
    CLSA_TRY(check_ptr(seq_lens, 4));
    CLSA_TRY(check_ptr(loss, 4));
    CLSA_TRY(check_ptr(dq_idx, 16));
    CLSA_TRY(check_ptr(dk_idx, 16));
    CLSA_TRY(check_common(shape, page_table, q_pos, true, true));
    const size_t need = align_up(sizeof(float) * clsa::kd_loss_ws_floats(g));
    if (!ws || ws_bytes < need || !aligned(ws, kAlign)) return CLSA_ERR_WORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool hook = t_hook.on;
    if (hook && hipEventRecord(t_hook.ev[0], st) != hipSuccess) return CLSA_ERR_HIP;
    CLSA_TRY(from_hip(clsa::launch_kd_loss(g, abar, q_idx, k_idx, page_table, seq_lens, q_pos,
                                           loss, dq_idx, dk_idx, static_cast<float *>(ws), st,
                                           hook ? t_hook.ev[1] : nullptr,
                                           hook ? t_hook.ev[2] : nullptr)));
    if (hook && hipEventRecord(t_hook.ev[3], st) != hipSuccess) return CLSA_ERR_HIP;
    return CLSA_OK;
}

const char *clsa_status_string(clsa_status status) {
    switch (status) {
        case CLSA_OK: return "CLSA_OK";
        case CLSA_ERR_INVALID_ARG: return "CLSA_ERR_INVALID_ARG";
        case CLSA_ERR_UNSUPPORTED: return "CLSA_ERR_UNSUPPORTED";
        case CLSA_ERR_WORKSPACE: return "CLSA_ERR_WORKSPACE";
        case CLSA_ERR_HIP: return "CLSA_ERR_HIP";
        case CLSA_ERR_SCRATCH_LIMIT: return "CLSA_ERR_SCRATCH_LIMIT";
    }
    return "CLSA_ERR_UNKNOWN";
}

clsa_status clsa_get_device_error(uint32_t *bits) {
    if (!bits) return CLSA_ERR_INVALID_ARG;
    *bits = 0;
    if (hipDeviceSynchronize() != hipSuccess) return CLSA_ERR_HIP;
    uint32_t v = 0;
    CLSA_TRY(from_hip(clsa::take_device_error_index_decode(&v)));
    CLSA_TRY(from_hip(clsa::take_device_error_index_prefill(&v)));
    CLSA_TRY(from_hip(clsa::take_device_error_topk(&v)));
    CLSA_TRY(from_hip(clsa::take_device_error_sparse_attn(&v)));
    CLSA_TRY(from_hip(clsa::take_device_error_kd(&v)));
    *bits = v;
    return CLSA_OK;
}

clsa_status clsa_set_phase_events(void *const *events, int32_t n) {
    if (n == 0) {
        t_hook.on = false;
        return CLSA_OK;
    }
    if (n < 4 || n > 4 + 2 * kHookLayers || (n & 1) || !events) return CLSA_ERR_INVALID_ARG;
    for (int i = 0; i < n; ++i)
        if (!events[i]) return CLSA_ERR_INVALID_ARG;
    for (int i = 0; i < n; ++i) t_hook.ev[i] = static_cast<hipEvent_t>(events[i]);
    t_hook.layers = (n - 4) / 2;
    t_hook.on = true;
    return CLSA_OK;
}

}  // extern "C"
