// Sparse GQA attention over the shared index set (Section 2.1, Eq. 4:
// O_t = Attn(Q_t, K_{S_t}, V_{S_t}); softmax attention as in Eq. 1; no
// positional encoding on this path).
//
// One workgroup (4 waves) = one (query row, KV head g, split of S).  A split is
// a run of 64-token chunks of the row's index list.  Per chunk:
//   * each 16-lane quarter-wave gathers one selected token's 256-byte K row and
//     256-byte V row of head g (16 bytes per lane), 4 chunks-rounds x 4 waves x
//     4 quarters = 64 tokens, all loads issued before any math;
//   * the G query heads of the GQA group share those rows: each lane dots its
//     8 key values with the matching 8 values of every head (v_dot2_f32_bf16),
//     a transpose-reduction over the 16 lanes leaves one (head, token) logit
//     per lane, and the logits go to LDS;
//   * one wave per head takes the chunk maximum and sum (base-2 exponentials),
//     updates the running max / denominator and rescales its accumulators
//     (online softmax), so a split of any length needs one pass;
//   * each lane accumulates weight x V for its 8 dimensions and G heads.
// At the end the accumulators are reduced over lanes and waves in LDS.  With
// one split the workgroup writes the bf16 output and lse itself; otherwise it
// writes fp32 partials (o, m, l) and a merge kernel combines the splits with
// the exact log-sum-exp rule.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

constexpr int kHeadDim = 128;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct AttnArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    const int32_t *page_table;
    const int32_t *idx;
    const int32_t *n_sel;
    uint16_t *out;      // direct output (splits == 1)
    float *lse;         // direct lse (splits == 1), may be null
    float *part_o;      // [rows, Hq, splits, 128]
    float *part_ml;     // [rows, Hq, splits, 2]
    int n_q, max_len, page_shift, max_pages, top_k, kv_heads, q_heads, splits, chunks_per_split;
    float scale_log2;   // softmax_scale * log2(e)
};

__host__ __device__ constexpr int pow2_at_least(int x) {
    return x <= 1 ? 1 : 2 * pow2_at_least((x + 1) / 2);
}

template <int G>
__global__ __launch_bounds__(256) void sparse_attn_kernel(AttnArgs a) {
    constexpr int NV = pow2_at_least(4 * G);   // logits per lane before the reduction
    constexpr int NO = pow2_at_least(8 * G);   // accumulators per lane before the reduction
    __shared__ float zs[G][64];                // logits -> weights of the current chunk
    __shared__ float s_scale[G];               // per-head rescale factor of this chunk
    __shared__ float s_ml[G][2];               // running max (log2 domain) and denominator
    __shared__ float red[4][G * kHeadDim];     // cross-wave reduction of the accumulators

    // flattened grid: ((row * kv_heads) + g) * splits + split
    const int split = blockIdx.x % a.splits;
    const int rg = blockIdx.x / a.splits;
    const int g = rg % a.kv_heads, row = rg / a.kv_heads;
    const int b = row / a.n_q;
    const int n = min(max(a.n_sel[row], 0), a.top_k);
    const int tok_begin = split * a.chunks_per_split * 64;
    const int Hq = a.kv_heads * G;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int qq = lane >> 4, sub = lane & 15;
    if (tok_begin >= n && !(split == 0 && a.splits == 1)) return;  // uniform
    const int tok_end = min(n, tok_begin + a.chunks_per_split * 64);
    const int row_elems = a.kv_heads * kHeadDim;

    uint4 qv[G];
#pragma unroll
    for (int h = 0; h < G; ++h)
        qv[h] = *reinterpret_cast<const uint4 *>(a.q + ((size_t)row * Hq + g * G + h) * kHeadDim +
                                                 sub * 8);
    if (tid < G) {
        s_ml[tid][0] = -INFINITY;
        s_ml[tid][1] = 0.0f;
    }
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int d = 0; d < 8; ++d) acc[h][d] = 0.0f;

    const int32_t *sel = a.idx + (size_t)row * a.top_k;
    for (int c0 = tok_begin; c0 < tok_end; c0 += 64) {
        uint4 kr[4], vr[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t = c0 + i * 16 + wave * 4 + qq;
            if (t < tok_end) {
                const int j = min(max(sel[t], 0), a.max_len - 1);
                const size_t off = token_offset(a.page_table, a.page_shift, a.max_pages,
                                                a.max_len, b, j, row_elems) +
                                   (size_t)g * kHeadDim + sub * 8;
                kr[i] = *reinterpret_cast<const uint4 *>(a.k + off);
                vr[i] = *reinterpret_cast<const uint4 *>(a.v + off);
            } else {
                kr[i] = make_uint4(0u, 0u, 0u, 0u);
                vr[i] = make_uint4(0u, 0u, 0u, 0u);
            }
        }
        // logits: value index i*G + h, transpose-reduced over the 16 lanes of the quarter
        float p[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) p[v] = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int h = 0; h < G; ++h) p[i * G + h] = dot8_bf16(kr[i], qv[h], 0.0f);
        {
            int cnt = NV;
#pragma unroll
            for (int m = 8; m >= 1; m >>= 1) {
                if (cnt > 1) {
                    const int hlf = cnt / 2;
                    const bool up = sub & m;
#pragma unroll
                    for (int v = 0; v < NV / 2; ++v) {
                        if (v < hlf) {
                            const float keep = up ? p[v + hlf] : p[v];
                            const float send = up ? p[v] : p[v + hlf];
                            p[v] = keep + __shfl_xor(send, m);
                        }
                    }
                    cnt = hlf;
                } else {
                    p[0] += __shfl_xor(p[0], m);
                }
            }
        }
        // lane `sub` now holds value indices [sub*NV/16, sub*NV/16 + NV/16) (NV >= 16)
        // or index sub / (16/NV) (NV < 16).
        constexpr int PER = NV >= 16 ? NV / 16 : 1;
#pragma unroll
        for (int v = 0; v < PER; ++v) {
            const int orig = NV >= 16 ? sub * PER + v : sub / (16 / NV);
            if (orig < 4 * G) {
                const int i = orig / G, h = orig - i * G;
                const int tl = i * 16 + wave * 4 + qq;
                const bool ok = c0 + tl < tok_end;
                zs[h][tl] = ok ? p[v] * a.scale_log2 : -INFINITY;
            }
        }
        __syncthreads();
        // per-head chunk statistics and online-softmax update
        for (int h = wave; h < G; h += 4) {
            const float z = zs[h][lane];
            float mx = z;
#pragma unroll
            for (int m = 32; m >= 1; m >>= 1) mx = fmaxf(mx, __shfl_xor(mx, m));
            const float m_old = s_ml[h][0];
            const float m_new = fmaxf(m_old, mx);
            const float w = exp2f(z - m_new);   // z = -inf -> 0
            float sum = w;
#pragma unroll
            for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m);
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
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int tl = i * 16 + wave * 4 + qq;
            float vf[8];
            vf[0] = bf16_lo(vr[i].x); vf[1] = bf16_hi(vr[i].x);
            vf[2] = bf16_lo(vr[i].y); vf[3] = bf16_hi(vr[i].y);
            vf[4] = bf16_lo(vr[i].z); vf[5] = bf16_hi(vr[i].z);
            vf[6] = bf16_lo(vr[i].w); vf[7] = bf16_hi(vr[i].w);
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float w = zs[h][tl];
#pragma unroll
                for (int d = 0; d < 8; ++d) acc[h][d] = fmaf(w, vf[d], acc[h][d]);
            }
        }
        __syncthreads();  // zs / s_scale are rewritten by the next chunk
    }

    // ---- reduce the accumulators over the 4 quarters of each wave (lanes ^16, ^32) ----
    float o[NO];
#pragma unroll
    for (int v = 0; v < NO; ++v) o[v] = 0.0f;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int d = 0; d < 8; ++d) o[h * 8 + d] = acc[h][d];
    {
        int cnt = NO;
#pragma unroll
        for (int m = 32; m >= 16; m >>= 1) {
            const int hlf = cnt / 2;
            const bool up = lane & m;
#pragma unroll
            for (int v = 0; v < NO / 2; ++v) {
                if (v < hlf) {
                    const float keep = up ? o[v + hlf] : o[v];
                    const float send = up ? o[v] : o[v + hlf];
                    o[v] = keep + __shfl_xor(send, m);
                }
            }
            cnt = hlf;
        }
    }
    // lane (qq, sub) holds value indices [qq*NO/4, qq*NO/4 + NO/4); index = h*8 + d
#pragma unroll
    for (int v = 0; v < NO / 4; ++v) {
        const int orig = qq * (NO / 4) + v;
        if (orig < 8 * G) {
            const int h = orig >> 3, d = orig & 7;
            red[wave][h * kHeadDim + sub * 8 + d] = o[v];
        }
    }
    __syncthreads();
    for (int e = tid; e < G * kHeadDim; e += 256) {
        const int h = e / kHeadDim, dim = e - h * kHeadDim;
        const float sum = red[0][e] + red[1][e] + red[2][e] + red[3][e];
        const int hq = g * G + h;
        if (a.splits == 1) {
            const float l = s_ml[h][1];
            const float val = l > 0.0f ? sum / l : 0.0f;
            a.out[((size_t)row * Hq + hq) * kHeadDim + dim] = (uint16_t)f32_to_bf16_bits(val);
            if (a.lse && dim == 0)
                a.lse[(size_t)row * Hq + hq] = l > 0.0f ? (s_ml[h][0] + log2f(l)) * kLn2 : -INFINITY;
        } else {
            const size_t slot = ((size_t)row * Hq + hq) * a.splits + split;
            a.part_o[slot * kHeadDim + dim] = sum;
            if (dim == 0) {
                a.part_ml[slot * 2] = s_ml[h][0];
                a.part_ml[slot * 2 + 1] = s_ml[h][1];
            }
        }
    }
}

// Combine the splits of one (row, query head): one wave, two dimensions per lane.
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a, int rows) {
    const int Hq = a.q_heads;
    const int unit = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (unit >= rows * Hq) return;
    const int lane = threadIdx.x & 63;
    const int row = unit / Hq, hq = unit - row * Hq;
    const int n = min(max(a.n_sel[row], 0), a.top_k);
    const int nsplit = min(a.splits, div_up(n, a.chunks_per_split * 64));
    const size_t base = ((size_t)row * Hq + hq) * a.splits;
    float mx = -INFINITY;
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, a.part_ml[(base + s) * 2]);
    float l = 0.0f, o0 = 0.0f, o1 = 0.0f;
    for (int s = 0; s < nsplit; ++s) {
        const float w = exp2f(a.part_ml[(base + s) * 2] - mx);
        l += w * a.part_ml[(base + s) * 2 + 1];
        const float2 po = *reinterpret_cast<const float2 *>(a.part_o + (base + s) * kHeadDim + lane * 2);
        o0 = fmaf(w, po.x, o0);
        o1 = fmaf(w, po.y, o1);
    }
    const float inv = l > 0.0f ? 1.0f / l : 0.0f;
    const uint32_t packed = f32_to_bf16_bits(o0 * inv) | (f32_to_bf16_bits(o1 * inv) << 16);
    *reinterpret_cast<uint32_t *>(a.out + ((size_t)row * Hq + hq) * kHeadDim + lane * 2) = packed;
    if (a.lse && lane == 0)
        a.lse[(size_t)row * Hq + hq] = l > 0.0f ? (mx + log2f(l)) * kLn2 : -INFINITY;
}

// Splits per (row, KV head): enough workgroups to cover the chip, at least one
// 64-token chunk each.
static void plan_splits(const Geometry &g, int &splits, int &chunks_per_split) {
    const int chunks = div_up(g.top_k, 64);
    const long units = (long)g.rows * g.kv_heads;
    long want = units > 0 ? (2048 + units - 1) / units : 1;
    if (want < 1) want = 1;
    if (want > chunks) want = chunks;
    chunks_per_split = div_up(chunks, (int)want);
    splits = div_up(chunks, chunks_per_split);
}

size_t attn_partial_floats(const Geometry &g) {
    int splits, cps;
    plan_splits(g, splits, cps);
    if (splits == 1) return 0;
    return (size_t)g.rows * g.q_heads * splits * (kHeadDim + 2);
}

template <int G>
static void launch_attn_g(const AttnArgs &a, dim3 grid, hipStream_t stream) {
    sparse_attn_kernel<G><<<grid, dim3(256), 0, stream>>>(a);
}

hipError_t launch_sparse_attn(const Geometry &g, const void *q, const void *k_cache,
                              const void *v_cache, const int32_t *page_table,
                              const int32_t *idx, const int32_t *n_sel, void *out, float *lse,
                              float *partials, hipStream_t stream) {
    AttnArgs a;
    a.q = static_cast<const uint16_t *>(q);
    a.k = static_cast<const uint16_t *>(k_cache);
    a.v = static_cast<const uint16_t *>(v_cache);
    a.page_table = page_table;
    a.idx = idx;
    a.n_sel = n_sel;
    a.out = static_cast<uint16_t *>(out);
    a.lse = lse;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.top_k = g.top_k;
    a.kv_heads = g.kv_heads;
    a.q_heads = g.q_heads;
    plan_splits(g, a.splits, a.chunks_per_split);
    a.scale_log2 = g.softmax_scale * kLog2e;
    const size_t part_o = (size_t)g.rows * g.q_heads * a.splits * kHeadDim;
    a.part_o = a.splits > 1 ? partials : nullptr;
    a.part_ml = a.splits > 1 ? partials + part_o : nullptr;
    if (g.rows == 0) return hipSuccess;
    const size_t blocks = (size_t)g.rows * g.kv_heads * a.splits;
    if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)blocks);
    switch (g.group) {
        case 1: launch_attn_g<1>(a, grid, stream); break;
        case 2: launch_attn_g<2>(a, grid, stream); break;
        case 4: launch_attn_g<4>(a, grid, stream); break;
        case 5: launch_attn_g<5>(a, grid, stream); break;
        case 8: launch_attn_g<8>(a, grid, stream); break;
        default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.splits == 1) return e;
    const int units = g.rows * g.q_heads;
    attn_merge_kernel<<<dim3(div_up(units, 4)), dim3(256), 0, stream>>>(a, g.rows);
    return hipGetLastError();
}

}  // namespace clsa
