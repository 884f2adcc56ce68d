// Eq. 2 for the new tokens of a step (Q_idx = H W_idx^Q, K_idx = H W_idx^K),
// together with the shared key and value of the same hidden states
// (K = H W^K, V = H W^V), fused with the cache write: the index query goes to
// its own buffer, the index key, key and value rows are written into the
// caches at each token's position.  One matrix product over the stacked
// weights [256 + 256 + 2 * kv_heads * 128, d_model] (each output feature's
// weight vector contiguous), bf16 inputs, fp32 accumulation, bf16 results
// rounded to nearest even.
//
// MFMA mapping (v_mfma_f32_16x16x32_bf16): A = 16 rows of h x 32 dims,
// B = 32 dims x 16 output features; lane l supplies row / feature (l & 15) for
// dims (l >> 4) * 8 .. +8 of each 32-dim step and receives C rows
// 4 * (l >> 4) + r (r = 0..3) of feature (l & 15).  A wave owns 16 rows x 64
// features (four feature tiles).
//   * few rows (decode): a workgroup of 8 waves splits d_model eight ways for
//     one 16-row x 16-feature tile, each wave issuing all of its loads before
//     its first product, and the eight partial tiles are added in LDS: the
//     weights (13 MB at d_model 2560, the bytes that bound this case) are then
//     read by 160 workgroups at once;
//   * many rows (prefill): four waves per workgroup on four row tiles of the
//     same 64 features (their weight loads meet in L1), each over all of
//     d_model with the next step's loads issued before the current products.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kProjFeat = 64;      // output features per wave tile
constexpr int kSplitWaves = 8;     // d_model split of the few-rows kernel
constexpr int kSplitMaxD = 3072;   // largest d_model of the few-rows kernel (register budget)

struct ProjArgs {
    const uint16_t *h;         // [rows, d]
    const uint16_t *w;         // [n_feat, d]
    const int32_t *pos;        // [rows]
    const int32_t *page_table;
    uint16_t *q_idx;           // [rows, 256]
    uint16_t *k_idx;           // index-key cache
    uint16_t *k_cache, *v_cache;
    int rows, d, n_q, max_len, page_shift, max_pages, kvw;  // kvw = kv_heads * 128
};

__device__ __forceinline__ bf16x8 ld8(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// Writes output feature f of row r (rows past the end are dropped; cache rows
// only for positions inside [0, max_len)).
template <bool PAGED>
__device__ __forceinline__ void store_feature(const ProjArgs &a, int r, int f, float v) {
    if (r >= a.rows) return;
    const uint16_t bits = (uint16_t)f32_to_bf16_bits(v);
    if (f < 256) {
        a.q_idx[(size_t)r * 256 + f] = bits;
        return;
    }
    const int p = a.pos[r];
    if (p < 0 || p >= a.max_len) return;
    const int b = r / a.n_q;
    size_t row;
    if (PAGED) {
        const int page = a.page_table[(size_t)b * a.max_pages + (p >> a.page_shift)];
        row = ((size_t)page << a.page_shift) + (p & ((1 << a.page_shift) - 1));
    } else {
        row = (size_t)b * a.max_len + p;
    }
    if (f < 512) a.k_idx[row * 256 + (f - 256)] = bits;
    else if (f < 512 + a.kvw) a.k_cache[row * a.kvw + (f - 512)] = bits;
    else a.v_cache[row * a.kvw + (f - 512 - a.kvw)] = bits;
}

// Few rows: one 16-row x 16-feature tile per workgroup, d_model split over 8
// waves of KS 32-dim steps each (d_model = 256 * KS).
template <int KS, bool PAGED>
__global__ __launch_bounds__(512) void project_splitk_kernel(ProjArgs a) {
    __shared__ float part[kSplitWaves][16][16 + 1];
    const int ft = blockIdx.x, rt = blockIdx.y;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int k0 = wave * KS * 32 + grp * 8;
    const uint16_t *hp = a.h + (size_t)min(rt * 16 + col, a.rows - 1) * a.d + k0;
    const uint16_t *wp = a.w + (size_t)(ft * 16 + col) * a.d + k0;
    bf16x8 av[KS], bv[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        av[s] = ld8(hp + s * 32);
        bv[s] = ld8(wp + s * 32);
    }
    __builtin_amdgcn_sched_barrier(0);  // every load in flight before the first product
    f32x4 c = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[s], bv[s], c, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 4; ++r) part[wave][4 * grp + r][col] = c[r];
    __syncthreads();
    if (threadIdx.x < 256) {  // 16 x 16 outputs
        const int rr = threadIdx.x >> 4, f = threadIdx.x & 15;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kSplitWaves; ++w) sum += part[w][rr][f];
        store_feature<PAGED>(a, rt * 16 + rr, ft * 16 + f, sum);
    }
}

// Many rows: four waves on four 16-row tiles of the same 64 features.
template <bool PAGED>
__global__ __launch_bounds__(256) void project_rows_kernel(ProjArgs a) {
    const int ft = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int r0 = (blockIdx.y * 4 + wave) * 16;
    if (r0 >= a.rows) return;  // uniform per wave; no barriers
    const uint16_t *hp = a.h + (size_t)min(r0 + col, a.rows - 1) * a.d + grp * 8;
    const uint16_t *wp = a.w + (size_t)(ft * kProjFeat + col) * a.d + grp * 8;
    const size_t wct = (size_t)16 * a.d;  // next feature tile
    f32x4 c[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) c[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    bf16x8 a0, a1, b0[4], b1[4];
    auto load = [&](int kb, bf16x8 &av, bf16x8 (&bv)[4]) {
        av = ld8(hp + kb);
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) bv[ct] = ld8(wp + ct * wct + kb);
    };
    auto mma = [&](const bf16x8 &av, const bf16x8 (&bv)[4]) {
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
            c[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv[ct], c[ct], 0, 0, 0);
    };
    load(0, a0, b0);
    for (int kb = 0; kb < a.d; kb += 64) {  // d is a multiple of 512
        load(kb + 32, a1, b1);
        mma(a0, b0);
        if (kb + 64 < a.d) load(kb + 64, a0, b0);
        mma(a1, b1);
    }
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r)
            store_feature<PAGED>(a, r0 + 4 * grp + r, ft * kProjFeat + ct * 16 + col, c[ct][r]);
}

bool project_supported(int d_model) {
    return d_model >= 512 && d_model <= 8192 && d_model % 512 == 0;
}

template <int KS>
static void launch_splitk(const ProjArgs &a, bool paged, dim3 grid, hipStream_t stream) {
    if (paged) project_splitk_kernel<KS, true><<<grid, dim3(512), 0, stream>>>(a);
    else project_splitk_kernel<KS, false><<<grid, dim3(512), 0, stream>>>(a);
}

hipError_t launch_project(const Geometry &g, int d_model, const void *h, const void *w,
                          const int32_t *pos, const int32_t *page_table, void *q_idx,
                          void *k_idx, void *k_cache, void *v_cache, hipStream_t stream) {
    if (!project_supported(d_model)) return hipErrorInvalidValue;
    ProjArgs a;
    a.h = static_cast<const uint16_t *>(h);
    a.w = static_cast<const uint16_t *>(w);
    a.pos = pos;
    a.page_table = page_table;
    a.q_idx = static_cast<uint16_t *>(q_idx);
    a.k_idx = static_cast<uint16_t *>(k_idx);
    a.k_cache = static_cast<uint16_t *>(k_cache);
    a.v_cache = static_cast<uint16_t *>(v_cache);
    a.rows = g.rows;
    a.d = d_model;
    a.n_q = g.n_q;
    a.max_len = g.max_len;
    a.page_shift = g.page_shift;
    a.max_pages = g.max_pages;
    a.kvw = g.kv_heads * 128;
    if (g.rows == 0) return hipSuccess;
    const int n_feat = 512 + 2 * a.kvw;  // a multiple of 64
    const bool paged = g.page_shift >= 0;
    if (g.rows <= 64 && d_model <= kSplitMaxD) {
        const dim3 grid(n_feat / 16, div_up(g.rows, 16));
        switch (d_model / 512) {
            case 1: launch_splitk<2>(a, paged, grid, stream); break;
            case 2: launch_splitk<4>(a, paged, grid, stream); break;
            case 3: launch_splitk<6>(a, paged, grid, stream); break;
            case 4: launch_splitk<8>(a, paged, grid, stream); break;
            case 5: launch_splitk<10>(a, paged, grid, stream); break;
            case 6: launch_splitk<12>(a, paged, grid, stream); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    const long row_groups = (g.rows + 63) / 64;
    if (row_groups > 65535) return hipErrorInvalidConfiguration;
    const dim3 grid(n_feat / kProjFeat, (unsigned)row_groups);
    if (paged) project_rows_kernel<true><<<grid, dim3(256), 0, stream>>>(a);
    else project_rows_kernel<false><<<grid, dim3(256), 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace clsa
