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
//   * many rows (prefill): a tiled product, 128 rows x 128 features per
//     workgroup of 4 waves (64 x 64 each, 4 x 4 tiles of 16 x 16), d_model in
//     steps of 64 staged through LDS (double-buffered: the next step's global
//     loads are in flight during the current products); the 128-feature tile
//     lies in one destination (index query, index key, K or V), so the bf16
//     results go back through LDS and leave as whole 256-byte rows.
#include "clsa_internal.h"
#include "device_common.h"

namespace clsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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
    int rtiles, ftiles, band;  // tiled kernel: 128-row and 128-feature tiles, row tiles per band
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

// Many rows: the tiled product.
constexpr int kGemmM = 128, kGemmN = 128, kGemmK = 64;
constexpr int kGemmPitch = kGemmK + 8;       // bf16 per staged row (16 bytes of padding)
constexpr int kGemmOutPitch = kGemmN + 8;    // bf16 per staged output row
constexpr size_t kGemmLds = sizeof(uint16_t) * 2 * 2 * kGemmM * kGemmPitch;

template <bool PAGED>
__global__ __launch_bounds__(256, 2) void project_gemm_kernel(ProjArgs a) {
    // two stages of A (rows of h) and B (features of w), 128 x 64 bf16 each
    // (dynamic LDS, kGemmLds bytes); the output tile (128 x 128 bf16) reuses it
    extern __shared__ __align__(16) uint16_t s_lds[];
    uint16_t(*s_ab)[2][kGemmM][kGemmPitch] =
        reinterpret_cast<uint16_t(*)[2][kGemmM][kGemmPitch]>(s_lds);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;  // the wave's 64 x 64 quadrant
    // Tile order: workgroups are dealt to the 8 XCDs in turn (L mod 8); XCD x
    // takes bands of `band` row tiles (8, fewer when there are few rows) and
    // walks, for each band, the feature tiles with the band's row tiles next to
    // each other, so that the workgroups in flight on an XCD share a few row
    // tiles and feature tiles per 64-wide step of d_model (their slices meet in
    // its L2).
    int rt, ft;
    {
        const int L = blockIdx.x, x = L & 7, q = L >> 3;
        const int per_band = a.band * a.ftiles;          // workgroups of one band
        const int band = 8 * (q / per_band) + x;         // bands dealt to the XCDs in turn
        const int qi = q % per_band;
        rt = a.band * band + qi % a.band;
        ft = qi / a.band;
    }
    if (rt >= a.rtiles) return;  // uniform: padding workgroups of the last bands
    const int f0 = ft * kGemmN, r0 = rt * kGemmM;
    // staging: thread t moves 16-byte pieces t + 256 i (i < 4) of each 128 x 64
    // tile: row (t >> 3) + 32 i, columns 8 (t & 7) .. + 8
    const int lrow = tid >> 3, lcol = (tid & 7) * 8;
    const uint16_t *hp[4], *wp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        hp[i] = a.h + (size_t)min(r0 + lrow + 32 * i, a.rows - 1) * a.d + lcol;  // tail rows: never stored
        wp[i] = a.w + (size_t)(f0 + lrow + 32 * i) * a.d + lcol;
    }
    // two register sets: the loads for step k + 2 are issued while step k is
    // computed, and step k + 1 (loaded a step earlier) goes to LDS after it;
    // every step issues its loads (the last two reload a valid step that is
    // never stored), so that the compiler's wait before each LDS store leaves
    // the newest 8 loads in flight
    u32x4 ra[2][4], rb[2][4];
    auto gload = [&](int set, int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            ra[set][i] = *reinterpret_cast<const u32x4 *>(hp[i] + k0);
            rb[set][i] = *reinterpret_cast<const u32x4 *>(wp[i] + k0);
        }
    };
    auto lstore = [&](int set, int st) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            *reinterpret_cast<u32x4 *>(&s_ab[st][0][lrow + 32 * i][lcol]) = ra[set][i];
            *reinterpret_cast<u32x4 *>(&s_ab[st][1][lrow + 32 * i][lcol]) = rb[set][i];
        }
    };
    f32x4 c[4][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) c[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nk = a.d / kGemmK;  // even (d_model is a multiple of 512)
    gload(0, 0);
    gload(1, kGemmK);
    lstore(0, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      for (int h = 0; h < 2; ++h) {   // unrolled by two so that register sets are static
        const int k = kt + h;
        const int st = h;
        gload(h, min(k + 2, nk - 1) * kGemmK);  // unconditional (the last steps reload a valid step, never stored): a static load count
#pragma unroll
        for (int ks = 0; ks < kGemmK / 32; ++ks) {
            bf16x8 av[4], bv[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                av[t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(
                                                       &s_ab[st][0][wm * 64 + t * 16 + col][ks * 32 + grp * 8]));
                bv[t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(
                                                       &s_ab[st][1][wn * 64 + t * 16 + col][ks * 32 + grp * 8]));
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
                    c[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[mt], bv[nt], c[mt][nt], 0, 0, 0);
        }
        if (k + 1 < nk) lstore(h ^ 1, h ^ 1);
        __syncthreads();
      }
    }
    // bf16 results into LDS: C tile (mt, nt) row 4 grp + r, column col
    uint16_t(*s_out)[kGemmOutPitch] = reinterpret_cast<uint16_t(*)[kGemmOutPitch]>(&s_ab[0][0][0][0]);
    static_assert(kGemmLds >= sizeof(uint16_t) * kGemmM * kGemmOutPitch, "output tile fits");
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                s_out[wm * 64 + mt * 16 + 4 * grp + r][wn * 64 + nt * 16 + col] =
                    (uint16_t)f32_to_bf16_bits(c[mt][nt][r]);
    __syncthreads();
    // whole rows out: 16 pieces of 16 bytes per row, 8 rows per pass of 128 threads
    const int piece = tid & 15;
    int dst_kind, width, fo;  // 0: index query, 1: index key, 2: K, 3: V
    if (f0 < 256) { dst_kind = 0; width = 256; fo = f0; }
    else if (f0 < 512) { dst_kind = 1; width = 256; fo = f0 - 256; }
    else if (f0 < 512 + a.kvw) { dst_kind = 2; width = a.kvw; fo = f0 - 512; }
    else { dst_kind = 3; width = a.kvw; fo = f0 - 512 - a.kvw; }
    for (int rr = tid >> 4; rr < kGemmM; rr += 16) {
        const int r = r0 + rr;
        if (r >= a.rows) break;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(&s_out[rr][piece * 8]);
        uint16_t *dst;
        if (dst_kind == 0) {
            dst = a.q_idx + (size_t)r * 256;
        } else {
            const int p = a.pos[r];
            if (p < 0 || p >= a.max_len) continue;
            const int b = r / a.n_q;
            size_t row;
            if (PAGED) {
                const int page = a.page_table[(size_t)b * a.max_pages + (p >> a.page_shift)];
                row = ((size_t)page << a.page_shift) + (p & ((1 << a.page_shift) - 1));
            } else {
                row = (size_t)b * a.max_len + p;
            }
            dst = (dst_kind == 1 ? a.k_idx : dst_kind == 2 ? a.k_cache : a.v_cache) + row * width;
        }
        *reinterpret_cast<u32x4 *>(dst + fo + piece * 8) = v;
    }
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
    const int n_feat = 512 + 2 * a.kvw;  // a multiple of 256 (kv_heads * 128 per K and V)
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
    a.rtiles = div_up(g.rows, kGemmM);
    a.ftiles = n_feat / kGemmN;
    // bands of up to 8 row tiles, dealt to the 8 XCDs in turn (the last round
    // padded); fewer row tiles per band when that still leaves XCDs idle
    a.band = a.rtiles >= 64 ? 8 : div_up(a.rtiles, 8);
    const long bands = div_up(a.rtiles, a.band);
    const long blocks = div_up((int)bands, 8) * 8 * (long)a.band * a.ftiles;
    if (blocks > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)blocks);
    const void *fn = paged ? reinterpret_cast<const void *>(&project_gemm_kernel<true>)
                           : reinterpret_cast<const void *>(&project_gemm_kernel<false>);
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kGemmLds);
    if (e != hipSuccess) return e;
    if (paged) project_gemm_kernel<true><<<grid, dim3(256), kGemmLds, stream>>>(a);
    else project_gemm_kernel<false><<<grid, dim3(256), kGemmLds, stream>>>(a);
    return hipGetLastError();
}

}  // namespace clsa
