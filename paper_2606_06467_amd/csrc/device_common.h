// Device helpers shared by the gfx950 kernels of libclsa.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clsa {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load with the non-temporal hint (streamed once; keep it out of the caches).
__device__ __forceinline__ uint4 load16_nt(const void *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Four packed bf16 pairs (16 bytes) -> dot with four other pairs, fp32 accumulate.
// v_dot2_f32_bf16: the two bf16 x bf16 products are exact in fp32.
__device__ __forceinline__ float dot8_bf16(uint4 a, uint4 b, float acc) {
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.x),
                                          __builtin_bit_cast(bf16x2, b.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.y),
                                          __builtin_bit_cast(bf16x2, b.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.z),
                                          __builtin_bit_cast(bf16x2, b.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.w),
                                          __builtin_bit_cast(bf16x2, b.w), acc, false);
    return acc;
}

// Lane exchanges without the LDS crossbar.  Inside a row of 16 lanes, DPP (a
// VALU operand modifier): lane i reads lane 15 - i (row mirror), 7 - i within
// its half-row (half mirror), i ^ 2 or i ^ 1 (quad permutes).  Across rows,
// the gfx950 permlane swaps: v_permlane32_swap(x, y) leaves lanes 0-31 with
// (x[i], x[i + 32]) and lanes 32-63 with (y[i - 32], y[i]); v_permlane16_swap
// does the same between rows 0 and 1 and between rows 2 and 3.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}

// The value of `x` held by this lane's exchange partner at distance M <= 8
// inside a row.  A transpose step needs a partner with the other value of bit M
// that shares every higher exchanged bit, so the mirrors serve M = 8 and 4.
template <int M>
__device__ __forceinline__ float row_partner(float x) {
    static_assert(M == 8 || M == 4 || M == 2 || M == 1, "inside a row");
    if constexpr (M == 8) return dpp_f32<0x140>(x);
    else if constexpr (M == 4) return dpp_f32<0x141>(x);
    else if constexpr (M == 2) return dpp_f32<0x4E>(x);
    else return dpp_f32<0xB1>(x);
}

// lo + partner's lo for lanes with bit M clear, hi + partner's hi for lanes with
// it set (M = 16 or 32): the exchange step across rows.
template <int M>
__device__ __forceinline__ float cross_row_step(float lo, float hi) {
    static_assert(M == 16 || M == 32, "across rows");
    const auto r = M == 32 ? __builtin_amdgcn_permlane32_swap(__float_as_uint(lo),
                                                              __float_as_uint(hi), false, false)
                           : __builtin_amdgcn_permlane16_swap(__float_as_uint(lo),
                                                              __float_as_uint(hi), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Transpose-reduction across lanes.  Each lane holds CNT partial values; at the
// exchange with its partner at distance M it keeps the half selected by
// (lane & M) and adds the partner's copy of that half, for M, M/2, ..., MSTOP.
// Once a single value is left the remaining exchanges are plain sums.  With
// CNT = 2^s values and s halving steps, lane L ends with value index (L's step
// bits, high to low) of the original CNT, summed over every lane the steps
// visited.  All sizes are compile-time so that every register index stays static.
template <int CNT, int M, int MSTOP, int NV>
__device__ __forceinline__ void transpose_reduce(float (&p)[NV], int lane) {
    if constexpr (M >= MSTOP) {
        if constexpr (CNT > 1) {
            constexpr int H = CNT / 2;
            if constexpr (M >= 16) {
#pragma unroll
                for (int v = 0; v < H; ++v) p[v] = cross_row_step<M>(p[v], p[v + H]);
            } else {
                const bool up = (lane & M) != 0;
#pragma unroll
                for (int v = 0; v < H; ++v) {
                    const float keep = up ? p[v + H] : p[v];
                    const float send = up ? p[v] : p[v + H];
                    p[v] = keep + row_partner<M>(send);
                }
            }
            transpose_reduce<H, M / 2, MSTOP, NV>(p, lane);
        } else {
            if constexpr (M >= 16) p[0] = cross_row_step<M>(p[0], p[0]);
            else p[0] += row_partner<M>(p[0]);
            transpose_reduce<1, M / 2, MSTOP, NV>(p, lane);
        }
    }
}

// Maximum / sum over the 16 lanes of this lane's row; every lane of the row
// gets the result (quad swaps, then the half and full row mirrors).
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp_f32<0xB1>(x));
    x = fmaxf(x, dpp_f32<0x4E>(x));
    x = fmaxf(x, dpp_f32<0x141>(x));
    return fmaxf(x, dpp_f32<0x140>(x));
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f32<0xB1>(x);
    x += dpp_f32<0x4E>(x);
    x += dpp_f32<0x141>(x);
    return x + dpp_f32<0x140>(x);
}

// Maximum / sum over all 64 lanes; every lane gets the result.
__device__ __forceinline__ float wave_max(float x) {
    x = fmaxf(x, dpp_f32<0xB1>(x));
    x = fmaxf(x, dpp_f32<0x4E>(x));
    x = fmaxf(x, dpp_f32<0x141>(x));
    x = fmaxf(x, dpp_f32<0x140>(x));
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp_f32<0xB1>(x);
    x += dpp_f32<0x4E>(x);
    x += dpp_f32<0x141>(x);
    x += dpp_f32<0x140>(x);
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// Order-preserving map of an fp32 score to uint32 (larger score -> larger key).
// -0.0 is mapped like +0.0 so that the two compare equal.
__device__ __forceinline__ uint32_t score_key(float s) {
    uint32_t u = __float_as_uint(s);
    if ((u << 1) == 0u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Device-side error bits of the kernels of one source file: every kernel
// source includes this header, so each code object holds its own copy, read and
// cleared from the host by take_source_device_error().  Raised when a device
// value the host cannot check lies outside its documented range and is clamped.
constexpr uint32_t kDevErrSeqLen = 1u;  // seq_lens[b] outside [0, max_len]
constexpr uint32_t kDevErrNSel = 2u;    // n_sel[r] outside [0, top_k]
static __device__ uint32_t g_device_error;

// One atomic per wave that meets the condition (called inside the branch that
// found it; the first active lane reports).
__device__ __forceinline__ void note_device_error(uint32_t bit) {
    const uint64_t active = __ballot(1);
    if ((uint64_t)__lane_id() == (uint64_t)__builtin_ctzll(active)) atomicOr(&g_device_error, bit);
}

// A sequence length clamped to [0, max_len]; out-of-range lengths are flagged.
__device__ __forceinline__ int clamp_len(int n, int max_len) {
    if (n < 0 || n > max_len) {
        note_device_error(kDevErrSeqLen);
        return n < 0 ? 0 : max_len;
    }
    return n;
}

// Host side: this source file's error bits on the current device, cleared.
// Synchronous (a debug path).
static inline hipError_t take_source_device_error(uint32_t *bits) {
    uint32_t v = 0;
    hipError_t e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_device_error), sizeof v, 0,
                                       hipMemcpyDeviceToHost);
    if (e != hipSuccess) return e;
    if (v) {
        const uint32_t zero = 0;
        e = hipMemcpyToSymbol(HIP_SYMBOL(g_device_error), &zero, sizeof zero, 0,
                              hipMemcpyHostToDevice);
    }
    *bits |= v;
    return e;
}

// Number of valid keys of query row (b, t).
__device__ __forceinline__ int valid_keys(const int32_t *seq_lens, const int32_t *q_pos,
                                          int causal, int b, int row, int max_len) {
    int n = clamp_len(seq_lens[b], max_len);
    if (causal) {
        int lim = q_pos[row] + 1;
        n = lim < n ? (lim < 0 ? 0 : lim) : n;
    }
    return n;
}

// Element offset of token j of sequence b in a cache with `row_elems` elements
// per token: contiguous [B, max_len, ...] or paged [P, page, ...].
__device__ __forceinline__ size_t token_offset(const int32_t *page_table, int page_shift,
                                               int max_pages, int max_len, int b, int j,
                                               int row_elems) {
    if (page_shift < 0) return ((size_t)b * max_len + j) * row_elems;
    const int page = page_table[(size_t)b * max_pages + (j >> page_shift)];
    return (((size_t)page << page_shift) + (j & ((1 << page_shift) - 1))) * row_elems;
}

}  // namespace clsa
