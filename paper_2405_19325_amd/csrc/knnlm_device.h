// Device helpers shared by the kernels: the dot-product word step and wave reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "knnlm_internal.h"

namespace knnlm {

template <knn_dtype DT>
struct Elem;
template <>
struct Elem<KNN_F32> {
    static constexpr int VEC = 4;   // elements per 16-byte chunk
    static constexpr int BYTES = 4;
    static constexpr int PER_WORD = 1;  // elements per 32-bit word
};
template <>
struct Elem<KNN_BF16> {
    static constexpr int VEC = 8;
    static constexpr int BYTES = 2;
    static constexpr int PER_WORD = 2;
};
template <>
struct Elem<KNN_F16> {
    static constexpr int VEC = 8;
    static constexpr int BYTES = 2;
    static constexpr int PER_WORD = 2;
};

// acc + the products of one 32-bit word of q with the same word of k: two
// packed 16-bit elements through the gfx950 dot2 instruction (fp32 accumulate),
// or one fp32 element through an FMA.  Every dot product and squared norm in
// the library is a chain of these calls over the words of a row, so equal
// inputs give equal bits on every path.
template <knn_dtype DT>
__device__ __forceinline__ float dot_word(uint32_t q, uint32_t k, float acc);

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

template <>
__device__ __forceinline__ float dot_word<KNN_F32>(uint32_t q, uint32_t k, float acc) {
    return fmaf(__uint_as_float(q), __uint_as_float(k), acc);
}
template <>
__device__ __forceinline__ float dot_word<KNN_BF16>(uint32_t q, uint32_t k, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q), __builtin_bit_cast(bf16x2_t, k), acc,
                                           false);
}
template <>
__device__ __forceinline__ float dot_word<KNN_F16>(uint32_t q, uint32_t k, float acc) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, q), __builtin_bit_cast(f16x2_t, k), acc, false);
}

// Streaming 16-byte load: every key byte is read exactly once, so the load
// carries the non-temporal hint and does not displace reusable cache lines.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// The four words of a 16-byte chunk, in order.
template <knn_dtype DT>
__device__ __forceinline__ float dot_chunk(const uint4 q, const uint4 k, float acc) {
    acc = dot_word<DT>(q.x, k.x, acc);
    acc = dot_word<DT>(q.y, k.y, acc);
    acc = dot_word<DT>(q.z, k.z, acc);
    acc = dot_word<DT>(q.w, k.w, acc);
    return acc;
}

// Word w of a row read with element loads (elements past d read as 0).
template <knn_dtype DT>
__device__ __forceinline__ uint32_t load_word(const void *row, int64_t w, int64_t d) {
    if constexpr (DT == KNN_F32) {
        return w < d ? __float_as_uint(static_cast<const float *>(row)[w]) : 0u;
    } else {
        const uint16_t *h = static_cast<const uint16_t *>(row);
        const int64_t i = 2 * w;
        const uint32_t lo = i < d ? h[i] : 0u;
        const uint32_t hi = i + 1 < d ? h[i + 1] : 0u;
        return lo | (hi << 16);
    }
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// Sum over the 64 lanes of a wave; every lane receives the same bits.  Within
// each 16-lane row, DPP exchanges (xor 1, xor 2, half-row mirror, row mirror)
// add partner lanes -- both partners add the same two operands, so the whole
// row ends with one value -- then the four row sums are read out to scalar
// registers and added as (r0 + r1) + (r2 + r3).  No LDS round trips.
__device__ __forceinline__ float wave_allsum(float v) {
    v += dpp_f32<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f32<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_f32<0x141>(v);  // row_half_mirror
    v += dpp_f32<0x140>(v);  // row_mirror
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
    return static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(static_cast<int>(old), static_cast<int>(v), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int lane) {
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), lane));
}

// min / max over the 64 lanes (every lane gets the result): DPP exchanges
// within each 16-lane row, then the four row results via readlane.
__device__ __forceinline__ float wave_allmin(float v) {
    v = fminf(v, dpp_f32<0xB1>(v));
    v = fminf(v, dpp_f32<0x4E>(v));
    v = fminf(v, dpp_f32<0x141>(v));
    v = fminf(v, dpp_f32<0x140>(v));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return fminf(fminf(r0, r1), fminf(r2, r3));
}

// A value every lane of the wave reads at the same address, read through the
// scalar data cache (a read only): it is waited for on its own counter, so
// that using it does not wait for the vector loads and stores in flight.
__device__ __forceinline__ int32_t load_scalar_i32(const int32_t *p) {
    return *reinterpret_cast<const __attribute__((address_space(4))) int32_t *>(reinterpret_cast<uintptr_t>(p));
}

__device__ __forceinline__ float wave_allmax(float v) {
    v = fmaxf(v, dpp_f32<0xB1>(v));
    v = fmaxf(v, dpp_f32<0x4E>(v));
    v = fmaxf(v, dpp_f32<0x141>(v));
    v = fmaxf(v, dpp_f32<0x140>(v));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

__device__ __forceinline__ uint32_t wave_allmin_u32(uint32_t v) {
    v = min(v, dpp_u32<0xB1>(v, v));
    v = min(v, dpp_u32<0x4E>(v, v));
    v = min(v, dpp_u32<0x141>(v, v));
    v = min(v, dpp_u32<0x140>(v, v));
    return min(min(readlane_u32(v, 0), readlane_u32(v, 16)), min(readlane_u32(v, 32), readlane_u32(v, 48)));
}

__device__ __forceinline__ uint32_t wave_allmax_u32(uint32_t v) {
    v = max(v, dpp_u32<0xB1>(v, v));
    v = max(v, dpp_u32<0x4E>(v, v));
    v = max(v, dpp_u32<0x141>(v, v));
    v = max(v, dpp_u32<0x140>(v, v));
    return max(max(readlane_u32(v, 0), readlane_u32(v, 16)), max(readlane_u32(v, 32), readlane_u32(v, 48)));
}

// Inclusive prefix sum over the lanes of a wave: DPP row shifts by 1, 2, 4, 8
// (lanes without a source add 0) scan each 16-lane row; the totals of the rows
// below are then added from readlane.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v, int lane) {
    v += dpp_u32<0x111>(0u, v);  // row_shr:1
    v += dpp_u32<0x112>(0u, v);  // row_shr:2
    v += dpp_u32<0x114>(0u, v);  // row_shr:4
    v += dpp_u32<0x118>(0u, v);  // row_shr:8
    const uint32_t r0 = readlane_u32(v, 15), r1 = readlane_u32(v, 31), r2 = readlane_u32(v, 47);
    const int row = lane >> 4;
    return v + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Distances are >= +0, so their fp32 bit patterns order like the values.
__device__ __forceinline__ float clamp_nonneg(float x) { return x > 0.0f ? x : 0.0f; }

// Set s owning query b: the s with query_offsets[s] <= b < query_offsets[s+1]
// (the last such s when empty sets share an offset).
__device__ __forceinline__ int64_t set_of_query(const int64_t *query_offsets, int64_t S, int64_t b) {
    int64_t lo = 0, hi = S;  // invariant: qo[lo] <= b < qo[hi]
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (query_offsets[mid] <= b) lo = mid; else hi = mid;
    }
    return lo;
}

}  // namespace knnlm
