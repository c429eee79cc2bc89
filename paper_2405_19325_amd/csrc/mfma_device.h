// Device helpers of the matrix-core distance kernels: the 16x16x32 MFMA with
// fp32 accumulation, squared norms of 16-byte chunks, and the lane reductions
// of the epilogues.
#pragma once

#include "knnlm_device.h"

namespace knnlm {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <knn_dtype DT>
__device__ __forceinline__ f32x4_t mfma16(const u32x4_t a, const u32x4_t b, f32x4_t c) {
    if constexpr (DT == KNN_BF16) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                       c, 0, 0, 0);
    } else {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b),
                                                      c, 0, 0, 0);
    }
}

// Sum of squares of a 16-byte chunk added to acc, word by word (dot2).
template <knn_dtype DT>
__device__ __forceinline__ float dot_vec(const u32x4_t v, float acc) {
    acc = dot_word<DT>(v.x, v.x, acc);
    acc = dot_word<DT>(v.y, v.y, acc);
    acc = dot_word<DT>(v.z, v.z, acc);
    return dot_word<DT>(v.w, v.w, acc);
}

// min / max over the 16 lanes of a row (every lane of the row gets it).
__device__ __forceinline__ float row16_min(float v) {
    v = fminf(v, dpp_f32<0xB1>(v));
    v = fminf(v, dpp_f32<0x4E>(v));
    v = fminf(v, dpp_f32<0x141>(v));
    return fminf(v, dpp_f32<0x140>(v));
}

__device__ __forceinline__ float row16_max(float v) {
    v = fmaxf(v, dpp_f32<0xB1>(v));
    v = fmaxf(v, dpp_f32<0x4E>(v));
    v = fmaxf(v, dpp_f32<0x141>(v));
    return fmaxf(v, dpp_f32<0x140>(v));
}

// Sum over the four lanes l % 16 == const (lane groups): every one of them gets it.
__device__ __forceinline__ float group4_sum(float v) {
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

// Slot of chunk c of row n in a swizzled LDS span buffer of CH 16-byte chunks per row.
template <int CH>
__device__ __forceinline__ int swz(int n, int c) { return n * CH + (c ^ (n & (CH - 1))); }

}  // namespace knnlm
