// Device helpers of the matrix-core distance kernels: the 16x16x32 MFMA with
// fp32 accumulation, squared norms of 16-byte chunks, and the lane reductions
// of the epilogues.
#pragma once

#include "knnlm_device.h"

namespace knnlm {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// The s_waitcnt immediate (gfx9 layout: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8) that waits until at most N vector memory operations are
// outstanding and leaves the other counters unconstrained.  Needed for loads
// that go straight to LDS, which no register use makes the compiler wait for.
template <int N>
constexpr int vmcnt_encoding() {
    static_assert(N >= 0 && N < 64, "vmcnt is six bits");
    return (N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8);
}
constexpr int kVmcntZero = vmcnt_encoding<0>();

// One 16-byte global load per lane straight into LDS: lane l's 16 bytes land at
// dst + l (dst is the wave's, the same in every lane).  Written as assembly so
// that the compiler, which cannot tell which LDS bytes such a load writes, does
// not make every later LDS read and barrier wait for all loads in flight; the
// caller waits for these loads itself (vmcnt_encoding), and the compiler's own
// vmcnt waits, not counting them, only wait longer than they need.  It sets
// M0, which the compiler reserves (a clobber of it is ignored): the kernels
// that use it leave M0 to these loads alone (their assembly sets it nowhere
// else).
__device__ __forceinline__ void load_to_lds_16(const void *src, u32x4_t *dst) {
    const uint32_t lds = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) u32x4_t *)dst)));
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds));
}

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
