// A plain read of a device buffer: the HBM read rate a streaming kernel can
// reach on this device, against which the distance stage's key streaming is
// judged (the distance stage reads each key once, so its time is bounded
// below by this read's).
#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

constexpr int kReadThreads = 256;
constexpr int kReadBlocks = 2048;  // about eight workgroups per CU
constexpr int kReadUnroll = 8;     // 16-byte loads in flight per lane

// Workgroup g reads the g-th of kReadBlocks contiguous pieces of the buffer
// (measured on MI355X: contiguous pieces per workgroup read about 15% faster
// than a grid-stride walk over the whole buffer).
__global__ __launch_bounds__(kReadThreads) void k_stream_read(const u32x4_t *buf, int64_t n16, uint32_t *out) {
    const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per;
    const int64_t b1 = b0 + per < n16 ? b0 + per : n16;
    int64_t i = b0 + threadIdx.x;
    uint32_t acc = 0u;
    for (; i + (kReadUnroll - 1) * kReadThreads < b1; i += kReadUnroll * kReadThreads) {
        u32x4_t v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) v[u] = __builtin_nontemporal_load(buf + i + u * kReadThreads);
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < b1; i += kReadThreads) {
        const u32x4_t v = __builtin_nontemporal_load(buf + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    // the loads must not be dropped: a store that (almost) never happens depends on them
    if (acc == 0x9e3779b9u) out[0] = acc;
}

}  // namespace

}  // namespace knnlm

extern "C" knn_status knn_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream) {
    using namespace knnlm;
    if (!buf || !sink || bytes < 16 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(buf) & 15u) != 0)
        return KNN_ERR_INVALID_ARG;
    hipLaunchKernelGGL(k_stream_read, dim3(kReadBlocks), dim3(kReadThreads), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4_t *>(buf), static_cast<int64_t>(bytes / 16), sink);
    return hipGetLastError() == hipSuccess ? KNN_OK : KNN_ERR_HIP;
}
