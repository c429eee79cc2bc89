// Mixture stage (paper Section 2.2, eq. non-parametric and eq. kNN-LM): a
// softmax of mu * s = -mu * d over the r neighbours, scatter-added onto the
// neighbours' value tokens (tokens no neighbour carries get 0; duplicates
// accumulate), then p_M = lambda * p_LM + (1 - lambda) * p_kNN.
//
// Grid (query, vocabulary tile).  Each workgroup recomputes the r softmax
// weights (r <= 4096 exps, negligible next to the row it writes), scatters
// those whose token falls in its tile into an LDS accumulator with LDS float
// atomics, then streams its slice of p_LM in and p_M out with 16-byte accesses.
// The max of mu*s is subtracted first (it is -mu times the smallest distance),
// so the largest weight is exactly 1 and the sum cannot overflow.  p_M is formed
// as fmaf(lambda, p_LM, acc * ((1 - lambda) / Z)), so lambda = 1 returns p_LM
// bit for bit.  The order of the LDS atomics is not fixed, so p_kNN may differ
// between runs in the last bits.
#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

constexpr int kMixWaves = kMixThreads / kWave;

__global__ __launch_bounds__(kMixThreads) void k_mix(MixArgs a) {
    __shared__ float acc[kMixTile];
    __shared__ float red[kMixWaves];
    __shared__ float sh_val;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int64_t b = blockIdx.x;
    const int64_t v0 = static_cast<int64_t>(blockIdx.y) * kMixTile;
    const int64_t v1 = (v0 + kMixTile < a.V) ? v0 + kMixTile : a.V;
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    const int64_t N = a.key_offsets[s + 1] - k0;
    const int32_t *ids = a.ids + b * a.r;
    const float *dd = a.dists + b * a.r;

    for (int i = tid; i < kMixTile; i += kMixThreads) acc[i] = 0.0f;

    // smallest distance over the neighbours (= largest mu * s)
    float m = __builtin_huge_valf();
    for (int j = tid; j < a.r; j += kMixThreads) m = fminf(m, dd[j]);
    m = wave_allmin(m);
    if (lane == 0) red[wave] = m;
    __syncthreads();
    if (tid == 0) {
        float t = red[0];
        for (int w = 1; w < kMixWaves; ++w) t = fminf(t, red[w]);
        sh_val = t;
    }
    __syncthreads();
    m = sh_val;
    __syncthreads();

    // normaliser Z and the scatter of this tile's tokens
    float z = 0.0f;
    for (int j = tid; j < a.r; j += kMixThreads) {
        const float w = expf(-a.mu * (dd[j] - m));
        z += w;
        const int32_t id = ids[j];
        if (id >= 0 && id < N) {
            const int32_t tok = a.values[k0 + id];
            if (tok >= v0 && tok < v1) atomicAdd(&acc[tok - v0], w);
        }
    }
    z = wave_allsum(z);
    if (lane == 0) red[wave] = z;
    __syncthreads();
    if (tid == 0) {
        float t = red[0];
        for (int w = 1; w < kMixWaves; ++w) t += red[w];
        sh_val = t;
    }
    __syncthreads();
    z = sh_val;

    const float lam = a.lambda;
    const float scale = (1.0f - lam) / z;
    const float *plm = a.p_lm + b * a.V;
    float *pm = a.p_m + b * a.V;
    const int64_t n = v1 - v0;
    const bool vec4 = ((reinterpret_cast<uintptr_t>(plm + v0) | reinterpret_cast<uintptr_t>(pm + v0)) & 15u) == 0;
    if (vec4) {
        const int64_t n4 = n / 4;
        const float4 *src = reinterpret_cast<const float4 *>(plm + v0);
        float4 *dst = reinterpret_cast<float4 *>(pm + v0);
        for (int64_t i = tid; i < n4; i += kMixThreads) {
            const float4 p = src[i];
            float4 o;
            o.x = fmaf(lam, p.x, acc[4 * i + 0] * scale);
            o.y = fmaf(lam, p.y, acc[4 * i + 1] * scale);
            o.z = fmaf(lam, p.z, acc[4 * i + 2] * scale);
            o.w = fmaf(lam, p.w, acc[4 * i + 3] * scale);
            dst[i] = o;
        }
        for (int64_t i = 4 * n4 + tid; i < n; i += kMixThreads) pm[v0 + i] = fmaf(lam, plm[v0 + i], acc[i] * scale);
    } else {
        for (int64_t i = tid; i < n; i += kMixThreads) pm[v0 + i] = fmaf(lam, plm[v0 + i], acc[i] * scale);
    }
}

}  // namespace

hipError_t launch_mix(const MixArgs &args, int64_t B, hipStream_t stream) {
    if (B == 0) return hipSuccess;
    const int64_t tiles = (args.V + kMixTile - 1) / kMixTile;
    if (tiles > 65535 || B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(B), static_cast<unsigned>(tiles));
    hipLaunchKernelGGL(k_mix, grid, dim3(kMixThreads), 0, stream, args);
    return hipGetLastError();
}

}  // namespace knnlm
