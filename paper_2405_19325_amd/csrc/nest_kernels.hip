// Relaxed speculative verification of NEST drafts (Section 3.4, eq. rejection,
// and Algorithm 1).  Draft j owns the rows draft_offsets[j] ..
// draft_offsets[j+1]-1 of a NEST step: row i carries max_w p_M(w), p_M of the
// draft token it checks and the lowest argmax of its p_M.  Token i is accepted
// while ratio_i = p_M(w^(i)) / (gamma * max_w p_M(w)) > 1/2 (the algorithm's
// threshold), or, with caller-drawn uniforms u_i, while u_i < min(1, ratio_i)
// (the equation read as a probability).  The first rejected row ends the
// draft: the count of accepted tokens and the rejected row's argmax (its
// replacement) are written; with no rejection every token is accepted and the
// replacement is -1.  All arithmetic in fp32, as ratio = p / (gamma * max).
//
// One wave per draft: 64 rows at a time load together (nothing waits on a
// decision before the loads), a ballot finds the first rejection.
#include "knnlm_device.h"
#include "select_internal.h"

namespace knnlm {

namespace {

constexpr int kVerifyWaves = 4;  // drafts per workgroup

__global__ __launch_bounds__(kVerifyWaves * kWave) void k_spec_verify(const float *p_max, const float *p_draft,
                                                                     const int32_t *next_token,
                                                                     const int64_t *draft_offsets, int64_t n_drafts,
                                                                     float gamma, const float *uniforms,
                                                                     int32_t *n_accept, int32_t *out_token) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kVerifyWaves + threadIdx.x / kWave;
    if (j >= n_drafts) return;  // the whole wave
    const int64_t r0 = draft_offsets[j], r1 = draft_offsets[j + 1];
    int64_t accepted = r1 - r0;
    int32_t token = -1;
    for (int64_t base = r0; base < r1; base += kWave) {
        const int64_t i = base + lane;
        const bool in = i < r1;
        const int64_t at = in ? i : r0;  // rows past the draft read its first row (unused)
        const float pd = p_draft[at], pm = p_max[at];
        const int32_t nt = next_token[at];
        const float u = uniforms != nullptr ? uniforms[at] : 0.0f;
        const float ratio = pd / (gamma * pm);
        const bool ok = uniforms != nullptr ? u < fminf(1.0f, ratio) : ratio > 0.5f;
        const uint64_t rejected = __ballot(in && !ok);
        if (rejected != 0ull) {
            const int first = __ffsll(static_cast<unsigned long long>(rejected)) - 1;
            accepted = base - r0 + first;
            token = __shfl(nt, first);
            break;
        }
    }
    if (lane == 0) {
        n_accept[j] = static_cast<int32_t>(accepted);
        out_token[j] = token;
    }
}

}  // namespace

hipError_t launch_spec_verify(const float *p_max, const float *p_draft, const int32_t *next_token,
                              const int64_t *draft_offsets, int64_t n_drafts, float gamma, const float *uniforms,
                              int32_t *n_accept, int32_t *out_token, hipStream_t stream) {
    if (n_drafts <= 0) return hipSuccess;
    const int64_t blocks = (n_drafts + kVerifyWaves - 1) / kVerifyWaves;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_spec_verify, dim3(static_cast<unsigned>(blocks)), dim3(kVerifyWaves * kWave), 0, stream, p_max,
                       p_draft, next_token, draft_offsets, n_drafts, gamma, uniforms, n_accept, out_token);
    return hipGetLastError();
}

}  // namespace knnlm
