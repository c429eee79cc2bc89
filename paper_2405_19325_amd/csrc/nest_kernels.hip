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
// One thread per draft: the rows are a handful per draft and the data a few
// bytes each, so the kernel is launch-bound.
#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

constexpr int kVerifyThreads = 256;

__global__ __launch_bounds__(kVerifyThreads) void k_spec_verify(const float *p_max, const float *p_draft,
                                                                const int32_t *next_token,
                                                                const int64_t *draft_offsets, int64_t n_drafts,
                                                                float gamma, const float *uniforms,
                                                                int32_t *n_accept, int32_t *out_token) {
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kVerifyThreads + threadIdx.x;
    if (j >= n_drafts) return;
    const int64_t r0 = draft_offsets[j], r1 = draft_offsets[j + 1];
    int32_t accepted = static_cast<int32_t>(r1 - r0), token = -1;
    for (int64_t i = r0; i < r1; ++i) {
        const float ratio = p_draft[i] / (gamma * p_max[i]);
        const bool ok = uniforms != nullptr ? uniforms[i] < fminf(1.0f, ratio) : ratio > 0.5f;
        if (!ok) {
            accepted = static_cast<int32_t>(i - r0);
            token = next_token[i];
            break;
        }
    }
    n_accept[j] = accepted;
    out_token[j] = token;
}

}  // namespace

hipError_t launch_spec_verify(const float *p_max, const float *p_draft, const int32_t *next_token,
                              const int64_t *draft_offsets, int64_t n_drafts, float gamma, const float *uniforms,
                              int32_t *n_accept, int32_t *out_token, hipStream_t stream) {
    if (n_drafts <= 0) return hipSuccess;
    const int64_t blocks = (n_drafts + kVerifyThreads - 1) / kVerifyThreads;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_spec_verify, dim3(static_cast<unsigned>(blocks)), dim3(kVerifyThreads), 0, stream, p_max,
                       p_draft, next_token, draft_offsets, n_drafts, gamma, uniforms, n_accept, out_token);
    return hipGetLastError();
}

}  // namespace knnlm
