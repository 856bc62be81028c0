// Discounted per-turn token advantage (Sec. 3.3) and loss-aggregation weight.
//
// One thread per token, grid-stride.  The rollout-level inputs are gathered
// (they are tiny and L2-resident); the discount beta^(T - t - 1) is formed by
// exact repeated multiplication in double, and each output is rounded once to
// float.
#include "leap_common.h"

namespace leap {
namespace {

__global__ __launch_bounds__(256) void token_advantages_kernel(
    const float* __restrict__ advantage, const int32_t* __restrict__ tok_rollout,
    const int32_t* __restrict__ tok_turn, const int32_t* __restrict__ n_turns,
    const int32_t* __restrict__ n_gen_tokens, int32_t n_rollouts, int64_t N, double gamma,
    int agg, double denominator, float* __restrict__ adv_tok, float* __restrict__ w_tok,
    int32_t* __restrict__ dev_err) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; k < N;
         k += stride) {
        const int i = tok_rollout[k];
        float a_out = 0.0f, w_out = 0.0f;
        if (i != -1) {
            bool ok = (i >= 0) && (i < n_rollouts);
            int t = 0, T = 0, ng = 0;
            if (ok) {
                t = tok_turn[k];
                T = n_turns[i];
                ng = n_gen_tokens[i];
                ok = (T >= 1) && (t >= 0) && (t < T) && (ng >= 1);
            }
            if (!ok) {
                count_error(dev_err);
            } else {
                const double A = static_cast<double>(advantage[i]);
                const double beta = (A >= 0.0) ? gamma : 1.0;
                double f = A;
                for (int e = T - t - 1; e > 0; --e) f *= beta;
                a_out = static_cast<float>(f);
                double w;
                if (agg == LEAP_AGG_SEQ_MEAN_TOKEN_MEAN)
                    w = 1.0 / (denominator * static_cast<double>(ng));
                else if (agg == LEAP_AGG_TOKEN_MEAN)
                    w = 1.0 / denominator;
                else
                    w = 1.0;
                w_out = static_cast<float>(w);
            }
        }
        adv_tok[k] = a_out;
        w_tok[k] = w_out;
    }
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_token_advantages(const float* advantage, const int32_t* tok_rollout,
                                           const int32_t* tok_turn, const int32_t* n_turns,
                                           const int32_t* n_gen_tokens, int32_t n_rollouts,
                                           int64_t N, float gamma, int32_t agg,
                                           double denominator, float* adv_tok, float* w_tok,
                                           int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    if (N < 0 || n_rollouts < 0) return LEAP_ERR_INVALID_ARG;
    if (!(gamma > 0.0f && gamma <= 1.0f)) return LEAP_ERR_INVALID_ARG;
    if (agg != LEAP_AGG_SEQ_MEAN_TOKEN_MEAN && agg != LEAP_AGG_TOKEN_MEAN && agg != LEAP_AGG_SUM)
        return LEAP_ERR_INVALID_ARG;
    if (agg != LEAP_AGG_SUM && !(denominator > 0.0 && __builtin_isfinite(denominator)))
        return LEAP_ERR_INVALID_ARG;
    if (N == 0) return LEAP_OK;
    if (!tok_rollout || !tok_turn || !adv_tok || !w_tok) return LEAP_ERR_INVALID_ARG;
    if (n_rollouts > 0 && (!advantage || !n_turns || !n_gen_tokens)) return LEAP_ERR_INVALID_ARG;
    const int block = 256;
    int64_t grid = (N + block - 1) / block;
    if (grid > 65536) grid = 65536;
    const leap::LaunchCheck lc;
    hipLaunchKernelGGL(token_advantages_kernel, dim3(static_cast<unsigned>(grid)), dim3(block), 0,
                       stream, advantage, tok_rollout, tok_turn, n_turns, n_gen_tokens,
                       n_rollouts, N, static_cast<double>(gamma), agg, denominator, adv_tok,
                       w_tok, dev_err);
    return lc.status();
}
