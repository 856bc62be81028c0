// The per-token objective of Sec. 3.1 (Eq. 3 per token: clipped importance
// ratio surrogate plus the reference KL term) as a scalar function of one
// row's log-sum-exp and token logit, and the fixed-order sum of the weighted
// per-row losses.  Shared by the logits-resident kernel and the fused
// LM-head path so both evaluate the same arithmetic.
#pragma once

#include "leap_common.h"

namespace leap {
namespace obj {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;

struct Params {
    float eps_lo, eps_hi, kl_coef, inv_temp;
    int kl_type;
};

// Per-token scalar epilogue.  lse2 = log2 sum_v 2^(x_v * c).
struct RowOut {
    float logp, loss, g, lse2;
};

// Hardware exp2 (v_exp_f32, about 1 ulp): no polynomial constants to keep in
// registers.
__device__ __forceinline__ float hw_exp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

__device__ __forceinline__ RowOut row_epilogue(float lse2, float xy, float old_lp, float ref_lp,
                                               float A, float w, const Params& p) {
    RowOut o;
    const float lse = lse2 * kLn2;
    const float logp = p.inv_temp * xy - lse;
    const float rho = hw_exp(logp - old_lp);
    const float clipped = fminf(fmaxf(rho, 1.0f - p.eps_lo), 1.0f + p.eps_hi);
    const float surr = fminf(rho * A, clipped * A);
    float kl, dkl;
    if (p.kl_type == LEAP_KL_K1) {
        kl = logp - ref_lp;
        dkl = 1.0f;
    } else if (p.kl_type == LEAP_KL_K2) {
        const float dd = logp - ref_lp;
        kl = 0.5f * dd * dd;
        dkl = dd;
    } else {
        const float dd = ref_lp - logp;
        const float em1 = hw_exp(dd) - 1.0f;
        kl = em1 - dd;
        dkl = -em1;
    }
    const bool active = (A > 0.0f && rho <= 1.0f + p.eps_hi) || (A < 0.0f && rho >= 1.0f - p.eps_lo);
    const float dl = (active ? -A * rho : 0.0f) + p.kl_coef * dkl;
    o.logp = logp;
    o.loss = -surr + p.kl_coef * kl;
    o.g = w * dl * p.inv_temp;
    o.lse2 = lse2;
    return o;
}

__device__ __forceinline__ void write_row_outputs(int64_t row, float logp, float loss, float w,
                                                  float* logp_out, float* tok_loss_out,
                                                  float* row_loss) {
    if (logp_out) logp_out[row] = logp;
    if (tok_loss_out) tok_loss_out[row] = loss;
    row_loss[row] = w * loss;
}

// Fixed-order sum of the per-row weighted losses (one workgroup); internal
// linkage so every source that launches it has its own copy.
namespace {
constexpr int kReduceBlock = 1024;

__global__ __launch_bounds__(kReduceBlock) void loss_reduce_kernel(const float* __restrict__ row_loss,
                                                                   int64_t N, float* __restrict__ loss_out) {
    __shared__ double s_w[kReduceBlock / kWave];
    const int tid = threadIdx.x;
    double acc = 0.0;
    for (int64_t k = tid; k < N; k += kReduceBlock) acc += static_cast<double>(row_loss[k]);
    acc = wave_sum_f64(acc);
    if ((tid & (kWave - 1)) == 0) s_w[tid / kWave] = acc;
    __syncthreads();
    if (tid == 0) {
        double t = 0.0;
        for (int w = 0; w < kReduceBlock / kWave; ++w) t += s_w[w];
        loss_out[0] = static_cast<float>(t);
    }
}

}  // namespace

}  // namespace obj
}  // namespace leap
