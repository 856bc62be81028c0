// Rank-based reward and GRPO advantage (Sec. 3.2, Eqs. 4-6).
//
// One group of G rollouts is handled by tpg = roundup(G, 64) threads; small
// groups share a workgroup (4 groups of <= 64 per 256 threads).  Each thread
// owns one rollout: the group's keys are staged in LDS, then every thread
// plays its G - 1 matches against the LDS copy (broadcast reads, no bank
// conflicts) and counts strict wins and losses.  Sums of d = wins - losses
// and d^2 go through wave butterflies and an LDS combine across the group's
// waves; the advantage is then formed in double precision from those exact
// integers and rounded once to float.
#include "leap_common.h"

namespace leap {
namespace {

constexpr int kMaxBlock = 1024;

template <bool kLex>
__global__ __launch_bounds__(kMaxBlock) void rank_tournament_kernel(
    const int32_t* __restrict__ pass_turn, const int32_t* __restrict__ speedup_q,
    const int32_t* __restrict__ n_tokens, int64_t n_groups, int G, int M, int norm, float eps,
    int tpg, int gpb, int32_t* __restrict__ n_worse, int32_t* __restrict__ n_better,
    int32_t* __restrict__ rank_r, float* __restrict__ reward, float* __restrict__ advantage,
    int32_t* __restrict__ dev_err) {
    __shared__ int s_r[kMaxBlock];
    __shared__ int s_s[kLex ? kMaxBlock : 1];
    __shared__ int s_n[kLex ? kMaxBlock : 1];
    __shared__ long long s_d[kMaxBlock / kWave];
    __shared__ long long s_d2[kMaxBlock / kWave];

    const int tid = threadIdx.x;
    const int gl = tid / tpg;  // group slot within the workgroup
    const int i = tid - gl * tpg;  // rollout within the group
    const int64_t g = static_cast<int64_t>(blockIdx.x) * gpb + gl;
    const bool mine = (g < n_groups) && (i < G);
    const int64_t idx = g * G + i;

    // Eq. 4: tier from the turn of first pass.
    int r = 0, s = 0, n = 0;
    if (mine) {
        const int m = pass_turn[idx];
        if (m < 0 || m > M) {
            count_error(dev_err);
            r = 0;
        } else {
            r = (m == 0) ? 0 : (M - m + 1);
        }
        if (kLex) {
            s = speedup_q[idx];
            n = n_tokens[idx];
        }
        s_r[tid] = r;
        if (kLex) {
            s_s[tid] = s;
            s_n[tid] = n;
        }
    }
    __syncthreads();

    // Eq. 5: the complete pairwise tournament against the LDS copy.
    int worse = 0, better = 0;
    if (mine) {
        const int base = gl * tpg;
        for (int j = 0; j < G; ++j) {
            const int rj = s_r[base + j];
            int c;
            if (kLex) {
                const int sj = s_s[base + j];
                const int nj = s_n[base + j];
                c = (r != rj) ? (r > rj ? 1 : -1)
                    : (s != sj) ? (s > sj ? 1 : -1)
                    : (n != nj) ? (n < nj ? 1 : -1) : 0;
            } else {
                c = (r > rj) - (r < rj);
            }
            // j == i compares equal and counts for neither side.
            worse += (c > 0);
            better += (c < 0);
        }
    }
    const int d = worse - better;

    // Group sums of d and d^2 (exact integers).
    const long long wd = wave_sum_i64(mine ? d : 0);
    const long long wd2 = wave_sum_i64(mine ? static_cast<long long>(d) * d : 0);
    const int wave = tid / kWave;
    if ((tid & (kWave - 1)) == 0) {
        s_d[wave] = wd;
        s_d2[wave] = wd2;
    }
    __syncthreads();
    if (!mine) return;
    long long sd = 0, sd2 = 0;
    const int w0 = (gl * tpg) / kWave, w1 = ((gl + 1) * tpg) / kWave;
    for (int w = w0; w < w1; ++w) {
        sd += s_d[w];
        sd2 += s_d2[w];
    }

    // Eq. 6, in double, rounded once.
    const double gm1 = static_cast<double>(G - 1);
    const double R = static_cast<double>(d) / gm1;
    if (n_worse) n_worse[idx] = worse;
    if (n_better) n_better[idx] = better;
    if (rank_r) rank_r[idx] = r;
    reward[idx] = static_cast<float>(R);

    double A;
    if (norm == LEAP_ADV_NONE) {
        A = R;
    } else {
        // mean R = sum d / (G (G-1)); unbiased variance of R from the exact
        // centred sum of squares sum d^2 - (sum d)^2 / G.
        const double mean = static_cast<double>(sd) / static_cast<double>(G) / gm1;
        const double css = static_cast<double>(sd2) -
                           static_cast<double>(sd) * static_cast<double>(sd) / static_cast<double>(G);
        const double var = css / (gm1 * gm1) / gm1;
        const double stdv = sqrt(var > 0.0 ? var : 0.0);
        A = (R - mean) / (stdv + static_cast<double>(eps));
    }
    advantage[idx] = static_cast<float>(A);
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_rank_advantages(const int32_t* pass_turn, const int32_t* speedup_q,
                                          const int32_t* n_tokens, int64_t n_groups, int32_t G,
                                          int32_t M, int32_t key, int32_t norm, float eps,
                                          int32_t* n_worse, int32_t* n_better, int32_t* rank_r,
                                          float* reward, float* advantage, int32_t* dev_err,
                                          hipStream_t stream) {
    using namespace leap;
    if (n_groups < 0 || G < 2 || G > 1024 || M < 1) return LEAP_ERR_INVALID_ARG;
    if (!(eps >= 0.0f) || !__builtin_isfinite(eps)) return LEAP_ERR_INVALID_ARG;
    if (key != LEAP_KEY_TURN && key != LEAP_KEY_LEX) return LEAP_ERR_INVALID_ARG;
    if (norm != LEAP_ADV_STD && norm != LEAP_ADV_NONE) return LEAP_ERR_INVALID_ARG;
    if (n_groups == 0) return LEAP_OK;
    if (!pass_turn || !reward || !advantage) return LEAP_ERR_INVALID_ARG;
    if (key == LEAP_KEY_LEX && (!speedup_q || !n_tokens)) return LEAP_ERR_INVALID_ARG;

    const int tpg = (G + kWave - 1) / kWave * kWave;
    const int gpb = tpg >= 256 ? 1 : 256 / tpg;
    const int block = tpg * gpb;
    const int64_t grid = (n_groups + gpb - 1) / gpb;
    if (grid > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
    const leap::LaunchCheck lc;
    if (key == LEAP_KEY_LEX) {
        hipLaunchKernelGGL(rank_tournament_kernel<true>, dim3(static_cast<unsigned>(grid)),
                           dim3(block), 0, stream, pass_turn, speedup_q, n_tokens, n_groups, G, M,
                           norm, eps, tpg, gpb, n_worse, n_better, rank_r, reward, advantage,
                           dev_err);
    } else {
        hipLaunchKernelGGL(rank_tournament_kernel<false>, dim3(static_cast<unsigned>(grid)),
                           dim3(block), 0, stream, pass_turn, speedup_q, n_tokens, n_groups, G, M,
                           norm, eps, tpg, gpb, n_worse, n_better, rank_r, reward, advantage,
                           dev_err);
    }
    return lc.status();
}
