// Training statistics of the method over one step's rollouts: the quantities
// of the pruning-range study (activated groups, per-rollout and per-group
// recovery after multi-turn debugging), the turn efficiency of the method
// comparison (total turns over passed samples), and the rollout-composition
// analysis (nonzero-advantage rollouts by group pass-rate bucket, outcome
// type and advantage sign).  Integer counters only, so the result does not
// depend on the order of the atomic additions.
//
// One wave per group: lanes walk the group's rollouts, wave sums give the
// group's counts, lane 0 adds them to the workgroup's LDS counters (64-bit
// LDS atomics), and the workgroup flushes its nonzero counters to the global
// array with one atomic each.
#include "leap_common.h"

namespace leap {
namespace {

constexpr int kStatsBlock = 256;
constexpr int kGroupsPerBlock = kStatsBlock / kWave;
constexpr int kMaxBuckets = 256;
constexpr int kHead = 9;  // groups .. passed rollouts
constexpr int kMaxCounters = kHead + 6 * kMaxBuckets;

enum {
    C_GROUPS = 0,
    C_ROLLOUTS,
    C_ACTIVATED,
    C_MULTI,
    C_RECOVERED,
    C_DEBUG_GROUPS,
    C_RECOVERED_GROUPS,
    C_TURNS,
    C_PASSED
};

__global__ __launch_bounds__(256) void stats_init_kernel(unsigned long long* counters, int n,
                                                         int64_t n_groups, int G) {
    for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x)
        counters[k] = k == C_GROUPS ? static_cast<unsigned long long>(n_groups)
                      : k == C_ROLLOUTS ? static_cast<unsigned long long>(n_groups) * G
                                        : 0ull;
}

__global__ __launch_bounds__(kStatsBlock) void rollout_stats_kernel(
    const int32_t* __restrict__ pass_turn, const int32_t* __restrict__ n_turns,
    const uint8_t* __restrict__ gate, const float* __restrict__ advantage, int64_t n_groups, int G,
    int M, int n_buckets, unsigned long long* __restrict__ counters, int32_t* __restrict__ dev_err) {
    __shared__ unsigned long long s_cnt[kMaxCounters];
    const int n_counters = kHead + 6 * n_buckets;
    for (int k = threadIdx.x; k < n_counters; k += kStatsBlock) s_cnt[k] = 0ull;
    __syncthreads();

    const int lane = threadIdx.x & (kWave - 1);
    const int64_t g = static_cast<int64_t>(blockIdx.x) * kGroupsPerBlock + threadIdx.x / kWave;
    if (g < n_groups) {
        const int64_t base = g * G;
        const bool activated = gate[g] != 0;
        int bad = 0, n_pass = 0, n_multi = 0, n_rec = 0;
        long long turns = 0;
        for (int i = lane; i < G; i += kWave) {
            const int m = pass_turn[base + i];
            const int T = n_turns[base + i];
            if (m < 0 || m > M || T < 1) {
                ++bad;
                continue;
            }
            turns += T;
            n_pass += m >= 1;
            if (activated && m != 1) {  // the first turn failed: debugging ran
                ++n_multi;
                n_rec += m >= 2;
            }
        }
        bad = wave_sum_i32(bad);
        n_pass = wave_sum_i32(n_pass);
        n_multi = wave_sum_i32(n_multi);
        n_rec = wave_sum_i32(n_rec);
        turns = wave_sum_i64(turns);
        if (lane == 0) {
            if (bad && dev_err) atomicAdd(dev_err, bad);
            atomicAdd(&s_cnt[C_TURNS], static_cast<unsigned long long>(turns));
            atomicAdd(&s_cnt[C_PASSED], static_cast<unsigned long long>(n_pass));
            if (activated) {
                atomicAdd(&s_cnt[C_ACTIVATED], 1ull);
                atomicAdd(&s_cnt[C_MULTI], static_cast<unsigned long long>(n_multi));
                atomicAdd(&s_cnt[C_RECOVERED], static_cast<unsigned long long>(n_rec));
                if (n_multi > 0) {
                    atomicAdd(&s_cnt[C_DEBUG_GROUPS], 1ull);
                    if (n_rec > 0) atomicAdd(&s_cnt[C_RECOVERED_GROUPS], 1ull);
                }
            }
        }
        if (advantage != nullptr) {
            // bucket of the group's observed pass rate, exact in integers
            int b = static_cast<int>(static_cast<int64_t>(n_pass) * n_buckets / G);
            b = b < n_buckets - 1 ? b : n_buckets - 1;
            int c[6] = {0, 0, 0, 0, 0, 0};  // (outcome, sign)
            for (int i = lane; i < G; i += kWave) {
                const int m = pass_turn[base + i];
                const int T = n_turns[base + i];
                const float a = advantage[base + i];
                if (m < 0 || m > M || T < 1 || a == 0.0f || a != a) continue;
                const int o = m == 1 ? 0 : (m >= 2 ? 1 : 2);
                ++c[o * 2 + (a > 0.0f ? 0 : 1)];
            }
#pragma unroll
            for (int k = 0; k < 6; ++k) {
                const int v = wave_sum_i32(c[k]);
                if (lane == 0 && v) atomicAdd(&s_cnt[kHead + b * 6 + k], static_cast<unsigned long long>(v));
            }
        }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < n_counters; k += kStatsBlock)
        if (k >= C_ACTIVATED && s_cnt[k]) atomicAdd(&counters[k], s_cnt[k]);  // 0, 1 set at init
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_rollout_stats(const int32_t* pass_turn, const int32_t* n_turns,
                                        const uint8_t* gate, const float* advantage,
                                        int64_t n_groups, int32_t G, int32_t M, int32_t n_buckets,
                                        int64_t* counters, int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    if (n_groups < 0 || G < 1 || G > 1024 || M < 1 || n_buckets < 1 || n_buckets > kMaxBuckets ||
        !counters)
        return LEAP_ERR_INVALID_ARG;
    if (n_groups > 0 && (!pass_turn || !n_turns || !gate)) return LEAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return LEAP_ERR_MISALIGNED;
    if (n_groups > 0x7fffffffLL) return LEAP_ERR_INVALID_ARG;
    const leap::LaunchCheck lc;
    const int n = kHead + 6 * n_buckets;
    unsigned long long* cnt = reinterpret_cast<unsigned long long*>(counters);
    hipLaunchKernelGGL(stats_init_kernel, dim3(1), dim3(256), 0, stream, cnt, n, n_groups, G);
    leap_status st = lc.status();
    if (st != LEAP_OK || n_groups == 0) return st;
    const int64_t blocks = (n_groups + kGroupsPerBlock - 1) / kGroupsPerBlock;
    hipLaunchKernelGGL(rollout_stats_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kStatsBlock), 0,
                       stream, pass_turn, n_turns, gate, advantage, n_groups, G, M, n_buckets, cnt,
                       dev_err);
    return lc.status();
}
