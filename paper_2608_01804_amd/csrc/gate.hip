// Difficulty-Conditioned Pruning gate (Sec. 3.1, Eqs. 1-2).
//
// One wave per group, four groups per 256-thread workgroup.  Each lane reads
// one first-turn outcome byte per 64-rollout slice; the wave ballot of
// "failed" lanes is popcounted, so N_fail needs no shared memory and no
// atomics.  Lane 0 applies the inclusive window of Eq. 2.
#include "leap_common.h"

namespace leap {
namespace {

constexpr int kGroupsPerBlock = 4;

__global__ __launch_bounds__(kGroupsPerBlock * kWave) void dcp_gate_kernel(
    const uint8_t* __restrict__ first_turn_pass, int64_t n_groups, int G, int tau_min,
    int tau_max, int32_t* __restrict__ n_fail, uint8_t* __restrict__ gate) {
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t g = static_cast<int64_t>(blockIdx.x) * kGroupsPerBlock + wave;
    if (g >= n_groups) return;  // uniform per wave
    const uint8_t* row = first_turn_pass + g * G;
    int nf = 0;
    for (int base = 0; base < G; base += kWave) {
        const int i = base + lane;
        const bool failed = (i < G) && (row[i] == 0);  // Eq. 1 indicator
        nf += __popcll(__ballot(failed));
    }
    if (lane == 0) {
        if (n_fail) n_fail[g] = nf;
        gate[g] = static_cast<uint8_t>((tau_min <= nf && nf <= tau_max) ? 1 : 0);  // Eq. 2
    }
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_dcp_gate(const uint8_t* first_turn_pass, int64_t n_groups, int32_t G,
                                   int32_t tau_min, int32_t tau_max, int32_t* n_fail,
                                   uint8_t* gate, hipStream_t stream) {
    using namespace leap;
    if (n_groups < 0 || G < 1 || G > 1024) return LEAP_ERR_INVALID_ARG;
    if (tau_min < 0 || tau_max > G || tau_min > tau_max) return LEAP_ERR_INVALID_ARG;
    if (n_groups == 0) return LEAP_OK;
    if (!first_turn_pass || !gate) return LEAP_ERR_INVALID_ARG;
    const int64_t grid = (n_groups + kGroupsPerBlock - 1) / kGroupsPerBlock;
    if (grid > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
    const leap::LaunchCheck lc;
    hipLaunchKernelGGL(dcp_gate_kernel, dim3(static_cast<unsigned>(grid)),
                       dim3(kGroupsPerBlock * kWave), 0, stream, first_turn_pass, n_groups, G,
                       tau_min, tau_max, n_fail, gate);
    return lc.status();
}

// Pass-rate window -> inclusive failure-count window, exactly.  With
// pass rate q(n) = (G - n) / G, n satisfies the lower end when
// (G - n) * lo_den > lo_num * G (strict) or >= (closed), and the upper end
// likewise; q is decreasing in n, so the admitted n form one interval.
LEAP_API leap_status leap_dcp_tau_from_pass_rate(int32_t G, int32_t lo_num, int32_t lo_den,
                                                 int32_t lo_strict, int32_t hi_num,
                                                 int32_t hi_den, int32_t hi_strict,
                                                 int32_t* tau_min, int32_t* tau_max) {
    if (G < 1 || lo_den <= 0 || hi_den <= 0 || !tau_min || !tau_max) return LEAP_ERR_INVALID_ARG;
    int32_t lo = -1, hi = -1;
    for (int32_t n = 0; n <= G; ++n) {
        const int64_t a_lo = static_cast<int64_t>(G - n) * lo_den;
        const int64_t b_lo = static_cast<int64_t>(lo_num) * G;
        const int64_t a_hi = static_cast<int64_t>(G - n) * hi_den;
        const int64_t b_hi = static_cast<int64_t>(hi_num) * G;
        const bool ok_lo = lo_strict ? (a_lo > b_lo) : (a_lo >= b_lo);
        const bool ok_hi = hi_strict ? (a_hi < b_hi) : (a_hi <= b_hi);
        if (ok_lo && ok_hi) {
            if (lo < 0) lo = n;
            hi = n;
        }
    }
    if (lo < 0) return LEAP_ERR_INVALID_ARG;
    *tau_min = lo;
    *tau_max = hi;
    return LEAP_OK;
}
