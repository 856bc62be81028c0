// Internal helpers shared by the libleap HIP sources (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "leap.h"

#define LEAP_API extern "C" __attribute__((visibility("default")))

namespace leap {

constexpr int kWave = 64;

// Launch errors of one entry point's own kernels.  Constructed before the
// call's first launch, it records the error the HIP runtime holds pending
// for this thread (without clearing it); status() reports LEAP_ERR_HIP only
// for a pending error that differs from it, i.e. one a launch of this call
// raised, and consumes that error.  An error the caller left pending before
// the call is neither reported nor cleared.
class LaunchCheck {
  public:
    LaunchCheck() : prior_(hipPeekAtLastError()) {}
    leap_status status() const {
        const hipError_t e = hipPeekAtLastError();
        if (e == hipSuccess || e == prior_) return LEAP_OK;
        (void)hipGetLastError();
        return LEAP_ERR_HIP;
    }

  private:
    hipError_t prior_;
};

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Count one data error on the optional device counter.
__device__ inline void count_error(int32_t* dev_err) {
    if (dev_err) atomicAdd(dev_err, 1);
}

// Butterfly sums over the 64 lanes of a wave; every lane ends with the total.
__device__ inline int wave_sum_i32(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ inline long long wave_sum_i64(long long v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ inline double wave_sum_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

}  // namespace leap
