// Internal helpers shared by the libleap HIP sources (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "leap.h"

#define LEAP_API extern "C" __attribute__((visibility("default")))

namespace leap {

constexpr int kWave = 64;

// Map the launch result of the HIP runtime onto the library's status.
inline leap_status launch_status() {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? LEAP_OK : LEAP_ERR_HIP;
}

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
