// Measurement helpers, not part of the method.
//
// HBM bandwidth probe.  It
// streams memory with the access shape of the fused kernel (16-byte
// non-temporal buffer accesses, 1024-lane workgroups, eight accesses in
// flight per lane) so the achievable read, write and read+write rates of the
// device can be set beside the published peak.
#include "leap_common.h"

namespace leap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeBlock = 1024;
constexpr int kProbeUnroll = 8;

template <int MODE>  // 0: copy, 1: read, 2: write
__global__ __launch_bounds__(kProbeBlock) void hbm_probe_kernel(const u32x4* __restrict__ src,
                                                                u32x4* __restrict__ dst,
                                                                int64_t n16) {
    const int64_t step = static_cast<int64_t>(gridDim.x) * kProbeBlock * kProbeUnroll;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kProbeBlock * kProbeUnroll + threadIdx.x;
         i < n16; i += step) {
        u32x4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) {
            const int64_t k = i + static_cast<int64_t>(u) * kProbeBlock;
            if (MODE != 2 && k < n16)
                v[u] = __builtin_nontemporal_load(src + k);
            else
                v[u] = u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) {
            const int64_t k = i + static_cast<int64_t>(u) * kProbeBlock;
            if (MODE == 1)
                acc ^= v[u];
            else if (k < n16)
                __builtin_nontemporal_store(v[u], dst + k);
        }
    }
    // keeps the reads of the read-only mode alive; practically never taken
    if (MODE == 1 && acc.x == 0x9e3779b9u && acc.y == 0x7f4a7c15u) dst[0] = acc;
}

// MFMA probe: four waves per workgroup, each issuing `iters` rounds of
// eight independent v_mfma_f32_16x16x32_bf16 on register operands (no
// memory traffic inside the loop), so the matrix cores' achievable bf16 rate
// -- at the clock the chip holds for pure MFMA work -- can be set beside the
// published peak and beside the fused LM head's rate.
//
// RANDOM == false: every operand is `one` (a run-time value, so nothing
// folds); with one == 1 every output element of an accumulator gains 32 per
// MFMA, and lane 0 of wave 0 writes its first accumulator's first element,
// iters * 32 (exact below 2^24), to sink[blockIdx.x] (-1 if the chains
// disagree).  Constant operands leave the multipliers' inputs unchanged from
// one MFMA to the next, so this is the rate at the lowest switching power.
//
// RANDOM == true: each chain multiplies its own pair of operand vectors,
// bf16 values of magnitude [1, 2) with random sign and mantissa bits per
// lane (MurmurHash3's 32-bit finaliser over lane, wave, chain and
// workgroup), so consecutive MFMAs switch about half of the input bits, as
// a GEMM over random data does; the chip's power limit then sets the clock.
// sink[blockIdx.x] receives a finite sum of the products.
constexpr int kMfmaProbeBlock = 256;
constexpr int kMfmaProbeChains = 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));

__device__ inline uint32_t fmix32(uint32_t h) {
    h ^= h >> 16;
    h *= 0x85ebca6bu;
    h ^= h >> 13;
    h *= 0xc2b2ae35u;
    h ^= h >> 16;
    return h;
}

// two bf16 of magnitude [1, 2): sign and 7 mantissa bits from the hash
__device__ inline uint32_t random_bf16_pair(uint32_t h) {
    const uint32_t lo = 0x3f80u | (h & 0x807fu);
    const uint32_t hi = 0x3f80u | ((h >> 16) & 0x807fu);
    return lo | (hi << 16);
}

__device__ inline bf16x8 random_operand(uint32_t seed) {
    u32x4v w;
    w.x = random_bf16_pair(fmix32(seed * 4u + 0u));
    w.y = random_bf16_pair(fmix32(seed * 4u + 1u));
    w.z = random_bf16_pair(fmix32(seed * 4u + 2u));
    w.w = random_bf16_pair(fmix32(seed * 4u + 3u));
    return __builtin_bit_cast(bf16x8, w);
}

template <bool RANDOM>
__global__ __launch_bounds__(kMfmaProbeBlock) void mfma_probe_kernel(int64_t iters, float one,
                                                                     float* __restrict__ sink) {
    bf16x8 a[kMfmaProbeChains], b[kMfmaProbeChains];
    f32x4 acc[kMfmaProbeChains];
#pragma unroll
    for (int c = 0; c < kMfmaProbeChains; ++c) {
        if (RANDOM) {
            const uint32_t base =
                ((blockIdx.x * kMfmaProbeBlock + threadIdx.x) * kMfmaProbeChains + c) * 2u;
            a[c] = random_operand(base);
            b[c] = random_operand(base + 1u);
        } else {
            const __bf16 v = static_cast<__bf16>(one);
            a[c] = bf16x8{v, v, v, v, v, v, v, v};
            b[c] = a[c];
        }
        acc[c] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    // The accumulators stay in AGPRs through the loop ("+a"): written with
    // the builtin, the compiler copies them between AGPRs and VGPRs on every
    // iteration, and the probe then measures those copies.
    // The compiler inserts no wait states around inline assembly, so the
    // operand and accumulator writes before the loop and the MFMA results
    // after it are separated from their readers by explicit s_nop (ample
    // for any pass count), tied to those registers so they stay in place.
    asm volatile("s_nop 7\n\ts_nop 7"
                 : "+a"(acc[0]), "+a"(acc[1]), "+a"(acc[2]), "+a"(acc[3]), "+a"(acc[4]),
                   "+a"(acc[5]), "+a"(acc[6]), "+a"(acc[7]), "+v"(a[0]), "+v"(a[1]), "+v"(a[2]),
                   "+v"(a[3]), "+v"(a[4]), "+v"(a[5]), "+v"(a[6]), "+v"(a[7]), "+v"(b[0]),
                   "+v"(b[1]), "+v"(b[2]), "+v"(b[3]), "+v"(b[4]), "+v"(b[5]), "+v"(b[6]),
                   "+v"(b[7]));
    for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < kMfmaProbeChains; ++c)
            asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                         : "+a"(acc[c])
                         : "v"(a[c]), "v"(b[c]));
    }
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(acc[0]), "+a"(acc[1]), "+a"(acc[2]), "+a"(acc[3]), "+a"(acc[4]),
                   "+a"(acc[5]), "+a"(acc[6]), "+a"(acc[7]));
    float v = acc[0].x;
    if (RANDOM) {
#pragma unroll
        for (int c = 1; c < kMfmaProbeChains; ++c) v += acc[c].x;
    } else {
#pragma unroll
        for (int c = 1; c < kMfmaProbeChains; ++c) v = (acc[c].x == v) ? v : -1.0f;
    }
    if (threadIdx.x == 0) sink[blockIdx.x] = v;
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_probe_mfma(int64_t iters, int32_t n_workgroups, int32_t random_operands,
                                     float* sink, hipStream_t stream) {
    using namespace leap;
    if (iters < 1 || n_workgroups < 1 || random_operands < 0 || random_operands > 1 || !sink)
        return LEAP_ERR_INVALID_ARG;
    const LaunchCheck lc;
    const dim3 grid(static_cast<unsigned>(n_workgroups)), block(kMfmaProbeBlock);
    if (random_operands)
        hipLaunchKernelGGL(mfma_probe_kernel<true>, grid, block, 0, stream, iters, 1.0f, sink);
    else
        hipLaunchKernelGGL(mfma_probe_kernel<false>, grid, block, 0, stream, iters, 1.0f, sink);
    return lc.status();
}

LEAP_API leap_status leap_probe_hbm(const void* src, void* dst, size_t bytes, int32_t mode,
                                    hipStream_t stream) {
    using namespace leap;
    if (mode < 0 || mode > 2 || (bytes & 15u) != 0) return LEAP_ERR_INVALID_ARG;
    if (bytes == 0) return LEAP_OK;
    if ((mode != 2 && !src) || !dst) return LEAP_ERR_INVALID_ARG;
    if ((mode != 2 && !aligned16(src)) || !aligned16(dst)) return LEAP_ERR_MISALIGNED;
    const leap::LaunchCheck lc;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return LEAP_ERR_HIP;
    const int64_t n16 = static_cast<int64_t>(bytes / 16);
    const int64_t per_block = static_cast<int64_t>(kProbeBlock) * kProbeUnroll;
    int64_t grid = (n16 + per_block - 1) / per_block;
    const int64_t cap = static_cast<int64_t>(cus > 0 ? cus : 1) * 2;
    if (grid > cap) grid = cap;
    const u32x4* s = static_cast<const u32x4*>(src);
    u32x4* d = static_cast<u32x4*>(dst);
    if (mode == 0)
        hipLaunchKernelGGL(hbm_probe_kernel<0>, dim3(grid), dim3(kProbeBlock), 0, stream, s, d, n16);
    else if (mode == 1)
        hipLaunchKernelGGL(hbm_probe_kernel<1>, dim3(grid), dim3(kProbeBlock), 0, stream, s, d, n16);
    else
        hipLaunchKernelGGL(hbm_probe_kernel<2>, dim3(grid), dim3(kProbeBlock), 0, stream, s, d, n16);
    return lc.status();
}
