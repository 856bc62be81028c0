// bf16 "NT" GEMM core on gfx950 MFMA: C[M][N] = sum_k A[m][k] * B[n][k], with
// A [M][lda] and B [N][ldb] both contiguous along k, fp32 accumulation, and
// the result handed to an epilogue functor instead of being stored.
//
//  * Workgroup tile 256 x 256, k-tiles of 32, 256 lanes = 4 waves in a 2 x 2
//    grid, each wave a 128 x 128 block of 4 x 4 v_mfma_f32_32x32x16_bf16
//    tiles (256 fp32 accumulators per lane, one wave per SIMD).
//  * Operand k-tiles go straight from HBM to LDS (buffer_load_dwordx4 ... lds,
//    no VGPR staging) into a ring of 4 stages of 32 KiB, three k-tiles ahead
//    of the one being multiplied.  The compiler does not track these LDS
//    writes, so each wave waits on its own vmcnt before the stage barrier.
//  * LDS rows are 64 bytes (32 bf16); the 16-byte chunk c of row r sits at
//    position c ^ ((r >> 2) & 3), so the 16-row MFMA fragment reads hit 64
//    distinct banks, and every load instruction fills 1 KiB contiguously.
//  * Tiles are numbered so the workgroups one XCD runs at once form a compact
//    GROUP x (32 / GROUP) patch (see tile_of_block).
//
// Operand fragments of v_mfma_f32_32x32x16_bf16 (lane l of 64): A row l%32
// with k = 8*(l/32) .. +7; B column l%32 with the same k; accumulator
// register r holds C[row (r/4)*8 + (l/32)*4 + r%4][column l%32].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace leap {
namespace gemm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4g __attribute__((ext_vector_type(4)));

constexpr int kBM = 256;
constexpr int kBN = 256;
constexpr int kBK = 32;
constexpr int kStages = 4;
constexpr int kThreads = 256;
constexpr int kTileBytes = kBM * kBK * 2;        // one operand k-tile in LDS (16 KiB)
constexpr int kStageBytes = 2 * kTileBytes;      // A and B
constexpr int kLdsBytes = kStages * kStageBytes;  // 128 KiB
// Word 3 of a raw gfx9 buffer descriptor (32-bit data format, no swizzle).
constexpr int kGemmBufferFlags = 0x00020000;
constexpr int kXcds = 8;
#ifndef LEAP_GEMM_GROUP_M
#define LEAP_GEMM_GROUP_M 4
#endif
constexpr int kGroupM = LEAP_GEMM_GROUP_M;

// Byte offset of chunk c (16 bytes) of row r inside an LDS operand tile.
__device__ __forceinline__ int lds_off(int r, int c) { return (r << 6) + ((c ^ ((r >> 2) & 3)) << 4); }

// s_waitcnt on vmcnt <= n only (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left at their "no wait" maxima).
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt((n & 0xf) | (((n >> 4) & 3) << 14) | (0x7 << 4) | (0xf << 8));
}

// Row and column of accumulator register r of lane l inside a 32 x 32 tile.
__device__ __forceinline__ int acc_row(int r, int lane) { return ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3); }
__device__ __forceinline__ int acc_col(int lane) { return lane & 31; }

struct Tile {
    int tm, tn;  // tile coordinates
    int wm, wn;  // wave coordinates inside the tile (0..1 each)
    int lane;
    // first row / column of the wave's 128 x 128 block
    __device__ int row0() const { return tm * kBM + wm * 128; }
    __device__ int col0() const { return tn * kBN + wn * 128; }
};

// Tile order.  Workgroup b runs on XCD b % 8 and each XCD starts its
// workgroups in increasing b, so XCD x is given the contiguous range
// [x * per, (x + 1) * per) of a grouped order: GROUP consecutive M-tiles are
// walked for each N-tile before the next N-tile.  The ~32 workgroups an XCD
// runs at once then cover GROUP x (32 / GROUP) tiles and fetch only that many
// A and B k-tiles per k-step into the XCD's L2.
template <int GROUP>
__device__ __forceinline__ bool tile_of_block(int tiles_m, int tiles_n, int& tm, int& tn) {
    const int total = tiles_m * tiles_n;
    const int per = (total + kXcds - 1) / kXcds;
    const int b = blockIdx.x;
    const int t = (b % kXcds) * per + b / kXcds;
    if (t >= total) return false;
    const int in_group = GROUP * tiles_n;
    const int g = t / in_group;
    const int first_m = g * GROUP;
    const int gm = (tiles_m - first_m) < GROUP ? (tiles_m - first_m) : GROUP;
    const int r = t - g * in_group;
    tm = first_m + r % gm;
    tn = r / gm;
    return true;
}

inline int gemm_grid(int tiles_m, int tiles_n) {
    const int total = tiles_m * tiles_n;
    const int per = (total + kXcds - 1) / kXcds;
    return per * kXcds;
}

// The k-loop; leaves the wave's 4 x 4 accumulator tiles in acc.  Requires
// K % 32 == 0, lda and ldb multiples of 8, and each operand within 4 GiB of
// its base (a_bytes, b_bytes: the readable extent; rows past it read as 0).
__device__ __forceinline__ void mainloop(const uint16_t* __restrict__ A, int64_t lda,
                                         uint32_t a_bytes, const uint16_t* __restrict__ B,
                                         int64_t ldb, uint32_t b_bytes, int K, int tm, int tn,
                                         uint8_t* smem, f32x16 (&acc)[4][4]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

    // DMA mapping: instruction q (0..3) of wave w fills rows (4w + q)*16 ..
    // +15 of a 256-row operand tile, 1 KiB; lane l writes row +l/4, LDS
    // position l%4, which holds chunk (l%4) ^ ((row >> 2) & 3) of that row.
    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(A), 0, a_bytes, kGemmBufferFlags);
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(B), 0, b_bytes, kGemmBufferFlags);
    uint32_t voff_a[4], voff_b[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int r = (wave * 4 + q) * 16 + (lane >> 2);
        const int c = (lane & 3) ^ ((r >> 2) & 3);
        voff_a[q] = static_cast<uint32_t>((static_cast<int64_t>(tm) * kBM + r) * lda * 2 + c * 16);
        voff_b[q] = static_cast<uint32_t>((static_cast<int64_t>(tn) * kBN + r) * ldb * 2 + c * 16);
    }
    auto issue = [&](int kt) {
        uint8_t* st = smem + (kt % kStages) * kStageBytes;
        const int koff = kt * kBK * 2;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                ra, (__attribute__((address_space(3))) void*)(st + (wave * 4 + q) * 1024), 16,
                voff_a[q], koff, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rb, (__attribute__((address_space(3))) void*)(st + kTileBytes + (wave * 4 + q) * 1024),
                16, voff_b[q], koff, 0, 0);
        }
    };
    auto compute = [&](int kt) {
        const uint8_t* sa = smem + (kt % kStages) * kStageBytes;
        const uint8_t* sb = sa + kTileBytes;
#pragma unroll
        for (int s = 0; s < kBK / 16; ++s) {
            const int c = 2 * s + (lane >> 5);
            bf16x8 af[4], bf[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                af[i] = *reinterpret_cast<const bf16x8*>(sa + lds_off(wm * 128 + i * 32 + (lane & 31), c));
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bf[j] = *reinterpret_cast<const bf16x8*>(sb + lds_off(wn * 128 + j * 32 + (lane & 31), c));
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
        }
    };

    // Each issue() is 8 loads per wave; before multiplying k-tile kt a wave
    // lets the (up to two) later k-tiles' loads stay in flight, then the
    // barrier makes every wave's part of stage kt visible.  The stage
    // refilled after the barrier held k-tile kt - 1, which every wave has
    // finished reading by then.
    const int KT = K / kBK;
    for (int p = 0; p < kStages - 1 && p < KT; ++p) issue(p);
    for (int kt = 0; kt < KT; ++kt) {
        const int later = KT - 1 - kt;
        if (later >= 2)
            wait_vmcnt<16>();
        else if (later == 1)
            wait_vmcnt<8>();
        else
            wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();
        if (kt + kStages - 1 < KT) issue(kt + kStages - 1);
        compute(kt);
    }
    // the epilogue may reuse the LDS
    __builtin_amdgcn_s_barrier();
}

// One kernel per epilogue.  The epilogue gets the accumulators, the tile and
// the (idle) LDS buffer; it is called after the last barrier of the k-loop.
template <class Epi>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1))) void
gemm_nt_kernel(const uint16_t* __restrict__ A, int64_t lda, uint32_t a_bytes,
               const uint16_t* __restrict__ B, int64_t ldb, uint32_t b_bytes, int K, int tiles_m,
               int tiles_n, Epi epi) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
    int tm, tn;
    if (!tile_of_block<kGroupM>(tiles_m, tiles_n, tm, tn)) return;
    f32x16 acc[4][4];
    mainloop(A, lda, a_bytes, B, ldb, b_bytes, K, tm, tn, smem, acc);
    const int wave = threadIdx.x >> 6;
    Tile t{tm, tn, wave >> 1, wave & 1, static_cast<int>(threadIdx.x & 63)};
    epi(acc, t, smem);
}

}  // namespace gemm
}  // namespace leap
