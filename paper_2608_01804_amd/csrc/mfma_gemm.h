// bf16 "NT" GEMM core on gfx950 MFMA: C[M][N] = sum_k A[m][k] * B[n][k], with
// A [M][lda] and B [N][ldb] both contiguous along k, fp32 accumulation, and
// the result handed to an epilogue functor instead of being stored.
//
//  * Workgroup tile 256 x 256, k-tiles of 64, 256 lanes = 4 waves in a 2 x 2
//    grid, each wave a 128 x 128 block of 4 x 4 v_mfma_f32_32x32x16_bf16
//    tiles (256 fp32 accumulators per lane, one wave per SIMD).
//  * Operand k-tiles go straight from HBM to LDS (buffer_load_dwordx4 ... lds,
//    no VGPR staging) into two stages of 64 KiB; each row's 128-byte
//    k-segment is one cache line fetched by one instruction.  The compiler
//    does not track these LDS writes, so each wave waits on its own vmcnt
//    before the stage barrier.
//  * A k-tile is four k = 16 sub-steps; the fragments of the next sub-step
//    (across the barrier, the next k-tile's first) are read from LDS while
//    the current 16 MFMAs run, one read per two MFMAs, and the next k-tile's
//    loads are spread one per MFMA after the barrier.  The per-CU vector
//    memory path (about 32 bytes per clock) is what a 256 x 256 bf16 tile
//    needs at the full MFMA rate, so keeping loads in flight under the MFMAs
//    is what sets the achieved rate.
//  * LDS rows are 128 bytes (64 bf16); the 16-byte chunk c of row r sits at
//    position c ^ ((r >> 1) & 7), so the 16-row MFMA fragment reads hit
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
constexpr int kBK = 64;
constexpr int kStages = 2;
constexpr int kThreads = 256;
constexpr int kTileBytes = kBM * kBK * 2;        // one operand k-tile in LDS (32 KiB)
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
__device__ __forceinline__ int lds_off(int r, int c) { return (r << 7) + ((c ^ ((r >> 1) & 7)) << 4); }

// s_waitcnt on vmcnt <= n only (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left at their "no wait" maxima).
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt((n & 0xf) | (((n >> 4) & 3) << 14) | (0x7 << 4) | (0xf << 8));
}

// Wait for this wave's LDS accesses (a tracked s_waitcnt, so the compiler's
// own bookkeeping stays exact), then the workgroup barrier; the "memory"
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void wait_lgkmcnt0() {
    __builtin_amdgcn_s_waitcnt(0xf | (0x7 << 4) | (0x3 << 14));  // lgkmcnt(0) only
}
__device__ __forceinline__ void stage_barrier() {
    wait_lgkmcnt0();
    asm volatile("s_barrier" ::: "memory");
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
// K % 64 == 0, lda and ldb multiples of 8, and every row offset the tiles
// reach ((tiles * 256) * ld * 2 bytes) below 4 GiB; a_bytes / b_bytes are the
// readable extents (rows past them read as 0).  On return every load has
// landed and every wave is past its last LDS read, so the epilogue may use
// the LDS.
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

    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(A), 0, a_bytes, kGemmBufferFlags);
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(B), 0, b_bytes, kGemmBufferFlags);
    // zero extent: loads through it fetch nothing and deliver zeros
    const __amdgpu_buffer_rsrc_t r0 =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(A), 0, 0, kGemmBufferFlags);
    // DMA mapping: instruction q (0..7) of wave w fills rows (8w + q)*8 .. +7
    // of a 256-row operand tile (1 KiB, LDS-contiguous); lane l writes row
    // +l/8 at LDS position l%8, which holds chunk (l%8) ^ ((row >> 1) & 7).
    uint32_t voff_a[8], voff_b[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int r = (wave * 8 + q) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        voff_a[q] = static_cast<uint32_t>((static_cast<int64_t>(tm) * kBM + r) * lda * 2 + c * 16);
        voff_b[q] = static_cast<uint32_t>((static_cast<int64_t>(tn) * kBN + r) * ldb * 2 + c * 16);
    }
    // Loads of k-tile kt into stage `stage`; live == false sends the same
    // instructions through the zero-extent descriptor (no memory traffic),
    // which keeps the instruction stream identical on every path.
    auto issue = [&](int kt, int stage, bool live) {
        uint8_t* st = smem + stage * kStageBytes;
        const int koff = kt * kBK * 2;
        const __amdgpu_buffer_rsrc_t sa = live ? ra : r0;
        const __amdgpu_buffer_rsrc_t sb = live ? rb : r0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                sa, (__attribute__((address_space(3))) void*)(st + (wave * 8 + q) * 1024), 16,
                voff_a[q], koff, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                sb, (__attribute__((address_space(3))) void*)(st + kTileBytes + (wave * 8 + q) * 1024),
                16, voff_b[q], koff, 0, 0);
        }
    };
    auto read = [&](int stage, int s, bf16x8(&af)[4], bf16x8(&bf)[4]) {
        // the previous sub-step's fragments landed during the MFMAs since
        // they were read; waiting here keeps at most 8 LDS reads in flight
        wait_lgkmcnt0();
        const uint8_t* sa = smem + stage * kStageBytes;
        const uint8_t* sb = sa + kTileBytes;
        const int c = 2 * s + (lane >> 5);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            af[i] = *reinterpret_cast<const bf16x8*>(sa + lds_off(wm * 128 + i * 32 + (lane & 31), c));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            bf[j] = *reinterpret_cast<const bf16x8*>(sb + lds_off(wn * 128 + j * 32 + (lane & 31), c));
    };
    auto mma = [&](const bf16x8(&af)[4], const bf16x8(&bf)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    };
    // one LDS read per two MFMAs
    auto spread_reads = [&]() {
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    // k-tile kt lives in stage kt % 2; k-tile kt + 2 refills stage kt % 2
    // after the barrier that ends k-tile kt.
    const int KT = K / kBK;
    issue(0, 0, true);
    issue(KT > 1 ? 1 : 0, 1, KT > 1);
    wait_vmcnt<16>();
    stage_barrier();
    bf16x8 a0[4], b0[4], a1[4], b1[4];
    read(0, 0, a0, b0);
    for (int kt = 0; kt + 1 < KT; ++kt) {
        const int cur = kt & 1;
        read(cur, 1, a1, b1);
        mma(a0, b0);
        spread_reads();
        read(cur, 2, a0, b0);
        mma(a1, b1);
        spread_reads();
        read(cur, 3, a1, b1);
        mma(a0, b0);
        spread_reads();
        // k-tile kt + 1 has landed everywhere and stage kt % 2 is free
        wait_vmcnt<0>();
        stage_barrier();
        read(cur ^ 1, 0, a0, b0);
        issue(kt + 2 < KT ? kt + 2 : 0, cur, kt + 2 < KT);
        mma(a1, b1);
#pragma unroll
        for (int g = 0; g < 16; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (LDS DMA)
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    {
        const int cur = (KT - 1) & 1;
        read(cur, 1, a1, b1);
        mma(a0, b0);
        read(cur, 2, a0, b0);
        mma(a1, b1);
        read(cur, 3, a1, b1);
        mma(a0, b0);
        mma(a1, b1);
    }
    // the zero-filling loads of the last slot have landed, every wave is
    // past its LDS reads: the epilogue may reuse the LDS
    wait_vmcnt<0>();
    stage_barrier();
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
