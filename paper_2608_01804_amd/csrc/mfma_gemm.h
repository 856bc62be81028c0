// bf16 "NT" GEMM core on gfx950 MFMA: C[M][N] = sum_k A[m][k] * B[n][k], with
// A [M][lda] and B [N][ldb] both contiguous along k, fp32 accumulation, and
// the result handed to an epilogue functor instead of being stored.
//
//  * Workgroup tile 256 x 256, k-tiles of 64, 256 lanes = 4 waves in a 2 x 2
//    grid, each wave a 128 x 128 block of 4 x 4 v_mfma_f32_32x32x16_bf16
//    tiles (256 fp32 accumulators per lane, one wave per SIMD).
//  * Operand k-tiles go straight from HBM to LDS (buffer_load_dwordx4 ... lds,
//    no VGPR staging); each row's 128-byte k-segment is one cache line
//    fetched by one instruction.  LDS holds two A slots and three B slots of
//    32 KiB (160 KiB): A k-tiles are loaded one k-tile ahead, B k-tiles two.
//    The compiler does not track these LDS writes, so each wave waits on its
//    own vmcnt before the stage barrier.
//  * The per-CU vector memory path moves about 32 bytes per clock, which is
//    what a 256 x 256 bf16 tile consumes at the full MFMA rate, and a wave
//    whose load cannot be accepted stalls its MFMA stream too.  So the 16
//    loads of a k-tile are spread one per four MFMAs over the whole k-tile
//    (second half of A(kt+1), then B(kt+2), then after the barrier the first
//    half of A(kt+2)), and the fragments of the next k = 16 sub-step are read
//    from LDS two per four MFMAs, in fenced groups of
//    [2 MFMA | load | 2 LDS reads + 2 MFMA].
//  * LDS rows are 128 bytes (64 bf16); the 16-byte chunk c of row r sits at
//    position c ^ ((r >> 1) & 7), so the 16-row MFMA fragment reads hit
//    distinct banks, and every load instruction fills 1 KiB contiguously.
//  * The wave index is made wave-uniform (readfirstlane) so every LDS
//    destination of the loads is computed in scalar registers and written to
//    M0 directly; a per-load v_readfirstlane into M0 stalls the MFMA stream.
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
constexpr int kASlots = 2;  // A k-tiles in LDS
constexpr int kBSlots = 3;  // B k-tiles in LDS
constexpr int kThreads = 256;
constexpr int kTileBytes = kBM * kBK * 2;        // one operand k-tile in LDS (32 KiB)
constexpr int kLdsBytes = (kASlots + kBSlots) * kTileBytes;  // 160 KiB
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
    // wave-uniform by construction; readfirstlane lets the compiler keep
    // the LDS destinations of the loads (M0) in scalar registers instead of
    // a v_readfirstlane per load, which costs ~12% of the MFMA issue rate
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(A), 0, a_bytes, kGemmBufferFlags);
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(B), 0, b_bytes, kGemmBufferFlags);
    // zero extent: loads through it fetch nothing and deliver zeros; used for
    // the slots past the last k-tile so every path issues the same stream
    const __amdgpu_buffer_rsrc_t rz =
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
    const int KT = K / kBK;
    // load q of A k-tile kt into its slot kt % 2 (zeros past the last k-tile)
    auto dma_a = [&](int kt, int q) {
        const bool live = kt < KT;
        uint8_t* st = smem + (kt & 1) * kTileBytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            live ? ra : rz, (__attribute__((address_space(3))) void*)(st + (wave * 8 + q) * 1024), 16,
            voff_a[q], (live ? kt : 0) * kBK * 2, 0, 0);
    };
    // load q of B k-tile kt into B slot `slot` (== kt % 3)
    auto dma_b = [&](int kt, int slot, int q) {
        const bool live = kt < KT;
        uint8_t* st = smem + (kASlots + slot) * kTileBytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            live ? rb : rz, (__attribute__((address_space(3))) void*)(st + (wave * 8 + q) * 1024), 16,
            voff_b[q], (live ? kt : 0) * kBK * 2, 0, 0);
    };
    // fragment f of sub-step s (f < 4: A rows block f; else B columns block f - 4)
    auto read1 = [&](int as, int bsl, int s, int f, bf16x8(&af)[4], bf16x8(&bf)[4]) {
        const int c = 2 * s + (lane >> 5);
        if (f < 4) {
            const uint8_t* sa = smem + as * kTileBytes;
            af[f] = *reinterpret_cast<const bf16x8*>(sa + lds_off(wm * 128 + f * 32 + (lane & 31), c));
        } else {
            const uint8_t* sb = smem + (kASlots + bsl) * kTileBytes;
            bf[f - 4] = *reinterpret_cast<const bf16x8*>(sb + lds_off(wn * 128 + (f - 4) * 32 + (lane & 31), c));
        }
    };
    // The 16 MFMAs of one sub-step on (xa, xb); meanwhile the fragments of
    // the next sub-step s into (ya, yb) (s < 0: none) and the four loads
    // dma(0..3), in four fenced groups [2 MFMA | load | 2 reads + 2 MFMA].
    // The wait first: the fragments in use were read a sub-step ago.
    auto batch = [&](const bf16x8(&xa)[4], const bf16x8(&xb)[4], int as, int bsl, int s,
                     bf16x8(&ya)[4], bf16x8(&yb)[4], auto&& dma) {
        wait_lgkmcnt0();
#pragma unroll
        for (int g = 0; g < 4; ++g) {
#pragma unroll
            for (int u = 0; u < 2; ++u)
                acc[g][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[g], xb[u], acc[g][u], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            dma(g);
            __builtin_amdgcn_sched_barrier(0);
            if (s >= 0) {
                read1(as, bsl, s, 2 * g, ya, yb);
                read1(as, bsl, s, 2 * g + 1, ya, yb);
            }
#pragma unroll
            for (int u = 2; u < 4; ++u)
                acc[g][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[g], xb[u], acc[g][u], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // A k-tile t in A slot t % 2, B k-tile t in B slot t % 3.  Per k-tile kt:
    // batch 1 loads the second half of A(kt+1), batches 2-3 load B(kt+2),
    // batch 4 (after the barrier) loads the first half of A(kt+2).
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_a(0, q);
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_b(0, 0, q);
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_b(1, 1, q);
#pragma unroll
    for (int q = 0; q < 4; ++q) dma_a(1, q);
    wait_vmcnt<12>();  // A(0), B(0) landed; B(1) and half of A(1) may fly
    stage_barrier();
    bf16x8 a0[4], b0[4], a1[4], b1[4];
    wait_lgkmcnt0();
#pragma unroll
    for (int f = 0; f < 8; ++f) read1(0, 0, 0, f, a0, b0);
    int bs = 0;  // B slot of k-tile kt
    for (int kt = 0; kt + 1 < KT; ++kt) {
        const int as = kt & 1;
        const int b2 = bs == 0 ? 2 : bs - 1;  // slot of B(kt+2) == slot of B(kt-1)
        const int bn = bs == 2 ? 0 : bs + 1;
        batch(a0, b0, as, bs, 1, a1, b1, [&](int g) { dma_a(kt + 1, 4 + g); });
        batch(a1, b1, as, bs, 2, a0, b0, [&](int g) { dma_b(kt + 2, b2, g); });
        batch(a0, b0, as, bs, 3, a1, b1, [&](int g) { dma_b(kt + 2, b2, 4 + g); });
        // A(kt+1) and B(kt+1) have landed (only B(kt+2) may still fly); after
        // the barrier A slot kt % 2 and B slot kt % 3 are free
        wait_vmcnt<8>();
        stage_barrier();
        batch(a1, b1, as ^ 1, bn, 0, a0, b0, [&](int g) { dma_a(kt + 2, g); });
        bs = bn;
    }
    {
        const int as = (KT - 1) & 1;
        auto none = [&](int) {};
        batch(a0, b0, as, bs, 1, a1, b1, none);
        batch(a1, b1, as, bs, 2, a0, b0, none);
        batch(a0, b0, as, bs, 3, a1, b1, none);
        batch(a1, b1, as, bs, -1, a0, b0, none);
    }
    // the zero-filling loads of the slots past the end have landed and every
    // wave is past its LDS reads: the epilogue may reuse the LDS
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
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    Tile t{tm, tn, wave >> 1, wave & 1, static_cast<int>(threadIdx.x & 63)};
    epi(acc, t, smem);
}

}  // namespace gemm
}  // namespace leap
