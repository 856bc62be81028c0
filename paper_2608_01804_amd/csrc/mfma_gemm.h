// bf16 "NT" GEMM core on gfx950 MFMA: C[M][N] = sum_k A[m][k] * B[n][k], with
// A [M][lda] and B [N][ldb] both contiguous along k, fp32 accumulation, and
// the result handed to an epilogue functor instead of being stored.
//
//  * Workgroup tile 256 x 256, k-tiles of 64, 256 lanes = 4 waves in a 2 x 2
//    grid, each wave a 128 x 128 block of 8 x 8 v_mfma_f32_16x16x32_bf16
//    tiles (256 fp32 accumulators per lane, one wave per SIMD).  Under the
//    chip's power limit this shape runs at a higher clock than 32x32x16 for
//    the same work (half the accumulator traffic per flop).
//  * Operand k-tiles go straight from HBM to LDS (buffer_load_dwordx4 ... lds,
//    no VGPR staging); each row's 128-byte k-segment is one cache line
//    fetched by one instruction.  LDS holds two A slots and three B slots of
//    32 KiB (160 KiB): A k-tiles are loaded one k-tile ahead, B k-tiles two.
//    The compiler does not track these LDS writes, so each wave waits on its
//    own vmcnt before the stage barrier.
//  * A k-tile is two k = 32 steps of 64 MFMAs.  The stage barrier sits
//    between them: step 0 streams in B(kt+2) and reads the step-1 fragments
//    of the same slots; after the barrier, step 1 streams A(kt+2) into the
//    A slot just freed and reads the step-0 fragments of k-tile kt+1.  Within
//    a step the 8 x 8 blocks run row by row: one load per row, the next
//    step's B fragments in rows 0-3 (into the second B register set), and the
//    next A fragment of row i right after row i, into the registers row i
//    has just finished with.
//  * LDS rows are 128 bytes (64 bf16); the 16-byte chunk c of row r sits at
//    position c ^ ((r >> 1) & 7), so the 16-row fragment reads hit distinct
//    banks and every load instruction fills 1 KiB contiguously.  The swizzle
//    term does not depend on the 16-row block, so the 8 fragment reads of a
//    step use one base register and immediate offsets.
//  * The wave index and the LDS slot bases are wave-uniform scalars
//    (readfirstlane): the loads' LDS destinations go to M0 from scalar
//    registers, and no vector address arithmetic sits between the MFMAs.
//    The k-loop runs two k-tiles per iteration, so the A slot base is a
//    compile-time part of the fragment reads' immediate offsets.
//  * Tiles are numbered so the workgroups one XCD runs at once form a compact
//    GROUP x (32 / GROUP) patch (see tile_of_block).
//
//  * A may instead be stored k-major ([K][lda], contiguous along m; AKM): its
//    k-tile is 64 LDS rows of 512 bytes (256 m), chunk c of row r at
//    c ^ (2 * ((r & 3) | ((r >> 3 & 1) << 2))), and each A fragment is two
//    ds_read_b64_tr_b16 (4 k each), which transpose 4 x 4 bf16 blocks
//    across each 16-lane group on the way out of the LDS.  The swizzle term
//    does depend on the 16-row block there, so each lane keeps 8 precomputed
//    fragment addresses, and the k-loop stays rolled (unrolled, the compiler
//    moved the accumulators between AGPRs every iteration).
//
// v_mfma_f32_16x16x32_bf16 (lane l of 64): A row l%16 with k = 8*(l/16) .. +7;
// B column l%16 with the same k; accumulator register r holds
// C[row 4*(l/16) + r][column l%16].  So acc[i][j][r] of lane l is
// C[row0 + 16 i + 4 (l / 16) + r][col0 + 16 j + l % 16] of the wave's block.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace leap {
namespace gemm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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

// Row and column of accumulator register r of lane l inside a 16 x 16 block.
__device__ __forceinline__ int acc_row(int r, int lane) { return ((lane >> 4) << 2) + r; }
__device__ __forceinline__ int acc_col(int lane) { return lane & 15; }

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
__device__ __forceinline__ bool tile_of_block(int b, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int total = tiles_m * tiles_n;
    const int per = (total + kXcds - 1) / kXcds;
    // a grid sized for more tiles than a run-time extent leaves: the blocks
    // past each XCD's share have nothing to do
    if (b / kXcds >= per) return false;
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

// The k-loop; leaves the wave's 8 x 8 accumulator blocks in acc.  Requires
// K % 64 == 0, lda and ldb multiples of 8, and every row offset the tiles
// reach ((tiles * 256) * ld * 2 bytes) below 4 GiB; a_bytes / b_bytes are the
// readable extents (rows past them read as 0).  With AKM, A is [K][lda] and
// every m-tile must lie inside a row (tiles_m * 256 <= lda).  On return every
// load has landed and every wave is past its last LDS read, so the epilogue
// may use the LDS.
//
// ds_read_b64_tr_b16, per 16-lane group: lane i receives element i % 4 of the
// 4-element (8-byte) rows that lanes i / 4, i / 4 + 4, i / 4 + 8 and
// i / 4 + 12 point at, in that order.  With lane 4e + q pointing at k-row
// k0 + e, columns m0 + 4q .. +3, lane i receives column m0 + i of k-rows
// k0 .. k0 + 3: the first (or second) half of an MFMA A fragment.
__device__ __forceinline__ uint32_t akm_swizzle(int r) {
    return static_cast<uint32_t>(((r & 3) | (((r >> 3) & 1) << 2)) << 1);
}

// A compile-time int (an LDS slot index known to the unrolled k-loop).
template <int V>
struct IntC {
    static constexpr int value = V;
};

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ bf16x8 read_a_km(const uint8_t* p) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * 512));
    const s16x8 both = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    return __builtin_bit_cast(bf16x8, both);
}

template <bool AKM>
__device__ __forceinline__ void mainloop(const uint16_t* __restrict__ A, int64_t lda,
                                         uint32_t a_bytes, const uint16_t* __restrict__ B,
                                         int64_t ldb, uint32_t b_bytes, int K, int tm, int tn,
                                         uint8_t* smem, f32x4 (&acc)[8][8]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;

#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{};

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
    // AKM: instruction q fills k-rows 2(8w + q) and +1; lane l writes k-row
    // +l/32 at position l%32, which holds chunk (l%32) ^ akm_swizzle(row).
    uint32_t voff_a[8], voff_b[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int r = (wave * 8 + q) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        if (AKM) {
            const int kr = 2 * (wave * 8 + q) + (lane >> 5);
            const int ca = static_cast<int>((lane & 31) ^ akm_swizzle(kr));
            voff_a[q] = static_cast<uint32_t>(static_cast<int64_t>(kr) * lda * 2 +
                                              (static_cast<int64_t>(tm) * kBM + ca * 8) * 2);
        } else {
            voff_a[q] = static_cast<uint32_t>((static_cast<int64_t>(tm) * kBM + r) * lda * 2 + c * 16);
        }
        voff_b[q] = static_cast<uint32_t>((static_cast<int64_t>(tn) * kBN + r) * ldb * 2 + c * 16);
    }
    // byte offset of A k-tile kt from k-tile 0
    const uint32_t a_kstep = AKM ? static_cast<uint32_t>(kBK * lda * 2) : kBK * 2;
    const int KT = K / kBK;
    // load q of A k-tile kt into its slot kt % 2 (zeros past the last k-tile)
    auto dma_a = [&](int kt, int q) {
        const bool live = kt < KT;
        uint8_t* st = smem + (kt & 1) * kTileBytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            live ? ra : rz, (__attribute__((address_space(3))) void*)(st + (wave * 8 + q) * 1024), 16,
            voff_a[q], (live ? kt : 0) * a_kstep, 0, 0);
    };
    // load q of B k-tile kt into B slot `slot` (== kt % 3)
    auto dma_b = [&](int kt, int slot, int q) {
        const bool live = kt < KT;
        uint8_t* st = smem + (kASlots + slot) * kTileBytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            live ? rb : rz, (__attribute__((address_space(3))) void*)(st + (wave * 8 + q) * 1024), 16,
            voff_b[q], (live ? kt : 0) * kBK * 2, 0, 0);
    };
    // Fragment f of step s: row wm*128 + 16f + l%16 (A) or wn*128 + 16f + l%16
    // (B), chunk 4s + l/16.  The swizzle term ((row >> 1) & 7) is the same for
    // every f, so fragment f sits f * 2048 bytes past fragment 0.
    const int lr = lane & 15, lc = lane >> 4;
    uint32_t lane_a[2], lane_b[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int pos = ((4 * s + lc) ^ ((lr >> 1) & 7)) << 4;
        lane_a[s] = static_cast<uint32_t>((wm * 128 + lr) * 128 + pos);
        lane_b[s] = static_cast<uint32_t>((wn * 128 + lr) * 128 + pos);
    }
    // AKM fragment f of step s, first half: lane 4e + q of group g points at
    // k-row 32s + 8g + e, columns wm*128 + 16f + 4q .. +3, i.e. chunk
    // wm*16 + 2f + q/2 (half q%2), swizzled by akm_swizzle(8g + e); the step
    // adds 32 rows (16 KiB), the second half 4 rows (2 KiB).
    uint32_t lane_akm[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) {
        const int e = lr >> 2, q = lr & 3;
        const int kr = 8 * lc + e;
        const uint32_t chunk = static_cast<uint32_t>(wm * 16 + 2 * f + (q >> 1)) ^ akm_swizzle(kr);
        lane_akm[f] = static_cast<uint32_t>(kr * 512) + chunk * 16 + static_cast<uint32_t>((q & 1) * 8);
    }
    auto read_a = [&](const uint8_t* slot, int s, int f) -> bf16x8 {
        if (AKM) return read_a_km(slot + lane_akm[f] + s * 16384);
        return *reinterpret_cast<const bf16x8*>(slot + lane_a[s] + f * 2048);
    };
    bf16x8 fa[8], fb0[8], fb1[8];
    // One k = 32 step: 64 MFMAs on (fa, xb), row by row over the 8 x 8
    // blocks.  Meanwhile the fragments of step s of the slots (as, bsl) (s < 0:
    // none): B into yb during rows 0-3, A block i into fa right after row i;
    // and the loads dma(i), one per row, after the row's second MFMA.
    // The A slot is a compile-time IntC inside the unrolled k-loop (its base
    // folds into the reads' immediate offsets) and a run-time int in the
    // tail; the B slot is always a run-time int.  Run-time slot bases are
    // opaque scalars: one vector add per step, and the 8 reads per operand
    // then use immediate offsets.
    auto step = [&](const bf16x8(&xb)[8], bf16x8(&yb)[8], auto as, int bsl, int s, auto&& dma) {
        const uint8_t* pas;
        if constexpr (std::is_integral<decltype(as)>::value)
            pas = smem + __builtin_amdgcn_readfirstlane(as * kTileBytes);
        else
            pas = smem + decltype(as)::value * kTileBytes;
        const uint32_t b_base = __builtin_amdgcn_readfirstlane((kASlots + bsl) * kTileBytes);
        const uint8_t* pb = smem + (b_base + lane_b[s < 0 ? 0 : s]);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], xb[j], acc[i][j], 0, 0, 0);
                if (j == 1) {
                    __builtin_amdgcn_sched_barrier(0);
                    dma(i);
                    __builtin_amdgcn_sched_barrier(0);
                    if (s >= 0 && i < 4) {
                        yb[2 * i] = *reinterpret_cast<const bf16x8*>(pb + (2 * i) * 2048);
                        yb[2 * i + 1] = *reinterpret_cast<const bf16x8*>(pb + (2 * i + 1) * 2048);
                    }
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            if (s >= 0) fa[i] = read_a(pas, s, i);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // A k-tile t in A slot t % 2, B k-tile t in B slot t % 3.
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_a(0, q);
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_b(0, 0, q);
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_b(1, 1, q);
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_a(1, q);
    wait_vmcnt<16>();  // A(0), B(0) landed; B(1) and A(1) may fly
    stage_barrier();
    {
        const uint8_t* pb = smem + kASlots * kTileBytes + lane_b[0];
#pragma unroll
        for (int f = 0; f < 8; ++f) {
            fa[f] = read_a(smem, 0, f);
            fb0[f] = *reinterpret_cast<const bf16x8*>(pb + f * 2048);
        }
    }
    int bs = 0;  // B slot of k-tile kt
    // one k-tile kt (not the last); as_a: its A slot kt % 2, an IntC or an int
    auto ktile = [&](int kt, auto as_a, auto as_b) {
        const int b2 = bs == 0 ? 2 : bs - 1;  // slot of B(kt+2) == slot of B(kt-1)
        const int bn = bs == 2 ? 0 : bs + 1;
        // step 0: step-1 fragments of the same slots; B(kt+2) streams in
        step(fb0, fb1, as_a, bs, 1, [&](int i) { dma_b(kt + 2, b2, i); });
        // k-tile kt+1 has landed (only B(kt+2) may still fly); after the
        // barrier A slot kt % 2 and B slot kt % 3 are free
        wait_vmcnt<8>();
        stage_barrier();
        // step 1: step-0 fragments of k-tile kt+1; A(kt+2) into A slot kt % 2
        step(fb1, fb0, as_b, bn, 0, [&](int i) { dma_a(kt + 2, i); });
        bs = bn;
    };
    int kt = 0;
    if constexpr (AKM) {
        // the k-major reads keep run-time slot bases: unrolled, this loop
        // measured 21% slower
        for (; kt + 1 < KT; ++kt) ktile(kt, kt & 1, (kt & 1) ^ 1);
    } else {
        // unrolled by two: the A slot bases become immediate offsets (2-4%
        // faster on every NT pass)
        for (; kt + 2 < KT; kt += 2) {
            ktile(kt, IntC<0>{}, IntC<1>{});
            ktile(kt + 1, IntC<1>{}, IntC<0>{});
        }
        if (kt + 1 < KT) ktile(kt, IntC<0>{}, IntC<1>{});
    }
    {
        const int as = (KT - 1) & 1;
        auto none = [&](int) {};
        step(fb0, fb1, as, bs, 1, none);
        step(fb1, fb0, as, bs, -1, none);
    }
    // the zero-filling loads of the slots past the end have landed and every
    // wave is past its LDS reads: the epilogue may reuse the LDS
    wait_vmcnt<0>();
    stage_barrier();
}

// A run-time extent of M or K: a count that only the device knows (the rows
// a compaction kernel kept), read by every workgroup at launch.  The grid and
// the static tiles_m / K are sized for the largest count; the run-time one is
// clamped to them.  M: tiles_m = max(min_units, ceil(count / 256)); K: K =
// 64 * max(min_units, ceil(count / 64)).
struct DynDim {
    const int32_t* count;  // nullptr: static extents
    int k_dim;             // 0: the count sets M, 1: it sets K
    int min_units;         // least number of M tiles or k-tiles
};

// One kernel per epilogue and A layout.  The epilogue gets the accumulators,
// the tile and the (idle) LDS buffer; it is called after the last barrier of
// the k-loop.  (Written out in the kernel body: the same steps behind an
// inlined device function made the compiler move the accumulators between
// AGPRs in the k-loop and spill them.)
template <class Epi, bool AKM = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1))) void
gemm_nt_kernel(const uint16_t* __restrict__ A, int64_t lda, uint32_t a_bytes,
               const uint16_t* __restrict__ B, int64_t ldb, uint32_t b_bytes, int K, int tiles_m,
               int tiles_n, Epi epi, DynDim dyn) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
    if (dyn.count) {
        const int n = *dyn.count;
        if (dyn.k_dim) {
            const int kt = max((n + kBK - 1) / kBK, dyn.min_units);
            K = min(K, kt * kBK);
        } else {
            tiles_m = min(tiles_m, max((n + kBM - 1) / kBM, dyn.min_units));
        }
    }
    int tm, tn;
    if (!tile_of_block<kGroupM>(blockIdx.x, tiles_m, tiles_n, tm, tn)) return;
    f32x4 acc[8][8];
    mainloop<AKM>(A, lda, a_bytes, B, ldb, b_bytes, K, tm, tn, smem, acc);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    Tile t{tm, tn, wave >> 1, wave & 1, static_cast<int>(threadIdx.x & 63)};
    epi(acc, t, smem);
}

}  // namespace gemm
}  // namespace leap
