// Row-reduction helpers shared by the libleap row kernels (gfx950, wave64):
// bf16 / fp16 packing, buffer-descriptor row access, the (max, sum-exp)
// merge in base-2 units and its wave / workgroup reductions.
#pragma once

#include "leap_common.h"
#include "objective.h"

namespace leap {
namespace row {

using obj::kLog2e;
using obj::kLn2;
using obj::Params;
constexpr uint32_t kNegInfBf16 = 0xFF80u;
constexpr uint32_t kNegInfPair = 0xFF80FF80u;
// Word 3 of a raw gfx9 buffer descriptor (32-bit data format, no swizzle).
constexpr int kBufferFlags = 0x00020000;
// Cache policies of the row loads and of the dlogits stores (buffer
// instruction aux bits: 0 = default, 2 = non-temporal).
constexpr int kLoadPolicy = 2;
constexpr int kStorePolicy = 2;

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf162v __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 u32x4_of(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
    u32x4 v = {a, b, c, d};
    return v;
}
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
    half2v h = {static_cast<_Float16>(a), static_cast<_Float16>(b)};
    return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    float2v f = {a, b};
    bf162v h = __builtin_convertvector(f, bf162v);
    return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ float f16_lo(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(half2v, w).x);
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(half2v, w).y);
}

// Replace the columns >= rem of a partial chunk by bf16 -inf.
__device__ __forceinline__ u32x4 mask_tail(u32x4 v, int rem) {
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (2 * q >= rem) w[q] = (w[q] & 0xffff0000u) | kNegInfBf16;
        if (2 * q + 1 >= rem) w[q] = (w[q] & 0x0000ffffu) | (kNegInfBf16 << 16);
    }
    return u32x4_of(w[0], w[1], w[2], w[3]);
}

// (m, s) pairs in base-2 units: s * 2^m.  Symmetric, so a butterfly leaves
// identical values in both lanes of every exchange.
__device__ __forceinline__ void ms_merge(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    if (M == -INFINITY) return;
    s = s * __builtin_amdgcn_exp2f(m - M) + s2 * __builtin_amdgcn_exp2f(m2 - M);
    m = M;
}

__device__ __forceinline__ void wave_ms_reduce(float& m, float& s) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o, kWave);
        const float s2 = __shfl_xor(s, o, kWave);
        ms_merge(m, s, m2, s2);
    }
}

// Block-wide (m, s) merge; every thread returns the same values.  The
// per-wave partials go through LDS and every wave then runs the same 64-lane
// butterfly over them (lanes past the wave count hold the identity
// (-inf, 0)), so the merge order is fixed and all waves agree bitwise.
template <int BLOCK>
__device__ __forceinline__ void block_ms_reduce(float& m, float& s, float* s_m, float* s_s,
                                                int tid) {
    constexpr int NW = BLOCK / kWave;
    wave_ms_reduce(m, s);
    if (NW == 1) return;
    const int lane = tid & (kWave - 1);
    if (lane == 0) {
        s_m[tid / kWave] = m;
        s_s[tid / kWave] = s;
    }
    __syncthreads();
    m = (lane < NW) ? s_m[lane] : -INFINITY;
    s = (lane < NW) ? s_s[lane] : 0.0f;
    wave_ms_reduce(m, s);
}

// Exponents below this give 2^d == 0 in fp32; clamping -inf to it keeps the
// entropy sum's products 2^d * d finite (0) without changing any 2^d.
constexpr float kMinExp2Arg = -256.0f;

// (m, s, t) triples in base-2 units for the entropy: s = sum 2^d and
// t = sum 2^d * d over the elements' exponents d relative to m.  Moving the
// reference from m to M >= m scales both by 2^(m - M) and adds (m - M) * s
// to t.  A side with m == -inf holds no element and adds nothing.  Symmetric
// like ms_merge.
__device__ __forceinline__ void mst_merge(float& m, float& s, float& t, float m2, float s2,
                                          float t2) {
    const float M = fmaxf(m, m2);
    if (M == -INFINITY) return;
    const float e1 = __builtin_amdgcn_exp2f(m - M);
    const float e2 = __builtin_amdgcn_exp2f(m2 - M);
    const float t1 = (m == -INFINITY) ? 0.0f : (t + (m - M) * s) * e1;
    const float u2 = (m2 == -INFINITY) ? 0.0f : (t2 + (m2 - M) * s2) * e2;
    t = t1 + u2;
    s = s * e1 + s2 * e2;
    m = M;
}

__device__ __forceinline__ void wave_mst_reduce(float& m, float& s, float& t) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o, kWave);
        const float s2 = __shfl_xor(s, o, kWave);
        const float t2 = __shfl_xor(t, o, kWave);
        mst_merge(m, s, t, m2, s2, t2);
    }
}

// Block-wide (m, s, t) merge, in the fixed order of block_ms_reduce.
template <int BLOCK>
__device__ __forceinline__ void block_mst_reduce(float& m, float& s, float& t, float* s_m,
                                                 float* s_s, float* s_t, int tid) {
    constexpr int NW = BLOCK / kWave;
    wave_mst_reduce(m, s, t);
    if (NW == 1) return;
    const int lane = tid & (kWave - 1);
    if (lane == 0) {
        s_m[tid / kWave] = m;
        s_s[tid / kWave] = s;
        s_t[tid / kWave] = t;
    }
    __syncthreads();
    m = (lane < NW) ? s_m[lane] : -INFINITY;
    s = (lane < NW) ? s_s[lane] : 0.0f;
    t = (lane < NW) ? s_t[lane] : 0.0f;
    wave_mst_reduce(m, s, t);
}

// Entropy in nats of a row from its merged (M, S, T): with p = 2^d / S,
// H = -sum p ln p = ln 2 * (log2 S - T / S).
__device__ __forceinline__ float entropy_of(float S, float T) {
    return kLn2 * (__builtin_amdgcn_logf(S) - T / S);
}

// Elementwise max of two packed fp16 pairs (maxNum: a quiet NaN operand is
// ignored).  Applied to raw bf16 words it orders them like their bf16 values
// for finite magnitudes below 2^121; the bf16 -inf pattern reads as a NaN.
__device__ __forceinline__ uint32_t pk_max_f16(uint32_t a, uint32_t b) {
    uint32_t d;
    asm("v_pk_max_f16 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
    return d;
}

// fp16 half of a packed word times s, in fp32 (v_fma_mix_f32 reads the fp16
// operand directly).
__device__ __forceinline__ float mix_lo(uint32_t h2, float s) {
    float d;
    asm("v_fma_mix_f32 %0, %1, %2, 0 op_sel_hi:[1,0,0]" : "=v"(d) : "v"(h2), "v"(s));
    return d;
}
__device__ __forceinline__ float mix_hi(uint32_t h2, float s) {
    float d;
    asm("v_fma_mix_f32 %0, %1, %2, 0 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(d) : "v"(h2),
        "v"(s));
    return d;
}

// fp16 bit pattern of a lane maximum -> the bf16 value it stands for, as
// fp32; a NaN pattern means the lane saw no finite value (-inf).
__device__ __forceinline__ float max_half_to_f32(uint32_t h) {
    h &= 0xffffu;
    if ((h & 0x7c00u) == 0x7c00u && (h & 0x03ffu) != 0u) return -INFINITY;
    return __uint_as_float(h << 16);
}

__device__ __forceinline__ bool row_live(float w, int y, int V) {
    return w != 0.0f && y >= 0 && y < V;
}

// Chunk j of a lane.  Slots below SAFE are in the row for every V the
// instantiation serves, so their slot offset goes in the scalar offset and
// all of them share one VGPR lane offset; trailing slots put the whole offset
// in the VGPR, where the descriptor's range check applies (a load past the
// row returns 0, a store past it is dropped).
template <int BLOCK, int SAFE>
__device__ __forceinline__ u32x4 load_chunk(__amdgpu_buffer_rsrc_t rs, int lane16, int j) {
    if (j < SAFE) return __builtin_amdgcn_raw_buffer_load_b128(rs, lane16, j * BLOCK * 16, kLoadPolicy);
    return __builtin_amdgcn_raw_buffer_load_b128(rs, lane16 + j * BLOCK * 16, 0, kLoadPolicy);
}

template <int BLOCK, int SAFE>
__device__ __forceinline__ void store_chunk(u32x4 v, __amdgpu_buffer_rsrc_t rs, int lane16, int j) {
    if (j < SAFE)
        __builtin_amdgcn_raw_buffer_store_b128(v, rs, lane16, j * BLOCK * 16, kStorePolicy);
    else
        __builtin_amdgcn_raw_buffer_store_b128(v, rs, lane16 + j * BLOCK * 16, 0, kStorePolicy);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const uint16_t* row, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(row), 0, bytes, kBufferFlags);
}

template <int BLOCK, int CH, int SAFE>
__device__ __forceinline__ void load_row(u32x4 (&x)[CH], const uint16_t* xrow, int nchunks,
                                         int lane16) {
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(xrow, nchunks * 16);
#pragma unroll
    for (int j = 0; j < CH; ++j) x[j] = load_chunk<BLOCK, SAFE>(rs, lane16, j);
}

// Empty trailing slots and the columns >= V of a partial last chunk become
// -inf.  Only slots j >= SAFE can reach past the row.
template <int BLOCK, int CH, int SAFE>
__device__ __forceinline__ void mask_row_tail(u32x4 (&x)[CH], int V, int tid) {
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
#pragma unroll
    for (int j = SAFE; j < CH; ++j) {
        if ((j + 1) * BLOCK > nfull) {
            const int c = j * BLOCK + tid;
            if (c >= nchunks)
                x[j] = u32x4_of(kNegInfPair, kNegInfPair, kNegInfPair, kNegInfPair);
            else if (c == nfull)
                x[j] = mask_tail(x[j], V & 7);
        }
    }
}

// Lane maximum of a register-resident row, over the raw bf16 words.
template <int CH>
__device__ __forceinline__ float row_lane_max(const u32x4 (&x)[CH]) {
    uint32_t mh = kNegInfPair;
#pragma unroll
    for (int j = 0; j < CH; ++j)
        mh = pk_max_f16(pk_max_f16(mh, x[j].x), pk_max_f16(x[j].y, pk_max_f16(x[j].z, x[j].w)));
    return fmaxf(max_half_to_f32(mh), max_half_to_f32(mh >> 16));
}

// Smallest register-resident configuration whose BLOCK*CH chunks cover V;
// SAFE is the CH of the entry before it with the same BLOCK (0 for the first
// of a BLOCK), which is what makes its leading slots provably full.  Index
// -1: V needs the streaming variant.
struct ResidentShape {
    int block, ch, safe;
};
constexpr ResidentShape kResidentShapes[] = {
    {64, 1, 0},     {64, 2, 1},     {64, 4, 2},     {64, 8, 4},     {256, 4, 0},
    {256, 8, 4},    {256, 12, 8},   {256, 16, 12},  {1024, 8, 0},   {1024, 12, 8},
    {1024, 16, 12}, {1024, 19, 16}, {1024, 20, 19}, {1024, 24, 20},
};
constexpr int kNumResidentShapes = sizeof(kResidentShapes) / sizeof(kResidentShapes[0]);

inline int pick_resident_shape(int V) {
    const int64_t nchunks = (static_cast<int64_t>(V) + 7) / 8;
    for (int i = 0; i < kNumResidentShapes; ++i)
        if (static_cast<int64_t>(kResidentShapes[i].block) * kResidentShapes[i].ch >= nchunks)
            return i;
    return -1;
}

}  // namespace row
}  // namespace leap
