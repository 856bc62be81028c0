// Fused per-token GRPO objective and logits gradient (Sec. 3.1, Eq. 3 per
// token), over bf16 [rows x vocab] logits.
//
// Design (gfx950, wave64):
//  * One workgroup per row.  For V up to 196608 the whole row is held in
//    VGPRs: each lane owns CH 16-byte chunks (8 bf16 each) at chunk index
//    j*BLOCK + lane, so every load and store instruction of a wave covers
//    1 KiB of contiguous HBM, and the row is read from HBM exactly once.
//    Buffer instructions address the row through one descriptor, so a lane
//    keeps one 32-bit offset instead of a 64-bit address per chunk.
//  * Pass A (registers only): the lane maximum with v_pk_max_f16 applied to
//    the raw bf16 words.  For finite values below 2^121 in magnitude the
//    fp16 reading of a bf16 bit pattern orders like the bf16 value, and the
//    bf16 -inf pattern reads as a quiet NaN, which the max ignores.
//  * Pass B (registers only): e = 2^(x*c - m_lane*c) with c = log2(e)/T
//    (one transcendental per element for the whole kernel), summed in fp32,
//    and re-packed as fp16 into the registers that held the logits (e is in
//    [0, 1]).
//  * One (max, sum) merge across the workgroup: wave butterfly, per-wave
//    partials through LDS, and the same butterfly in every wave, so all
//    threads hold bitwise identical values.  Every thread then evaluates the
//    scalar per-token epilogue (log-prob, ratio, clipped surrogate, KL,
//    dloss/dlogp) redundantly.
//  * Pass C: dlogits = scale_lane * e with v_fma_mix_f32 reading the fp16
//    value directly, packed to bf16 with v_cvt_pk_bf16_f32 (RNE) and stored
//    16 bytes at a time; the token's own column gets g * (1 - p_y).
//  * Rows with zero weight are not read: their dlogits row is zero-filled.
//  * Larger vocabularies use a streaming variant that re-reads the row.
// The per-row weighted losses go to a workspace and a single-workgroup
// kernel sums them in a fixed order (bitwise reproducible).
#include "leap_common.h"

namespace leap {
namespace {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;
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

struct Params {
    float eps_lo, eps_hi, kl_coef, inv_temp;
    int kl_type;
};

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

// Per-token scalar epilogue.  lse2 = log2 sum_v 2^(x_v * c).
struct RowOut {
    float logp, loss, g, lse2;
};

// Hardware exp2 / log2 (v_exp_f32, v_log_f32, about 1 ulp): no polynomial
// constants, which would otherwise be hoisted into registers in the
// persistent row loop.
__device__ __forceinline__ float hw_exp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

__device__ __forceinline__ RowOut row_epilogue(float lse2, float xy, float old_lp, float ref_lp,
                                               float A, float w, const Params& p) {
    RowOut o;
    const float lse = lse2 * kLn2;
    const float logp = p.inv_temp * xy - lse;
    const float rho = hw_exp(logp - old_lp);
    const float clipped = fminf(fmaxf(rho, 1.0f - p.eps_lo), 1.0f + p.eps_hi);
    const float surr = fminf(rho * A, clipped * A);
    float kl, dkl;
    if (p.kl_type == LEAP_KL_K1) {
        kl = logp - ref_lp;
        dkl = 1.0f;
    } else if (p.kl_type == LEAP_KL_K2) {
        const float dd = logp - ref_lp;
        kl = 0.5f * dd * dd;
        dkl = dd;
    } else {
        const float dd = ref_lp - logp;
        const float em1 = hw_exp(dd) - 1.0f;
        kl = em1 - dd;
        dkl = -em1;
    }
    const bool active = (A > 0.0f && rho <= 1.0f + p.eps_hi) || (A < 0.0f && rho >= 1.0f - p.eps_lo);
    const float dl = (active ? -A * rho : 0.0f) + p.kl_coef * dkl;
    o.logp = logp;
    o.loss = -surr + p.kl_coef * kl;
    o.g = w * dl * p.inv_temp;
    o.lse2 = lse2;
    return o;
}

// Zero the dlogits row of an excluded token.
template <int BLOCK>
__device__ __forceinline__ void zero_row(uint16_t* drow, int V, int tid) {
    const int nfull = V >> 3;
    u32x4* d4 = reinterpret_cast<u32x4*>(drow);
    for (int c = tid; c < nfull; c += BLOCK) d4[c] = u32x4_of(0u, 0u, 0u, 0u);
    for (int e = (nfull << 3) + tid; e < V; e += BLOCK) drow[e] = 0;
}

__device__ __forceinline__ void write_row_outputs(int64_t row, float logp, float loss, float w,
                                                  float* logp_out, float* tok_loss_out,
                                                  float* row_loss) {
    if (logp_out) logp_out[row] = logp;
    if (tok_loss_out) tok_loss_out[row] = loss;
    row_loss[row] = w * loss;
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

// ---------------------------------------------------------------------------
// Register-resident, persistent variant: BLOCK threads x CH chunks x 8
// columns >= V.  Slots j < SAFE are full for every V this instantiation is
// picked for (BLOCK*SAFE < number of chunks), so only the trailing slots
// carry range checks.
// ---------------------------------------------------------------------------
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

template <int BLOCK, int CH, int SAFE>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void
grpo_rows_resident(const uint16_t* logits, int64_t ld, int V,
                   const int32_t* __restrict__ token_ids, const float* __restrict__ old_logp,
                   const float* __restrict__ ref_logp, const float* __restrict__ adv_tok,
                   const float* __restrict__ w_tok, Params p, float* __restrict__ logp_out,
                   float* __restrict__ tok_loss_out, float* __restrict__ row_loss,
                   uint16_t* dlogits, int32_t* __restrict__ dev_err) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    const int tid = threadIdx.x;
    const int lane16 = tid * 16;
    const int64_t row = blockIdx.x;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
    const uint16_t* xrow = logits + row * ld;
    uint16_t* drow = dlogits + row * ld;

    const float w = w_tok[row];
    const int y = token_ids[row];
    if (!row_live(w, y, V)) {
        if (tid == 0) {
            if (w != 0.0f) count_error(dev_err);  // token id out of range
            write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
        }
        zero_row<BLOCK>(drow, V, tid);
        return;
    }

    // The whole row into registers: one read of HBM.
    u32x4 x[CH];
    load_row<BLOCK, CH, SAFE>(x, xrow, nchunks, lane16);
    const float xy = __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
    // Only the trailing slots can reach past the row: empty slots and the
    // columns >= V of a partial chunk become -inf.
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

    // Pass A: lane maximum over the raw bf16 words.
    uint32_t mh = kNegInfPair;
#pragma unroll
    for (int j = 0; j < CH; ++j)
        mh = pk_max_f16(pk_max_f16(mh, x[j].x), pk_max_f16(x[j].y, pk_max_f16(x[j].z, x[j].w)));
    const float m = fmaxf(max_half_to_f32(mh), max_half_to_f32(mh >> 16));

    // Keep the bf16 words as the only live copy of the row.
#pragma unroll
    for (int j = 0; j < CH; ++j) asm volatile("" : "+v"(x[j]));

    // Pass B: e = 2^(x c - m c) summed in fp32 and kept as fp16 in place.
    // Chunk j's inputs are tied to chunk j-1's output so about one chunk of
    // fp32 temporaries is live at once.
    const float c2 = kLog2e * p.inv_temp;
    const float mc = (m == -INFINITY) ? 0.0f : m * c2;
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (j > 0) asm volatile("" : "+v"(x[j]) : "v"(x[j - 1]));
        uint32_t wv[4] = {x[j].x, x[j].y, x[j].z, x[j].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float a = __builtin_amdgcn_exp2f(fmaf(bf_lo(wv[q]), c2, -mc));
            const float b = __builtin_amdgcn_exp2f(fmaf(bf_hi(wv[q]), c2, -mc));
            s += a;
            s += b;
            wv[q] = pack_f16(a, b);
        }
        x[j] = u32x4_of(wv[0], wv[1], wv[2], wv[3]);
    }

    float M = (m == -INFINITY) ? -INFINITY : mc;
    float S = s;
    block_ms_reduce<BLOCK>(M, S, s_m, s_s, tid);
    if (M == -INFINITY) {  // every logit of the row is -inf
        if (tid == 0) {
            count_error(dev_err);
            write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
        }
        zero_row<BLOCK>(drow, V, tid);
        return;
    }
    const float lse2 = M + __builtin_amdgcn_logf(S);
    const RowOut o = row_epilogue(lse2, xy, old_logp[row], ref_logp[row], adv_tok[row], w, p);

    // Pass C: dlogits = -g * p_v = sc * e_v; the token's column gets g (1 - p_y).
    const float sc = -o.g * __builtin_amdgcn_exp2f(mc - lse2);
    const float dy = o.g * (1.0f - hw_exp(o.logp));
    const int cy_rel = (y >> 3) - tid;  // chunk of the token, relative to this lane
    const int ey = y & 7;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, nfull * 16);
    u32x4 prev = u32x4_of(0u, 0u, 0u, 0u);
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        asm volatile("" : "+v"(x[j]) : "v"(prev));
        const uint32_t wv[4] = {x[j].x, x[j].y, x[j].z, x[j].w};
        float d[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            d[2 * q] = mix_lo(wv[q], sc);
            d[2 * q + 1] = mix_hi(wv[q], sc);
        }
        if (cy_rel == j * BLOCK) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e == ey) d[e] = dy;
        }
        const u32x4 out = u32x4_of(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]),
                                   pack_bf16(d[4], d[5]), pack_bf16(d[6], d[7]));
        if (j < SAFE || tid < nfull - j * BLOCK) {
            store_chunk<BLOCK, SAFE>(out, rd, lane16, j);
        } else if (tid == nfull - j * BLOCK && nfull != nchunks) {  // partial last chunk
            const int c = j * BLOCK + tid;
            const int rem = V & 7;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e < rem)
                    drow[(c << 3) + e] = static_cast<uint16_t>(pack_bf16(d[e], 0.0f) & 0xffffu);
        }
        prev = out;
    }
    if (tid == 0) write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
}

// ---------------------------------------------------------------------------
// Streaming variant for any V: online (max, sum) over the row, then a second
// read to form dlogits.  Each chunk is read and written by one thread only,
// so in-place use is safe.
// ---------------------------------------------------------------------------
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void grpo_rows_stream(
    const uint16_t* logits, int64_t ld, int V, const int32_t* __restrict__ token_ids,
    const float* __restrict__ old_logp, const float* __restrict__ ref_logp,
    const float* __restrict__ adv_tok, const float* __restrict__ w_tok, Params p,
    float* __restrict__ logp_out, float* __restrict__ tok_loss_out, float* __restrict__ row_loss,
    uint16_t* dlogits, int32_t* __restrict__ dev_err) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
    const uint16_t* xrow = logits + row * ld;
    uint16_t* drow = dlogits + row * ld;

    const float w = w_tok[row];
    const int y = token_ids[row];
    bool live = (w != 0.0f);
    if (live && (y < 0 || y >= V)) {
        if (tid == 0) count_error(dev_err);
        live = false;
    }
    if (!live) {
        zero_row<BLOCK>(drow, V, tid);
        if (tid == 0) write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
        return;
    }
    const float xy = __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
    const float c2 = kLog2e * p.inv_temp;
    const u32x4* src = reinterpret_cast<const u32x4*>(xrow);

    float m = -INFINITY, s = 0.0f;  // base-2 units
    for (int c = tid; c < nchunks; c += BLOCK) {
        u32x4 v = src[c];
        if (c == nfull) v = mask_tail(v, V & 7);
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
        float f[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            f[2 * q] = bf_lo(wv[q]) * c2;
            f[2 * q + 1] = bf_hi(wv[q]) * c2;
        }
        float cm = f[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) cm = vmax(cm, f[e]);
        if (cm == -INFINITY) continue;
        if (cm > m) {
            s = (m == -INFINITY) ? 0.0f : s * exp2f(m - cm);
            m = cm;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) s += exp2f(f[e] - m);
    }
    float M = m, S = s;
    block_ms_reduce<BLOCK>(M, S, s_m, s_s, tid);
    if (M == -INFINITY) {
        if (tid == 0) count_error(dev_err);
        zero_row<BLOCK>(drow, V, tid);
        if (tid == 0) write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
        return;
    }
    const float lse2 = M + log2f(S);
    const RowOut o = row_epilogue(lse2, xy, old_logp[row], ref_logp[row], adv_tok[row], w, p);
    const float dy = o.g * (1.0f - expf(o.logp));
    const int cy = y >> 3;
    const int ey = y & 7;
    u32x4* dst = reinterpret_cast<u32x4*>(drow);
    for (int c = tid; c < nchunks; c += BLOCK) {
        const u32x4 v = src[c];
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
        float d[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            d[2 * q] = -o.g * exp2f(fmaf(bf_lo(wv[q]), c2, -lse2));
            d[2 * q + 1] = -o.g * exp2f(fmaf(bf_hi(wv[q]), c2, -lse2));
        }
        if (c == cy) d[ey] = dy;
        if (c < nfull) {
            dst[c] = u32x4_of(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]), pack_bf16(d[4], d[5]),
                                pack_bf16(d[6], d[7]));
        } else {
            const int rem = V & 7;
            for (int e = 0; e < rem; ++e)
                drow[(c << 3) + e] = static_cast<uint16_t>(pack_bf16(d[e], 0.0f) & 0xffffu);
        }
    }
    if (tid == 0) write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
}

// Fixed-order sum of the per-row weighted losses (one workgroup).
constexpr int kReduceBlock = 1024;

__global__ __launch_bounds__(kReduceBlock) void loss_reduce_kernel(const float* __restrict__ row_loss,
                                                                   int64_t N, float* __restrict__ loss_out) {
    __shared__ double s_w[kReduceBlock / kWave];
    const int tid = threadIdx.x;
    double acc = 0.0;
    for (int64_t k = tid; k < N; k += kReduceBlock) acc += static_cast<double>(row_loss[k]);
    acc = wave_sum_f64(acc);
    if ((tid & (kWave - 1)) == 0) s_w[tid / kWave] = acc;
    __syncthreads();
    if (tid == 0) {
        double t = 0.0;
        for (int w = 0; w < kReduceBlock / kWave; ++w) t += s_w[w];
        loss_out[0] = static_cast<float>(t);
    }
}

// ---------------------------------------------------------------------------
// Host dispatch
// ---------------------------------------------------------------------------
using RowKernel = void (*)(const uint16_t*, int64_t, int, const int32_t*, const float*,
                           const float*, const float*, const float*, Params, float*, float*,
                           float*, uint16_t*, int32_t*);

struct RowConfig {
    RowKernel fn;
    int block;
    int ch;  // 0: streaming variant
};

#define LEAP_RES(B, C, S) RowConfig{grpo_rows_resident<B, C, S>, B, C}

// Smallest resident configuration whose BLOCK*CH*8 columns cover V.  SAFE of
// each entry is the CH of the entry before it with the same BLOCK (0 for the
// first), which is what makes its leading slots provably full.
RowConfig pick_row_config(int V) {
    static const RowConfig table[] = {
        LEAP_RES(64, 1, 0),     LEAP_RES(64, 2, 1),     LEAP_RES(64, 4, 2),
        LEAP_RES(64, 8, 4),     LEAP_RES(256, 4, 0),    LEAP_RES(256, 8, 4),
        LEAP_RES(256, 12, 8),   LEAP_RES(256, 16, 12),  LEAP_RES(1024, 8, 0),
        LEAP_RES(1024, 12, 8),  LEAP_RES(1024, 16, 12), LEAP_RES(1024, 19, 16),
        LEAP_RES(1024, 20, 19), LEAP_RES(1024, 24, 20),
    };
    const int64_t nchunks = (static_cast<int64_t>(V) + 7) / 8;
    for (const RowConfig& r : table)
        if (static_cast<int64_t>(r.block) * r.ch >= nchunks) return r;
    return RowConfig{grpo_rows_stream<1024>, 1024, 0};
}

#undef LEAP_RES

}  // namespace
}  // namespace leap

LEAP_API size_t leap_grpo_workspace_size(int64_t N, int32_t V) {
    (void)V;
    // one fp32 weighted loss per row, in whole 256-byte lines
    const size_t b = static_cast<size_t>(N > 0 ? N : 1) * sizeof(float);
    return (b + 255) & ~static_cast<size_t>(255);
}

LEAP_API leap_status leap_grpo_logprob_loss_fwd_bwd(
    const void* logits_bf16, int64_t ld, int64_t N, int32_t V, const int32_t* token_ids,
    const float* old_logp, const float* ref_logp, const float* adv_tok, const float* w_tok,
    const leap_grpo_params* params, float* logp_out, float* tok_loss_out, float* loss_out,
    void* dlogits_bf16, void* workspace, size_t ws_bytes, int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    if (N < 0 || V < 1 || ld < V || !params || !loss_out) return LEAP_ERR_INVALID_ARG;
    const leap_grpo_params& pp = *params;
    if (!(pp.clip_eps_low >= 0.0f) || !(pp.clip_eps_high >= 0.0f) || !(pp.kl_coef >= 0.0f) ||
        !(pp.inv_temperature > 0.0f) || !__builtin_isfinite(pp.clip_eps_low) ||
        !__builtin_isfinite(pp.clip_eps_high) || !__builtin_isfinite(pp.kl_coef) ||
        !__builtin_isfinite(pp.inv_temperature))
        return LEAP_ERR_INVALID_ARG;
    if (pp.kl_type != LEAP_KL_K3 && pp.kl_type != LEAP_KL_K1 && pp.kl_type != LEAP_KL_K2)
        return LEAP_ERR_UNSUPPORTED;
    if (N > 0) {
        if (!logits_bf16 || !dlogits_bf16 || !token_ids || !old_logp || !ref_logp || !adv_tok ||
            !w_tok)
            return LEAP_ERR_INVALID_ARG;
        if (!aligned16(logits_bf16) || !aligned16(dlogits_bf16) || (ld & 7) != 0)
            return LEAP_ERR_MISALIGNED;
        if (N > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
        // dlogits must be logits itself or not overlap it.
        const uintptr_t a0 = reinterpret_cast<uintptr_t>(logits_bf16);
        const uintptr_t b0 = reinterpret_cast<uintptr_t>(dlogits_bf16);
        const uintptr_t bytes = static_cast<uintptr_t>(N) * static_cast<uintptr_t>(ld) * 2u;
        if (a0 != b0 && a0 < b0 + bytes && b0 < a0 + bytes) return LEAP_ERR_INVALID_ARG;
    }
    if (!workspace || ws_bytes < leap_grpo_workspace_size(N, V)) return LEAP_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 3u) != 0) return LEAP_ERR_MISALIGNED;

    const Params p{pp.clip_eps_low, pp.clip_eps_high, pp.kl_coef, pp.inv_temperature, pp.kl_type};
    float* row_loss = static_cast<float*>(workspace);
    if (N > 0) {
        const RowConfig rc = pick_row_config(V);
        hipLaunchKernelGGL(rc.fn, dim3(static_cast<unsigned>(N)), dim3(rc.block), 0, stream,
                           static_cast<const uint16_t*>(logits_bf16), ld, V, token_ids, old_logp,
                           ref_logp, adv_tok, w_tok, p, logp_out, tok_loss_out, row_loss,
                           static_cast<uint16_t*>(dlogits_bf16), dev_err);
        const leap_status st = launch_status();
        if (st != LEAP_OK) return st;
    }
    hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(kReduceBlock), 0, stream, row_loss, N,
                       loss_out);
    return launch_status();
}
