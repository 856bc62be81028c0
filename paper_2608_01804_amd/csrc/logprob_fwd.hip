// Forward-only token log-probabilities: the old-policy and reference forward
// passes whose outputs enter the ratio and the KL term of the per-token
// objective (Sec. 3.1, Eq. 3).
//
// Same row layout as the fused kernel: one workgroup per row, the row held in
// VGPRs for V up to 196608 (one HBM read, lane maximum with v_pk_max_f16 on the
// raw bf16 words, one v_exp_f32 per element, one (max, sum) merge), a
// streaming online-softmax variant beyond that.  Only 2V bytes are read and 4
// written per row (8 with the optional per-row entropy, which adds a third
// accumulator t = sum 2^d * d beside the sum-exp: the ENT variants).
#include "read_only_shapes.h"
#include "row_common.h"

namespace leap {
namespace {

using namespace row;

__device__ __forceinline__ bool fwd_skip(const float* w_tok, int64_t row) {
    return w_tok != nullptr && w_tok[row] == 0.0f;
}

template <int BLOCK, int CH, int SAFE, bool ENT>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void
logprob_rows_resident(const uint16_t* __restrict__ logits, int64_t ld, int V,
                      const int32_t* __restrict__ token_ids, const float* __restrict__ w_tok,
                      float inv_temp, float* __restrict__ logp_out,
                      float* __restrict__ entropy_out, int32_t* __restrict__ dev_err) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    __shared__ float s_t[ENT ? BLOCK / kWave : 1];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    if (fwd_skip(w_tok, row)) {
        if (tid == 0) {
            logp_out[row] = 0.0f;
            if (ENT) entropy_out[row] = 0.0f;
        }
        return;
    }
    const int y = token_ids[row];
    if (y < 0 || y >= V) {
        if (tid == 0) {
            count_error(dev_err);
            logp_out[row] = __builtin_nanf("");
            if (ENT) entropy_out[row] = __builtin_nanf("");
        }
        return;
    }
    const uint16_t* xrow = logits + row * ld;
    u32x4 x[CH];
    load_row<BLOCK, CH, SAFE>(x, xrow, (V + 7) >> 3, tid * 16);
    const float xy = __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
    mask_row_tail<BLOCK, CH, SAFE>(x, V, tid);
    const float m = row_lane_max<CH>(x);

    const float c2 = kLog2e * inv_temp;
    const float mc = (m == -INFINITY) ? 0.0f : m * c2;
    float s = 0.0f;
    float t = 0.0f;  // ENT: sum of 2^d * d
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        const uint32_t wv[4] = {x[j].x, x[j].y, x[j].z, x[j].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if constexpr (ENT) {
                const float da = vmax(fmaf(bf_lo(wv[q]), c2, -mc), kMinExp2Arg);
                const float db = vmax(fmaf(bf_hi(wv[q]), c2, -mc), kMinExp2Arg);
                const float a = __builtin_amdgcn_exp2f(da);
                const float b = __builtin_amdgcn_exp2f(db);
                s += a;
                s += b;
                t = fmaf(a, da, t);
                t = fmaf(b, db, t);
            } else {
                s += __builtin_amdgcn_exp2f(fmaf(bf_lo(wv[q]), c2, -mc));
                s += __builtin_amdgcn_exp2f(fmaf(bf_hi(wv[q]), c2, -mc));
            }
        }
    }
    float M = (m == -INFINITY) ? -INFINITY : mc;
    float S = s;
    float T = t;
    if constexpr (ENT)
        block_mst_reduce<BLOCK>(M, S, T, s_m, s_s, s_t, tid);
    else
        block_ms_reduce<BLOCK>(M, S, s_m, s_s, tid);
    if (tid == 0) {
        if (M == -INFINITY) {
            count_error(dev_err);
            logp_out[row] = __builtin_nanf("");
            if (ENT) entropy_out[row] = __builtin_nanf("");
        } else {
            logp_out[row] = inv_temp * xy - (M + __builtin_amdgcn_logf(S)) * kLn2;
            if (ENT) entropy_out[row] = entropy_of(S, T);
        }
    }
}

template <int BLOCK, bool ENT>
__global__ __launch_bounds__(BLOCK) void logprob_rows_stream(
    const uint16_t* __restrict__ logits, int64_t ld, int V, const int32_t* __restrict__ token_ids,
    const float* __restrict__ w_tok, float inv_temp, float* __restrict__ logp_out,
    float* __restrict__ entropy_out, int32_t* __restrict__ dev_err) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    __shared__ float s_t[ENT ? BLOCK / kWave : 1];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    if (fwd_skip(w_tok, row)) {
        if (tid == 0) {
            logp_out[row] = 0.0f;
            if (ENT) entropy_out[row] = 0.0f;
        }
        return;
    }
    const int y = token_ids[row];
    if (y < 0 || y >= V) {
        if (tid == 0) {
            count_error(dev_err);
            logp_out[row] = __builtin_nanf("");
            if (ENT) entropy_out[row] = __builtin_nanf("");
        }
        return;
    }
    const uint16_t* xrow = logits + row * ld;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
    const float c2 = kLog2e * inv_temp;
    const u32x4* src = reinterpret_cast<const u32x4*>(xrow);
    float m = -INFINITY, s = 0.0f;  // base-2 units
    float t = 0.0f;                 // ENT: sum of 2^d * d, d = f - m
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
            if constexpr (ENT) {
                if (m == -INFINITY) {
                    t = 0.0f;
                } else {
                    const float dm = m - cm;
                    t = (t + dm * s) * __builtin_amdgcn_exp2f(dm);
                }
            }
            s = (m == -INFINITY) ? 0.0f : s * __builtin_amdgcn_exp2f(m - cm);
            m = cm;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if constexpr (ENT) {
                const float d = vmax(f[e] - m, kMinExp2Arg);
                const float a = __builtin_amdgcn_exp2f(d);
                s += a;
                t = fmaf(a, d, t);
            } else {
                s += __builtin_amdgcn_exp2f(f[e] - m);
            }
        }
    }
    if constexpr (ENT)
        block_mst_reduce<BLOCK>(m, s, t, s_m, s_s, s_t, tid);
    else
        block_ms_reduce<BLOCK>(m, s, s_m, s_s, tid);
    if (tid == 0) {
        if (m == -INFINITY) {
            count_error(dev_err);
            logp_out[row] = __builtin_nanf("");
            if (ENT) entropy_out[row] = __builtin_nanf("");
        } else {
            const float xy = __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
            logp_out[row] = inv_temp * xy - (m + __builtin_amdgcn_logf(s)) * kLn2;
            if (ENT) entropy_out[row] = entropy_of(s, t);
        }
    }
}

using FwdKernel = void (*)(const uint16_t*, int64_t, int, const int32_t*, const float*, float,
                           float*, float*, int32_t*);

struct FwdConfig {
    FwdKernel fn;      // without the entropy output
    FwdKernel fn_ent;  // with it
    int block;
};

#define LEAP_FWD(B, C, S) \
    FwdConfig{logprob_rows_resident<B, C, S, false>, logprob_rows_resident<B, C, S, true>, B},

FwdConfig pick_fwd_config(int V) {
    static const FwdConfig table[] = {LEAP_READ_ONLY_SHAPES(LEAP_FWD)};
    static_assert(sizeof(table) / sizeof(table[0]) == kNumReadOnlyShapes, "shape table");
    const int i = pick_read_only_shape(V);
    if (i < 0) return FwdConfig{logprob_rows_stream<1024, false>, logprob_rows_stream<1024, true>, 1024};
    return table[i];
}

#undef LEAP_FWD

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_logprob_fwd(const void* logits_bf16, int64_t ld, int64_t N, int32_t V,
                                      const int32_t* token_ids, const float* w_tok,
                                      float inv_temperature, float* logp_out,
                                      float* entropy_out, int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    if (N < 0 || V < 1 || ld < V) return LEAP_ERR_INVALID_ARG;
    if (!(inv_temperature > 0.0f) || !__builtin_isfinite(inv_temperature))
        return LEAP_ERR_INVALID_ARG;
    if (V > LEAP_MAX_V) return LEAP_ERR_UNSUPPORTED;
    if (N == 0) return LEAP_OK;
    if (!logits_bf16 || !token_ids || !logp_out) return LEAP_ERR_INVALID_ARG;
    if (!aligned16(logits_bf16) || (ld & 7) != 0) return LEAP_ERR_MISALIGNED;
    if (N > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
    const leap::LaunchCheck lc;
    const FwdConfig fc = pick_fwd_config(V);
    hipLaunchKernelGGL(entropy_out ? fc.fn_ent : fc.fn, dim3(static_cast<unsigned>(N)),
                       dim3(fc.block), 0, stream, static_cast<const uint16_t*>(logits_bf16), ld, V,
                       token_ids, w_tok, inv_temperature, logp_out, entropy_out, dev_err);
    return lc.status();
}
