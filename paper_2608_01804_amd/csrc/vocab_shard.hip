// Vocabulary-parallel form of the per-token objective (Sec. 3.1, Eq. 3 per
// token) for logits split by vocabulary across devices: each shard reduces
// its columns of every row to a partial (max, sum) and, if it holds the
// rollout token, that token's logit; the partials of all shards (gathered by
// the caller) merge into the row's log-sum-exp and the same per-token
// objective as the unsharded kernel; each shard then writes its own slice of
// dlogits from the row's g and log-sum-exp.
//
//  * leap_vocab_shard_stats: one workgroup per row, the shard's row held in
//    VGPRs (the fused kernel's layout: 16-byte chunks at j*BLOCK + lane),
//    lane maximum on the raw bf16 words, one v_exp_f32 per element, one
//    workgroup (max, sum) merge; 16 bytes out per row.
//  * leap_vocab_merge_objective: one wave per row, lanes over shards, the
//    same symmetric (max, sum) butterfly; the per-token epilogue shared with
//    the fused kernel; a fixed-order reduction of the weighted loss.
//  * leap_vocab_shard_bwd: one workgroup per row streaming 16-byte chunks,
//    dlogits = g * (onehot - 2^(x c - lse2)); excluded rows are zero-filled
//    without reading the logits.
#include "objective.h"
#include "read_only_shapes.h"
#include "row_common.h"

namespace leap {
namespace {

using namespace row;
using obj::RowOut;

// Partial of one row on one shard: m2 = max(x) * c (base-2 units), s = sum
// 2^(x c - m2), zy = the token's logit when this shard holds it, owned = 1
// then (else 0).  An excluded row, or a shard whose columns are all -inf,
// gives (-inf, 0, 0, owned).
__device__ __forceinline__ void write_partial(float4* out, int64_t row, float m2, float s, float zy,
                                              float owned) {
    out[row] = make_float4(m2, s, zy, owned);
}

// ENT variants also write t = sum 2^(x c - m2) * (x c - m2) to partial_t
// (0 for an excluded row or an all -inf shard): the entropy's partial.
template <int BLOCK, int CH, int SAFE, bool ENT>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void
shard_stats_resident(const uint16_t* __restrict__ logits, int64_t ld, int V, int vocab_start,
                     const int32_t* __restrict__ token_ids, const float* __restrict__ w_tok,
                     float inv_temp, float4* __restrict__ partial, float* __restrict__ partial_t) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    __shared__ float s_t[ENT ? BLOCK / kWave : 1];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    const int yl = token_ids[row] - vocab_start;
    const bool owned = yl >= 0 && yl < V;
    if (w_tok != nullptr && w_tok[row] == 0.0f) {
        if (tid == 0) {
            write_partial(partial, row, -INFINITY, 0.0f, 0.0f, owned ? 1.0f : 0.0f);
            if (ENT) partial_t[row] = 0.0f;
        }
        return;
    }
    const uint16_t* xrow = logits + row * ld;
    u32x4 x[CH];
    load_row<BLOCK, CH, SAFE>(x, xrow, (V + 7) >> 3, tid * 16);
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
        const float zy = owned ? __uint_as_float(static_cast<uint32_t>(xrow[yl]) << 16) : 0.0f;
        write_partial(partial, row, M, M == -INFINITY ? 0.0f : S, zy, owned ? 1.0f : 0.0f);
        if (ENT) partial_t[row] = M == -INFINITY ? 0.0f : T;
    }
}

// Any shard width: online (max, sum) over the row's chunks.
template <int BLOCK, bool ENT>
__global__ __launch_bounds__(BLOCK) void shard_stats_stream(
    const uint16_t* __restrict__ logits, int64_t ld, int V, int vocab_start,
    const int32_t* __restrict__ token_ids, const float* __restrict__ w_tok, float inv_temp,
    float4* __restrict__ partial, float* __restrict__ partial_t) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    __shared__ float s_t[ENT ? BLOCK / kWave : 1];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    const int yl = token_ids[row] - vocab_start;
    const bool owned = yl >= 0 && yl < V;
    if (w_tok != nullptr && w_tok[row] == 0.0f) {
        if (tid == 0) {
            write_partial(partial, row, -INFINITY, 0.0f, 0.0f, owned ? 1.0f : 0.0f);
            if (ENT) partial_t[row] = 0.0f;
        }
        return;
    }
    const uint16_t* xrow = logits + row * ld;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
    const float c2 = kLog2e * inv_temp;
    const u32x4* src = reinterpret_cast<const u32x4*>(xrow);
    float m = -INFINITY, s = 0.0f;
    float t = 0.0f;  // ENT: sum of 2^d * d, d = f - m
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
        const float zy = owned ? __uint_as_float(static_cast<uint32_t>(xrow[yl]) << 16) : 0.0f;
        write_partial(partial, row, m, m == -INFINITY ? 0.0f : s, zy, owned ? 1.0f : 0.0f);
        if (ENT) partial_t[row] = m == -INFINITY ? 0.0f : t;
    }
}

using StatsKernel = void (*)(const uint16_t*, int64_t, int, int, const int32_t*, const float*,
                             float, float4*, float*);

struct StatsConfig {
    StatsKernel fn;      // without the entropy partial
    StatsKernel fn_ent;  // with it
    int block;
};

#define LEAP_SHARD(B, C, S) \
    StatsConfig{shard_stats_resident<B, C, S, false>, shard_stats_resident<B, C, S, true>, B},

StatsConfig pick_stats_config(int V) {
    static const StatsConfig table[] = {LEAP_READ_ONLY_SHAPES(LEAP_SHARD)};
    static_assert(sizeof(table) / sizeof(table[0]) == kNumReadOnlyShapes, "shape table");
    const int i = pick_read_only_shape(V);
    if (i < 0) return StatsConfig{shard_stats_stream<1024, false>, shard_stats_stream<1024, true>, 1024};
    return table[i];
}

#undef LEAP_SHARD

// ---------------------------------------------------------------------------
// Merge: one wave per row, lanes over shards in index order.
// ---------------------------------------------------------------------------
// ENT: the shards' entropy partials merge with their (max, sum) pairs as
// (max, sum, t) triples, and the row's entropy goes to entropy_out.
template <bool ENT>
__global__ __launch_bounds__(256) void merge_objective_kernel(
    const float4* __restrict__ partials, const float* __restrict__ partials_t, int n_shards,
    int64_t N, int V_total, const int32_t* __restrict__ token_ids,
    const float* __restrict__ old_logp, const float* __restrict__ ref_logp,
    const float* __restrict__ adv_tok, const float* __restrict__ w_tok, obj::Params p,
    float* __restrict__ logp_out, float* __restrict__ tok_loss_out,
    float* __restrict__ entropy_out, float* __restrict__ row_loss, float2* __restrict__ row_state,
    int32_t* __restrict__ dev_err) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (256 / kWave) + threadIdx.x / kWave;
    if (row >= N) return;
    const float w = w_tok[row];
    const int y = token_ids[row];
    auto exclude = [&](bool count) {
        if (lane == 0) {
            if (count) count_error(dev_err);
            obj::write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
            row_state[row] = make_float2(0.0f, INFINITY);
            if (ENT) entropy_out[row] = 0.0f;
        }
    };
    if (!row_live(w, y, V_total)) {
        exclude(w != 0.0f);  // token id out of range
        return;
    }
    float m = -INFINITY, s = 0.0f, t = 0.0f, zy = 0.0f;
    int owners = 0;
    for (int k = lane; k < n_shards; k += kWave) {
        const float4 q = partials[static_cast<int64_t>(k) * N + row];
        if constexpr (ENT)
            mst_merge(m, s, t, q.x, q.y, partials_t[static_cast<int64_t>(k) * N + row]);
        else
            ms_merge(m, s, q.x, q.y);
        if (q.w != 0.0f) {
            ++owners;
            zy += q.z;
        }
    }
    if constexpr (ENT)
        wave_mst_reduce(m, s, t);
    else
        wave_ms_reduce(m, s);
    owners = wave_sum_i32(owners);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) zy += __shfl_xor(zy, o, kWave);
    if (owners != 1 || m == -INFINITY) {  // inconsistent sharding, or every logit -inf
        exclude(true);
        return;
    }
    if (lane != 0) return;
    const float lse2 = m + __builtin_amdgcn_logf(s);
    const RowOut o = obj::row_epilogue(lse2, zy, old_logp[row], ref_logp[row], adv_tok[row], w, p);
    obj::write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
    row_state[row] = make_float2(o.g, lse2);
    if (ENT) entropy_out[row] = entropy_of(s, t);
}

// ---------------------------------------------------------------------------
// Shard backward: one workgroup per row.
// ---------------------------------------------------------------------------
constexpr int kBwdBlock = 256;
constexpr int kBwdBatch = 4;

__global__ __launch_bounds__(kBwdBlock) void shard_bwd_kernel(
    const uint16_t* logits, int64_t ld, int V, int vocab_start, const int32_t* __restrict__ token_ids,
    const float2* __restrict__ row_state, float inv_temp, uint16_t* dlogits) {
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    const float2 st = row_state[row];
    const float g = st.x, lse2 = st.y;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
    uint16_t* drow = dlogits + row * ld;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, nfull * 16);
    if (g == 0.0f) {  // excluded row (or zero weight): zeros, logits not read
        for (int c = tid; c < nchunks; c += kBwdBlock) {
            if (c < nfull) {
                __builtin_amdgcn_raw_buffer_store_b128(u32x4_of(0u, 0u, 0u, 0u), rd, c * 16, 0,
                                                       kStorePolicy);
            } else {
                for (int e = 0; e < (V & 7); ++e) drow[(c << 3) + e] = 0;
            }
        }
        return;
    }
    const uint16_t* xrow = logits + row * ld;
    // whole chunks: ld % 8 == 0 keeps the partial last chunk inside the row
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(xrow, nchunks * 16);
    const float c2 = kLog2e * inv_temp;
    const int yl = token_ids[row] - vocab_start;
    // kBwdBatch chunks per thread are loaded before any is processed, so the
    // loads of a batch are in flight together (past the row: zeros)
    for (int cb = tid; cb < nchunks; cb += kBwdBatch * kBwdBlock) {
        u32x4 vb[kBwdBatch];
#pragma unroll
        for (int b = 0; b < kBwdBatch; ++b)
            vb[b] = __builtin_amdgcn_raw_buffer_load_b128(rs, (cb + b * kBwdBlock) * 16, 0, kLoadPolicy);
#pragma unroll
        for (int b = 0; b < kBwdBatch; ++b) {
            const int c = cb + b * kBwdBlock;
            if (c >= nchunks) break;
            const uint32_t wv[4] = {vb[b].x, vb[b].y, vb[b].z, vb[b].w};
            float d[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                d[2 * q] = -g * __builtin_amdgcn_exp2f(fmaf(bf_lo(wv[q]), c2, -lse2));
                d[2 * q + 1] = -g * __builtin_amdgcn_exp2f(fmaf(bf_hi(wv[q]), c2, -lse2));
            }
            const int e0 = c << 3;
            if (yl >= e0 && yl < e0 + 8) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (e0 + e == yl) d[e] += g;
            }
            if (c < nfull) {
                const u32x4 out = u32x4_of(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]),
                                           pack_bf16(d[4], d[5]), pack_bf16(d[6], d[7]));
                __builtin_amdgcn_raw_buffer_store_b128(out, rd, c * 16, 0, kStorePolicy);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (e < (V & 7)) drow[e0 + e] = static_cast<uint16_t>(pack_bf16(d[e], 0.0f) & 0xffffu);
            }
        }
    }
}

bool params_ok(const leap_grpo_params& pp) {
    return pp.clip_eps_low >= 0.0f && pp.clip_eps_high >= 0.0f && pp.kl_coef >= 0.0f &&
           pp.inv_temperature > 0.0f && __builtin_isfinite(pp.clip_eps_low) &&
           __builtin_isfinite(pp.clip_eps_high) && __builtin_isfinite(pp.kl_coef) &&
           __builtin_isfinite(pp.inv_temperature);
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_vocab_shard_stats(const void* logits_bf16, int64_t ld, int64_t N,
                                            int32_t V_shard, int32_t vocab_start,
                                            const int32_t* token_ids, const float* w_tok,
                                            float inv_temperature, float* partial,
                                            float* partial_t, hipStream_t stream) {
    using namespace leap;
    if (N < 0 || V_shard < 1 || ld < V_shard || vocab_start < 0) return LEAP_ERR_INVALID_ARG;
    if (!(inv_temperature > 0.0f) || !__builtin_isfinite(inv_temperature))
        return LEAP_ERR_INVALID_ARG;
    if (V_shard > LEAP_MAX_V) return LEAP_ERR_UNSUPPORTED;
    if (N == 0) return LEAP_OK;
    if (!logits_bf16 || !token_ids || !partial) return LEAP_ERR_INVALID_ARG;
    if (!aligned16(logits_bf16) || (ld & 7) != 0 || !aligned16(partial)) return LEAP_ERR_MISALIGNED;
    if (N > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
    const leap::LaunchCheck lc;
    const StatsConfig sc = pick_stats_config(V_shard);
    hipLaunchKernelGGL(partial_t ? sc.fn_ent : sc.fn, dim3(static_cast<unsigned>(N)),
                       dim3(sc.block), 0, stream, static_cast<const uint16_t*>(logits_bf16), ld,
                       V_shard, vocab_start, token_ids, w_tok, inv_temperature,
                       reinterpret_cast<float4*>(partial), partial_t);
    return lc.status();
}

LEAP_API size_t leap_vocab_merge_workspace_size(int64_t N) {
    const size_t b = static_cast<size_t>(N > 0 ? N : 1) * sizeof(float);
    return (b + 255) & ~static_cast<size_t>(255);
}

LEAP_API leap_status leap_vocab_merge_objective(
    const float* partials, const float* partials_t, int32_t n_shards, int64_t N, int32_t V_total,
    const int32_t* token_ids, const float* old_logp, const float* ref_logp, const float* adv_tok,
    const float* w_tok, const leap_grpo_params* params, float* logp_out, float* tok_loss_out,
    float* entropy_out, float* loss_out, float* row_state, void* workspace, size_t ws_bytes,
    int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    if (N < 0 || n_shards < 1 || V_total < 1 || !params || !loss_out) return LEAP_ERR_INVALID_ARG;
    if (!params_ok(*params)) return LEAP_ERR_INVALID_ARG;
    const leap_grpo_params& pp = *params;
    if (pp.kl_type != LEAP_KL_K3 && pp.kl_type != LEAP_KL_K1 && pp.kl_type != LEAP_KL_K2)
        return LEAP_ERR_UNSUPPORTED;
    if (N > 0) {
        if (!partials || !token_ids || !old_logp || !ref_logp || !adv_tok || !w_tok || !row_state)
            return LEAP_ERR_INVALID_ARG;
        if (entropy_out && !partials_t) return LEAP_ERR_INVALID_ARG;
        if (!aligned16(partials) || (reinterpret_cast<uintptr_t>(row_state) & 7u) != 0)
            return LEAP_ERR_MISALIGNED;
        if (N > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
    }
    if (!workspace || ws_bytes < leap_vocab_merge_workspace_size(N)) return LEAP_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 3u) != 0) return LEAP_ERR_MISALIGNED;
    const leap::LaunchCheck lc;
    const obj::Params p{pp.clip_eps_low, pp.clip_eps_high, pp.kl_coef, pp.inv_temperature, pp.kl_type};
    float* row_loss = static_cast<float*>(workspace);
    if (N > 0) {
        hipLaunchKernelGGL(entropy_out ? merge_objective_kernel<true> : merge_objective_kernel<false>,
                           dim3(static_cast<unsigned>((N + 3) / 4)), dim3(256), 0, stream,
                           reinterpret_cast<const float4*>(partials), partials_t, n_shards, N,
                           V_total, token_ids, old_logp, ref_logp, adv_tok, w_tok, p, logp_out,
                           tok_loss_out, entropy_out, row_loss,
                           reinterpret_cast<float2*>(row_state), dev_err);
        const leap_status st = lc.status();
        if (st != LEAP_OK) return st;
    }
    hipLaunchKernelGGL(obj::loss_reduce_kernel, dim3(1), dim3(obj::kReduceBlock), 0, stream,
                       row_loss, N, loss_out);
    return lc.status();
}

LEAP_API leap_status leap_vocab_shard_bwd(const void* logits_bf16, int64_t ld, int64_t N,
                                          int32_t V_shard, int32_t vocab_start,
                                          const int32_t* token_ids, const float* row_state,
                                          float inv_temperature, void* dlogits_bf16,
                                          hipStream_t stream) {
    using namespace leap;
    if (N < 0 || V_shard < 1 || ld < V_shard || vocab_start < 0) return LEAP_ERR_INVALID_ARG;
    if (!(inv_temperature > 0.0f) || !__builtin_isfinite(inv_temperature))
        return LEAP_ERR_INVALID_ARG;
    if (V_shard > LEAP_MAX_V) return LEAP_ERR_UNSUPPORTED;
    if (N == 0) return LEAP_OK;
    if (!logits_bf16 || !token_ids || !row_state || !dlogits_bf16) return LEAP_ERR_INVALID_ARG;
    if (!aligned16(logits_bf16) || !aligned16(dlogits_bf16) || (ld & 7) != 0 ||
        (reinterpret_cast<uintptr_t>(row_state) & 7u) != 0)
        return LEAP_ERR_MISALIGNED;
    if (N > 0x7fffffff) return LEAP_ERR_INVALID_ARG;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(logits_bf16);
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(dlogits_bf16);
    const uintptr_t bytes = static_cast<uintptr_t>(N) * static_cast<uintptr_t>(ld) * 2u;
    if (a0 != b0 && a0 < b0 + bytes && b0 < a0 + bytes) return LEAP_ERR_INVALID_ARG;
    const leap::LaunchCheck lc;
    hipLaunchKernelGGL(shard_bwd_kernel, dim3(static_cast<unsigned>(N)), dim3(kBwdBlock), 0, stream,
                       static_cast<const uint16_t*>(logits_bf16), ld, V_shard, vocab_start,
                       token_ids, reinterpret_cast<const float2*>(row_state), inv_temperature,
                       static_cast<uint16_t*>(dlogits_bf16));
    return lc.status();
}
