// Fused LM head + per-token GRPO objective: the objective of Sec. 3.1 (Eq. 3
// per token: log-softmax at the rollout token, clipped importance ratio,
// reference KL) on logits z = H W^T that are never written to HBM, with the
// gradients dH = dZ W and dW = dZ^T H, where dZ = d(sum_k w_k l_k)/dz.
//
// Steps of one call, all on the caller's stream:
//  0. Excluded rows (w == 0: padding, prompt and feedback tokens) take no
//     part in the objective or the gradients, so the call drops them first:
//     a two-kernel compaction lists the live rows in order (rows[j], j <
//     n_live; -1 after) and gives the excluded rows their zero outputs.
//     Every GEMM below runs over the n_live compacted rows only; its grid is
//     sized for N and the tiles past n_live (a device count) exit at once.
//  1. The live rows of H are gathered into Hc [N_pad][H] and, for dW, into
//     Ht [H][N_pad]; W is transposed into Wt [H][V_pad] for dH (all zero
//     padded), because the GEMM core takes B contiguous along the
//     contraction index (and A either way: contiguous along it, or k-major
//     through transposing LDS reads).
//  2. Stats GEMM  Z = Hc W^T on MFMA.  Its epilogue turns every row of a
//     256 x 256 tile into a partial (max, sum 2^(z c - max)) in base-2 units
//     (c = log2(e) / T).
//  3. Combine: one wave per live row merges the row's partials in a fixed
//     order into the log-sum-exp, forms the rollout token's logit as a dot
//     product and evaluates the same per-token objective as the
//     logits-resident kernel (log-prob, ratio, surrogate, KL, loss and
//     g = w dloss/dlogp / T).  A fixed-order reduction sums the loss.
//  4. Per vocabulary chunk (32768 columns, 16384 for very large N): the Z
//     tiles are recomputed and the epilogue writes dZ = g (onehot - p) in
//     bf16, row-major [n_live rows][chunk]; then dW[chunk] = dZ^T Hc (dZ read
//     k-major) and dH (+)= dZ W[chunk] run as two more GEMMs with fp32
//     epilogues, dH scattered back to the live rows' places; the excluded
//     rows of dH are written as zeros.
// Executed work is 8 n_live H V flops (the forward GEMM is recomputed once).
#include "mfma_gemm.h"
#include "row_common.h"

namespace leap {
namespace {

using gemm::acc_row;
using gemm::acc_col;
using gemm::f32x4;
using gemm::Tile;
using obj::Params;
using obj::RowOut;
using row::bf_hi;
using row::bf_lo;
using row::ms_merge;
using row::pack_bf16;
using row::row_live;
using row::u32x4;
using row::wave_ms_reduce;

// Vocabulary columns per backward chunk: 32768 (fewer dH read-add-write
// passes, 1.2% faster than 16384 at 16384 x 151936 x 4096 for 1 GiB more
// workspace), or 16384 when a 32768-wide dZ chunk would pass the GEMM core's
// 4 GiB operand limit (N above ~65000).
constexpr int kChunkCols = 32768;
constexpr int kChunkColsNarrow = 16384;
constexpr int kTile = gemm::kBM;  // 256: rows and columns of a GEMM tile

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

template <bool B>
struct Flag {
    static constexpr bool value = B;
};

// ---------------------------------------------------------------------------
// Live-row compaction.  Live row: w != 0 (a live row with a bad token id
// stays in the list; the combine kernel counts and excludes it).  Pass 1
// counts the live rows of each segment of kSeg rows; pass 2 gives each
// segment its base (the counts before it, in order), lists its live rows in
// row order, writes the excluded rows' outputs (log-prob, per-token loss and
// weighted loss 0), and fills the list's tail with -1 up to N_pad.
// ---------------------------------------------------------------------------
constexpr int kSeg = 4096;
constexpr int kSegThreads = 256;
constexpr int kSegRowsPerThread = kSeg / kSegThreads;  // 16 consecutive rows

__device__ __forceinline__ int block_sum_256(int v, int* s_part) {
    v = wave_sum_i32(v);
    const int tid = threadIdx.x;
    __syncthreads();  // s_part may still be read by an earlier call
    if ((tid & (kWave - 1)) == 0) s_part[tid / kWave] = v;
    __syncthreads();
    return s_part[0] + s_part[1] + s_part[2] + s_part[3];
}

__global__ __launch_bounds__(kSegThreads) void live_count_kernel(const float* __restrict__ w_tok,
                                                                 int64_t N,
                                                                 int32_t* __restrict__ seg_count) {
    __shared__ int s_part[kSegThreads / kWave];
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kSeg;
    int c = 0;
    for (int i = threadIdx.x; i < kSeg; i += kSegThreads) {
        const int64_t r = r0 + i;
        if (r < N && w_tok[r] != 0.0f) ++c;
    }
    c = block_sum_256(c, s_part);
    if (threadIdx.x == 0) seg_count[blockIdx.x] = c;
}

__global__ __launch_bounds__(kSegThreads) void compact_rows_kernel(
    const float* __restrict__ w_tok, int64_t N, int64_t N_pad, const int32_t* __restrict__ seg_count,
    int n_seg, int32_t* __restrict__ rows, int32_t* __restrict__ n_live,
    float* __restrict__ logp_out, float* __restrict__ tok_loss_out, float* __restrict__ row_loss) {
    __shared__ int s_part[kSegThreads / kWave];
    __shared__ int s_scan[kSegThreads / kWave];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int b = blockIdx.x;
    int before = 0, all = 0;
    for (int i = tid; i < n_seg; i += kSegThreads) {
        const int c = seg_count[i];
        all += c;
        if (i < b) before += c;
    }
    const int base = block_sum_256(before, s_part);
    const int total = block_sum_256(all, s_part);
    // this thread's 16 consecutive rows
    const int64_t r0 = static_cast<int64_t>(b) * kSeg + static_cast<int64_t>(tid) * kSegRowsPerThread;
    uint32_t live = 0;
#pragma unroll
    for (int e = 0; e < kSegRowsPerThread; ++e) {
        const int64_t r = r0 + e;
        if (r < N && w_tok[r] != 0.0f) live |= 1u << e;
    }
    // exclusive scan of the per-thread counts over the block, in thread order
    const int cnt = __popc(live);
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int up = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += up;
    }
    if (lane == kWave - 1) s_scan[wave] = incl;
    __syncthreads();
    int pos = base + incl - cnt;
    for (int w = 0; w < wave; ++w) pos += s_scan[w];
#pragma unroll
    for (int e = 0; e < kSegRowsPerThread; ++e) {
        const int64_t r = r0 + e;
        if (r >= N) break;
        if (live & (1u << e)) {
            rows[pos++] = static_cast<int32_t>(r);
        } else {
            if (logp_out) logp_out[r] = 0.0f;
            if (tok_loss_out) tok_loss_out[r] = 0.0f;
            row_loss[r] = 0.0f;
        }
    }
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kSegThreads;
    for (int64_t j = total + static_cast<int64_t>(b) * kSegThreads + tid; j < N_pad; j += stride)
        rows[j] = -1;
    if (b == 0 && tid == 0) *n_live = total;
}

// ---------------------------------------------------------------------------
// Transpose with zero padding, optionally through a row list:
// dst[c][r] = src[s(r)][c] for r < R, and 0 for R <= r < ld_dst, for every
// c < C, where s(r) = r without a list, or s(r) = rows[r] with one (-1: a
// zero row).  With rows_out, the (gathered) rows are also written as they
// are: rows_out[r][c] = src[s(r)][c].  dst may be null (rows_out only).
// 64 x 64 tiles through LDS; C % 8 == 0.
// ---------------------------------------------------------------------------
constexpr int kTr = 64;

__global__ __launch_bounds__(256) void transpose_pad_kernel(const uint16_t* __restrict__ src,
                                                            int64_t R, int C, int64_t ld_src,
                                                            const int32_t* __restrict__ rows,
                                                            uint16_t* __restrict__ dst,
                                                            int64_t ld_dst,
                                                            uint16_t* __restrict__ rows_out,
                                                            int64_t ld_out) {
    __shared__ uint32_t t[kTr][kTr / 2 + 1];  // row r of the tile: 64 bf16 packed in pairs
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kTr;
    const int c0 = blockIdx.y * kTr;
    const int tid = threadIdx.x;
    {
        const int rr = tid >> 2, cc = (tid & 3) * 16;
        const int64_t r = r0 + rr;
        int64_t sr = -1;
        if (r < R) sr = rows ? static_cast<int64_t>(rows[r]) : r;
        u32x4 a = {0u, 0u, 0u, 0u}, b = {0u, 0u, 0u, 0u};
        if (sr >= 0) {
            const uint16_t* p = src + sr * ld_src + c0 + cc;
            if (c0 + cc < C) a = *reinterpret_cast<const u32x4*>(p);
            if (c0 + cc + 8 < C) b = *reinterpret_cast<const u32x4*>(p + 8);
        }
        if (rows_out && r < R) {
            uint16_t* q = rows_out + r * ld_out + c0 + cc;
            if (c0 + cc < C) *reinterpret_cast<u32x4*>(q) = a;
            if (c0 + cc + 8 < C) *reinterpret_cast<u32x4*>(q + 8) = b;
        }
        uint32_t* d = &t[rr][cc / 2];
        d[0] = a.x, d[1] = a.y, d[2] = a.z, d[3] = a.w;
        d[4] = b.x, d[5] = b.y, d[6] = b.z, d[7] = b.w;
    }
    if (!dst) return;  // uniform: the whole grid writes rows only
    __syncthreads();
    const int cc = tid >> 2, rr = (tid & 3) * 16;
    if (c0 + cc >= C) return;
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t lo = t[rr + 2 * e][cc >> 1], hi = t[rr + 2 * e + 1][cc >> 1];
        w[e] = (cc & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    uint16_t* q = dst + static_cast<int64_t>(c0 + cc) * ld_dst + r0 + rr;
    *reinterpret_cast<u32x4*>(q) = u32x4{w[0], w[1], w[2], w[3]};
    *reinterpret_cast<u32x4*>(q + 8) = u32x4{w[4], w[5], w[6], w[7]};
}

// Zero the rows of an [N][H] fp32 matrix whose weight is 0 (the excluded
// rows of dH); one workgroup per row, 16-byte stores (H % 64 == 0).
__global__ __launch_bounds__(256) void zero_excluded_rows_kernel(float* __restrict__ C, int H,
                                                                 const float* __restrict__ w_tok,
                                                                 int64_t N) {
    for (int64_t r = blockIdx.x; r < N; r += gridDim.x) {
        if (w_tok[r] != 0.0f) continue;
        f32x4* p = reinterpret_cast<f32x4*>(C + r * H);
        for (int c = threadIdx.x; c < H / 4; c += 256) __builtin_nontemporal_store(f32x4{}, p + c);
    }
}

__global__ __launch_bounds__(256) void fill_zero_f32_kernel(float* __restrict__ p, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
        p[i] = 0.0f;
}

// ---------------------------------------------------------------------------
// Stats epilogue.  Accumulator register r of lane l in 16 x 16 block (i, j)
// of a wave holds row 16 i + 4 (l / 16) + r, column 16 j + l % 16, so the 16
// lanes with the same l / 16 share those rows.  Per group of four row blocks
// each lane first folds its 8 columns of each of its 16 rows, then the 16
// lanes do a reduce-scatter: at every step a lane keeps half of its (max,
// sum) pairs, sends the other half to its partner and merges what it
// receives.  The partners are DPP lane moves inside each 16-lane row: mirror
// (lane i and 15 - i), half mirror (i and 7 - i within 8), then the quad
// swaps (xor 2, xor 1); the lane of each pair with bit 3, 2, 1, 0 set keeps
// the upper half, so after the four steps lane l holds the pair of one row
// over the wave's 128 columns (the row of pair index l % 16).  The two waves
// covering the same rows merge through LDS.  The rollout token's logit is
// not taken here (the combine kernel forms it as a dot product).
// ---------------------------------------------------------------------------
// (max, sum) merge without a branch: an empty side (-inf, 0) contributes
// exp2(-inf) = 0, and two empty sides give (-inf, 0).
__device__ __forceinline__ void ms_merge_sel(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    const float Ms = M == -INFINITY ? 0.0f : M;
    s = s * __builtin_amdgcn_exp2f(m - Ms) + s2 * __builtin_amdgcn_exp2f(m2 - Ms);
    m = M;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2, 3, 0, 1]
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1, 0, 3, 2]

// One reduce-scatter step over HALF pairs; the partner of lane i (by the DPP
// move CTRL) differs from it in bit log2(HALF) and agrees in the higher ones.
template <int HALF, int CTRL>
__device__ __forceinline__ void scatter_step(float (&m)[16], float (&s)[16], int lane) {
    const bool up = (lane & HALF) != 0;
#pragma unroll
    for (int k = 0; k < HALF; ++k) {
        const float sm = up ? m[k] : m[k + HALF];
        const float ss = up ? s[k] : s[k + HALF];
        float km = up ? m[k + HALF] : m[k];
        float ks = up ? s[k + HALF] : s[k];
        const float rm = dpp_f32<CTRL>(sm);
        const float rs = dpp_f32<CTRL>(ss);
        ms_merge_sel(km, ks, rm, rs);
        m[k] = km;
        s[k] = ks;
    }
}

struct StatsEpi {
    float2* part;  // [N][tiles_v] (max, sum) in base-2 units
    int64_t N;
    int V, tiles_v;
    float c2;  // log2(e) / T

    __device__ __forceinline__ void operator()(f32x4 (&acc)[8][8], const Tile& t, uint8_t* smem) const {
        // the k-loop's last barrier has every wave past its LDS reads
        float2* s_ms = reinterpret_cast<float2*>(smem);
        const int tid = threadIdx.x;
        const int64_t row0 = static_cast<int64_t>(t.tm) * kTile;
        const int lane = t.lane, c = lane & 15;
        const int col0 = t.col0();
        // Columns past V (only in the last vocabulary tile) count as -inf.
        // The max is taken on the raw accumulators (c2 > 0 keeps the order,
        // and rounding is monotonic, so m * c2 is the max of the scaled
        // values) and each term is one fma: 2^(z c2 - m c2).
        bool colok[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) colok[j] = col0 + j * 16 + c < V;
        const bool full = col0 + 128 <= V;
        auto fold = [&](float (&m)[16], float (&s)[16], int G, auto full_c) {
            constexpr bool kFull = decltype(full_c)::value;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = 4 * G + ii;
                    float z[8];
                    float mx = -INFINITY;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        z[j] = (kFull || colok[j]) ? acc[i][j][r] : -INFINITY;
                        mx = fmaxf(mx, z[j]);
                    }
                    const float m2 = mx * c2;  // -inf for an empty row part
                    const float nm = m2 == -INFINITY ? 0.0f : -m2;
                    float sum = 0.0f;
#pragma unroll
                    for (int j = 0; j < 8; ++j) sum += __builtin_amdgcn_exp2f(fmaf(z[j], c2, nm));
                    m[4 * ii + r] = m2;
                    s[4 * ii + r] = sum;
                }
        };
#pragma unroll
        for (int G = 0; G < 2; ++G) {  // row blocks 4G .. 4G+3; pair k = 4 (i - 4G) + r
            float m[16], s[16];
            if (full)
                fold(m, s, G, Flag<true>{});
            else
                fold(m, s, G, Flag<false>{});
            scatter_step<8, kDppRowMirror>(m, s, lane);
            scatter_step<4, kDppRowHalfMirror>(m, s, lane);
            scatter_step<2, kDppQuadXor2>(m, s, lane);
            scatter_step<1, kDppQuadXor1>(m, s, lane);
            {
                const int rw = t.wm * 128 + (4 * G + (c >> 2)) * 16 + acc_row(c & 3, lane);
                s_ms[t.wn * kTile + rw] = make_float2(m[0], s[0]);
            }
            // keep the next group's accumulators in AGPRs until they are used
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
        const float2 a = s_ms[tid], b = s_ms[kTile + tid];
        float M = a.x, S = a.y;
        ms_merge(M, S, b.x, b.y);
        const int64_t r = row0 + tid;
        if (r < N) part[r * tiles_v + t.tn] = make_float2(M, S);
    }
};

// ---------------------------------------------------------------------------
// Combine: one wave per row.
// ---------------------------------------------------------------------------
// Compacted row j (of n_rows = N_pad) is caller row rows[j]; the row's
// partials and its (g, lse2) are at j, its outputs at rows[j].
__global__ __launch_bounds__(256) void lm_combine_kernel(
    const float2* __restrict__ part, int tiles_v, const uint16_t* __restrict__ hidden,
    const uint16_t* __restrict__ weight, int H, const int32_t* __restrict__ rows,
    int64_t n_rows, int V, const int32_t* __restrict__ token_ids, const float* __restrict__ old_logp,
    const float* __restrict__ ref_logp, const float* __restrict__ adv_tok,
    const float* __restrict__ w_tok, Params p, float* __restrict__ logp_out,
    float* __restrict__ tok_loss_out, float* __restrict__ row_loss, float* __restrict__ g_out,
    float* __restrict__ lse2_out, float* __restrict__ dzy_out, int32_t* __restrict__ dev_err) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t j = static_cast<int64_t>(blockIdx.x) * (256 / kWave) + (threadIdx.x / kWave);
    if (j >= n_rows) return;
    // Past the live rows, and excluded tokens: g = 0 and an infinite
    // log-sum-exp make every dZ entry of the row exactly zero.
    const int64_t row = rows[j];
    if (row < 0) {
        if (lane == 0) g_out[j] = 0.0f, lse2_out[j] = INFINITY, dzy_out[j] = 0.0f;
        return;
    }
    const float w = w_tok[row];
    const int y = token_ids[row];
    if (!row_live(w, y, V)) {
        if (lane == 0) {
            if (w != 0.0f) count_error(dev_err);  // token id out of range
            obj::write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
            g_out[j] = 0.0f;
            lse2_out[j] = INFINITY;
            dzy_out[j] = 0.0f;
        }
        return;
    }
    // the rollout token's logit z_y = H[row] . W[y]: fp32 products of the
    // bf16 operands, lanes over 16-byte chunks (H % 64 == 0), a fixed-order
    // wave sum
    float zy = 0.0f;
    {
        const u32x4* hr = reinterpret_cast<const u32x4*>(hidden + row * H);
        const u32x4* wr = reinterpret_cast<const u32x4*>(weight + static_cast<int64_t>(y) * H);
        for (int c = lane; c < H / 8; c += kWave) {
            const u32x4 a = hr[c], b = wr[c];
            zy = fmaf(bf_lo(a.x), bf_lo(b.x), zy);
            zy = fmaf(bf_hi(a.x), bf_hi(b.x), zy);
            zy = fmaf(bf_lo(a.y), bf_lo(b.y), zy);
            zy = fmaf(bf_hi(a.y), bf_hi(b.y), zy);
            zy = fmaf(bf_lo(a.z), bf_lo(b.z), zy);
            zy = fmaf(bf_hi(a.z), bf_hi(b.z), zy);
            zy = fmaf(bf_lo(a.w), bf_lo(b.w), zy);
            zy = fmaf(bf_hi(a.w), bf_hi(b.w), zy);
        }
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) zy += __shfl_xor(zy, o, kWave);
    }
    float m = -INFINITY, s = 0.0f;
    for (int t = lane; t < tiles_v; t += kWave) {
        const float2 q = part[j * tiles_v + t];
        ms_merge(m, s, q.x, q.y);
    }
    wave_ms_reduce(m, s);
    if (lane != 0) return;
    if (m == -INFINITY) {  // every logit of the row is -inf
        count_error(dev_err);
        obj::write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
        g_out[j] = 0.0f;
        lse2_out[j] = INFINITY;
        dzy_out[j] = 0.0f;
        return;
    }
    const float lse2 = m + __builtin_amdgcn_logf(s);
    const RowOut o = obj::row_epilogue(lse2, zy, old_logp[row], ref_logp[row], adv_tok[row], w, p);
    obj::write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
    g_out[j] = o.g;
    lse2_out[j] = lse2;
    // the token's own dZ entry, g (1 - p_y), in fp32 from the log-prob: the
    // dZ epilogue stores it in place of -g p_y, so it keeps its relative
    // precision when p_y is close to 1
    dzy_out[j] = o.g * (1.0f - obj::hw_exp(o.logp));
}

// ---------------------------------------------------------------------------
// dZ epilogue: dz = g (onehot - 2^(z c - lse2)), zero past V, rounded to
// bf16, stored row-major with 16-byte non-temporal stores (read back only by
// the next two GEMMs, after it has left the caches anyway).  A lane holds
// rows 4h .. 4h+3 (h = lane / 16) of column l % 16 of each 16 x 16 block;
// blocks are taken in column pairs (j, j+1) and transposed through a
// per-wave LDS area: each lane writes the 4 rows of its column of both
// blocks (8 bytes each), then two ds_read_b64_tr_b16 hand lane 4q + p of
// group h row 4h + p, columns 8q .. 8q+7 of the pair (the read pointer of
// lane j is column 8 (j % 4) + j / 4, then 4 columns on).  Every element is
// first -g p; the one lane of the grid that stores a row's token column
// then replaces that element with the row's g (1 - p_y), formed in fp32 by
// the combine kernel (rounding -g p_y to bf16 first and adding g would cost
// up to 2^-9 |g|, far more than g (1 - p_y) itself when p_y is near 1).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float dpp_quad_xor1(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_quad_xor2(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
}

// In: d[e] = M[row e][column q] where q = lane % 4.  Out: d[b] = M[row q][column b].
__device__ __forceinline__ void quad_transpose(float (&d)[4], int lane) {
    const bool odd = (lane & 1) != 0;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const float recv = dpp_quad_xor1(odd ? d[2 * a] : d[2 * a + 1]);
        if (odd)
            d[2 * a] = recv;
        else
            d[2 * a + 1] = recv;
    }
    const bool hi = (lane & 2) != 0;
    const float r0 = dpp_quad_xor2(hi ? d[0] : d[2]);
    const float r1 = dpp_quad_xor2(hi ? d[1] : d[3]);
    if (hi) {
        d[0] = r0, d[1] = r1;
    } else {
        d[2] = r0, d[3] = r1;
    }
}

constexpr int kDzStageBase = 4096;  // after the per-row arrays (4 KiB)
constexpr int kDzStageBuf = 1024;   // [h][32 columns][4 rows] bf16
static_assert(kDzStageBase + 4 * 2 * kDzStageBuf <= gemm::kLdsBytes, "dZ staging exceeds the LDS");

__device__ __forceinline__ uint2 read_tr16(const uint8_t* p) {
    typedef __attribute__((address_space(3))) gemm::s16x4 lds_s16x4;
    return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p)));
}

// Element e (0..7) of 8 packed bf16 set to v (rounded to bf16).
__device__ __forceinline__ u32x4 set_element(u32x4 x, int e, float v) {
    const int wi = e >> 1;
    const bool hi = (e & 1) != 0;
    uint32_t w = wi == 0 ? x.x : wi == 1 ? x.y : wi == 2 ? x.z : x.w;
    const uint32_t nb = pack_bf16(v, 0.0f) & 0xffffu;
    w = hi ? ((w & 0xffffu) | (nb << 16)) : ((w & 0xffff0000u) | nb);
    return u32x4{wi == 0 ? w : x.x, wi == 1 ? w : x.y, wi == 2 ? w : x.z, wi == 3 ? w : x.w};
}

struct DzEpi {
    const int32_t* token_ids;  // [N], caller rows
    const int32_t* rows;       // [N_pad], compacted row -> caller row (-1: none)
    const float* lse2;         // [N_pad], compacted rows
    const float* g;            // [N_pad], compacted rows
    const float* dzy;          // [N_pad], compacted rows: the token column's g (1 - p_y)
    uint16_t* dz;              // [N_pad][ld_dz], compacted rows, chunk-local columns
    int64_t ld_dz;
    int64_t N;                 // rows of lse2 / g / rows (N_pad)
    int V, c0;  // vocabulary size, first column of the chunk
    float c2;

    __device__ __forceinline__ void operator()(f32x4 (&acc)[8][8], const Tile& t, uint8_t* smem) const {
        float* s_l = reinterpret_cast<float*>(smem);
        float* s_g = s_l + kTile;
        int* s_y = reinterpret_cast<int*>(s_g + kTile);
        float* s_dy = reinterpret_cast<float*>(s_y + kTile);
        const int tid = threadIdx.x;
        const int64_t row0 = static_cast<int64_t>(t.tm) * kTile;
        {
            const int64_t r = row0 + tid;
            if (r < N) {
                s_l[tid] = lse2[r];
                s_g[tid] = g[r];
                const int src = rows[r];
                const int y = src >= 0 ? token_ids[src] : -1;
                s_y[tid] = (y >= c0 && y < V) ? y - c0 : -1;
                s_dy[tid] = dzy[r];
            } else {
                s_l[tid] = INFINITY;
                s_g[tid] = 0.0f;
                s_y[tid] = -1;
                s_dy[tid] = 0.0f;
            }
        }
        __syncthreads();
        const int lane = t.lane, c = lane & 15, h = lane >> 4;
        const int q = c >> 2, p = c & 3;  // the lane stores row 4h + p, columns 8q .. 8q+7
        const int vw = t.col0();          // chunk-local column of the wave's block
        uint8_t* stage = smem + kDzStageBase + (t.wm * 2 + t.wn) * 2 * kDzStageBuf;
        const int wr = (h * 32 + c) * 8;
        const int rd = (h * 32 + 8 * p + q) * 8;
        // Every column of the wave's block inside the vocabulary (all but the
        // last tile of the vocabulary): no per-element range select.
        auto tile_body = [&](auto full) {
            constexpr bool kFull = decltype(full)::value;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int rb = t.wm * 128 + i * 16;  // tile row of the block
                const int rs = rb + 4 * h + p;       // the row this lane stores
                const int ys = s_y[rs];
                const float dys = s_dy[rs];
                // the lane's 4 rows: read once (the staging writes below
                // would otherwise force re-reads)
                float lr[4], ngr[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    lr[r] = s_l[rb + acc_row(r, lane)];
                    ngr[r] = -s_g[rb + acc_row(r, lane)];
                }
#pragma unroll
                for (int jp = 0; jp < 4; ++jp) {
                    uint8_t* buf = stage + (jp & 1) * kDzStageBuf;
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int v = vw + (2 * jp + e) * 16 + c;
                        const bool colok = kFull || c0 + v < V;
                        float d[4];
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float pz = __builtin_amdgcn_exp2f(acc[i][2 * jp + e][r] * c2 - lr[r]);
                            d[r] = colok ? fmaf(ngr[r], pz, 0.0f) : 0.0f;  // -g p, +0 for g = 0
                        }
                        *reinterpret_cast<uint2*>(buf + wr + e * 128) =
                            make_uint2(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]));
                    }
                    const uint2 lo = read_tr16(buf + rd), hi = read_tr16(buf + rd + 32);
                    u32x4 out = u32x4{lo.x, lo.y, hi.x, hi.y};
                    const int v0 = vw + 32 * jp + 8 * q;
                    const int off = ys - v0;  // the row's token column (chunk-local, -1: none)
                    if (static_cast<unsigned>(off) < 8u) out = set_element(out, off, dys);
                    __builtin_nontemporal_store(out, reinterpret_cast<u32x4*>(dz + (row0 + rs) * ld_dz + v0));
                }
            }
        };
        if (c0 + vw + 128 <= V)
            tile_body(Flag<true>{});
        else
            tile_body(Flag<false>{});
    }
};

// fp32 result tile into C[rows][cols] (leading dimension ldc, 16-byte aligned
// rows): stored, or added to what C holds.  The 4 x 4 transpose inside each
// lane quad gives every lane 4 consecutive columns of one row, so each store
// (and each load of the accumulating form) moves 16 bytes per lane; the
// stores are non-temporal (the result is not read again by this call, or
// only by the next chunk's accumulation).
// With row_map, result row m goes to C row row_map[m] (-1: dropped).
template <bool ACCUMULATE>
struct StoreF32Epi {
    float* C;
    int64_t ldc;
    int64_t rows;
    int cols;
    const int32_t* row_map;  // nullable

    __device__ __forceinline__ void operator()(f32x4 (&acc)[8][8], const Tile& t, uint8_t*) const {
        const int lane = t.lane;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t m = t.row0() + i * 16 + acc_row(lane & 3, lane);
            int64_t dst = m < rows ? m : -1;
            if (row_map && dst >= 0) dst = row_map[dst];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                float d[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
                quad_transpose(d, lane);  // row 4h + lane%4, columns of the lane quad
                const int n0 = t.col0() + j * 16 + (acc_col(lane) & ~3);
                if (dst < 0) continue;
                float* p = C + dst * ldc + n0;
                if (n0 + 3 < cols) {
                    float4 v = make_float4(d[0], d[1], d[2], d[3]);
                    if (ACCUMULATE) {
                        const float4 o = *reinterpret_cast<const float4*>(p);
                        v.x += o.x, v.y += o.y, v.z += o.z, v.w += o.w;
                    }
                    __builtin_nontemporal_store(f32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<f32x4*>(p));
                } else {
#pragma unroll
                    for (int b = 0; b < 4; ++b)
                        if (n0 + b < cols) p[b] = ACCUMULATE ? p[b] + d[b] : d[b];
                }
            }
        }
    }
};

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
struct Dims {
    int64_t N, N_pad;
    int V, V_pad, H, H_pad, tiles_v, Vc, n_chunks, n_seg;
};

Dims dims_of(int64_t N, int V, int H) {
    Dims d;
    d.N = N;
    d.N_pad = round_up(N > 0 ? N : 1, kTile);
    d.V = V;
    d.V_pad = static_cast<int>(round_up(V, kTile));
    d.H = H;
    d.H_pad = static_cast<int>(round_up(H, kTile));
    d.tiles_v = d.V_pad / kTile;
    const bool wide_fits = static_cast<uint64_t>(d.N_pad) * kChunkCols * 2u < (1ull << 32) - 64u;
    const int vc = wide_fits ? kChunkCols : kChunkColsNarrow;
    d.Vc = d.V_pad < vc ? d.V_pad : vc;
    d.n_chunks = (d.V_pad + d.Vc - 1) / d.Vc;
    d.n_seg = static_cast<int>((d.N_pad + kSeg - 1) / kSeg);
    return d;
}

struct Layout {
    size_t ht, hc, wt, part, lse2, g, dzy, row_loss, dz, rows, seg, n_live, total;
};

// The transposed weight Wt [H][V_pad] bf16, zero padded.
size_t wt_bytes(const Dims& d) { return static_cast<size_t>(d.H) * d.V_pad * 2; }

Layout layout_of(const Dims& d) {
    Layout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += (bytes + 255) & ~static_cast<size_t>(255);
        return at;
    };
    L.ht = take(static_cast<size_t>(d.H) * d.N_pad * 2);
    L.hc = take(static_cast<size_t>(d.N_pad) * d.H * 2);
    L.part = take(static_cast<size_t>(d.N_pad) * d.tiles_v * sizeof(float2));
    L.lse2 = take(static_cast<size_t>(d.N_pad) * 4);
    L.g = take(static_cast<size_t>(d.N_pad) * 4);
    L.dzy = take(static_cast<size_t>(d.N_pad) * 4);
    L.row_loss = take(static_cast<size_t>(d.N_pad) * 4);
    L.dz = take(static_cast<size_t>(d.N_pad) * d.Vc * 2);
    L.rows = take(static_cast<size_t>(d.N_pad) * 4);
    L.seg = take(static_cast<size_t>(d.n_seg) * 4);
    L.n_live = take(4);
    L.wt = take(wt_bytes(d));  // last: not needed with a caller's transposed weight
    L.total = off;
    return L;
}

// The GEMM core addresses each operand with 32-bit byte offsets: the last
// row any tile touches must start below 4 GiB.
bool fits32(int64_t rows_padded, int64_t ld) {
    return static_cast<uint64_t>(rows_padded) * static_cast<uint64_t>(ld) * 2u < (1ull << 32) - 64u;
}

bool shapes_fit(const Dims& d) {
    return fits32(d.N_pad, d.H) &&       // H, Hc [N_pad][H]
           fits32(d.V_pad, d.H) &&       // W   [V][H]
           fits32(d.H_pad, d.N_pad) &&   // Ht  [H][N_pad]
           fits32(d.N_pad, d.Vc) &&      // dZ  [N_pad][chunk]
           fits32(d.H_pad, d.V_pad);     // Wt  [H][V_pad]
}

uint32_t extent32(uint64_t bytes) {
    return bytes > 0xffffffffull ? 0xffffffffu : static_cast<uint32_t>(bytes);
}

// One GEMM C = A B^T: M and K are the largest extents (the grid is sized
// for them); dyn, if it has a count, shrinks M or K at run time.
template <bool AKM = false, class Epi>
leap_status gemm_nt(const uint16_t* A, int64_t lda, uint64_t a_bytes, const uint16_t* B, int64_t ldb,
                    uint64_t b_bytes, int K, int64_t M, int64_t Ncols, const Epi& epi,
                    gemm::DynDim dyn, hipStream_t stream, const LaunchCheck& lc) {
    const int tiles_m = static_cast<int>((M + kTile - 1) / kTile);
    const int tiles_n = static_cast<int>((Ncols + kTile - 1) / kTile);
    hipLaunchKernelGGL((gemm::gemm_nt_kernel<Epi, AKM>), dim3(gemm::gemm_grid(tiles_m, tiles_n)),
                       dim3(gemm::kThreads), 0, stream, A, lda, extent32(a_bytes), B, ldb,
                       extent32(b_bytes), K, tiles_m, tiles_n, epi, dyn);
    return lc.status();
}

}  // namespace
}  // namespace leap

LEAP_API size_t leap_lmhead_workspace_size(int64_t N, int32_t V, int32_t H) {
    using namespace leap;
    if (N < 0 || V < 1 || H < 1) return 0;
    return layout_of(dims_of(N, V, H)).total;
}

LEAP_API size_t leap_lmhead_weight_t_size(int32_t V, int32_t H) {
    using namespace leap;
    if (V < 1 || H < 1) return 0;
    return wt_bytes(dims_of(0, V, H));
}

LEAP_API leap_status leap_lmhead_transpose_weight(const void* weight_bf16, int32_t V, int32_t H,
                                                  void* weight_t_bf16, size_t bytes,
                                                  hipStream_t stream) {
    using namespace leap;
    if (V < 1 || H < 1 || !weight_bf16 || !weight_t_bf16) return LEAP_ERR_INVALID_ARG;
    if (H % 64 != 0) return LEAP_ERR_UNSUPPORTED;
    const Dims d = dims_of(0, V, H);
    if (!fits32(d.V_pad, d.H) || !fits32(d.H_pad, d.V_pad)) return LEAP_ERR_UNSUPPORTED;
    if (!aligned16(weight_bf16) || !aligned16(weight_t_bf16)) return LEAP_ERR_MISALIGNED;
    if (bytes < wt_bytes(d)) return LEAP_ERR_WORKSPACE;
    const leap::LaunchCheck lc;
    hipLaunchKernelGGL(transpose_pad_kernel, dim3(static_cast<unsigned>(d.V_pad / kTr), (H + kTr - 1) / kTr),
                       dim3(256), 0, stream, static_cast<const uint16_t*>(weight_bf16),
                       static_cast<int64_t>(V), H, static_cast<int64_t>(H), nullptr,
                       static_cast<uint16_t*>(weight_t_bf16), static_cast<int64_t>(d.V_pad), nullptr,
                       int64_t{0});
    return lc.status();
}

LEAP_API leap_status leap_grpo_lmhead_fwd_bwd(
    const void* hidden_bf16, const void* weight_bf16, const void* weight_t_bf16, int64_t N, int32_t V,
    int32_t H,
    const int32_t* token_ids, const float* old_logp, const float* ref_logp, const float* adv_tok,
    const float* w_tok, const leap_grpo_params* params, float* logp_out, float* tok_loss_out,
    float* loss_out, float* dhidden, float* dweight, int32_t accumulate_dweight, void* workspace,
    size_t ws_bytes, int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    if (N < 0 || N > 0x7fffffffLL - kTile || V < 1 || H < 1 || !params || !loss_out)
        return LEAP_ERR_INVALID_ARG;
    if (accumulate_dweight != 0 && accumulate_dweight != 1) return LEAP_ERR_INVALID_ARG;
    const leap_grpo_params& pp = *params;
    if (!(pp.clip_eps_low >= 0.0f) || !(pp.clip_eps_high >= 0.0f) || !(pp.kl_coef >= 0.0f) ||
        !(pp.inv_temperature > 0.0f) || !__builtin_isfinite(pp.clip_eps_low) ||
        !__builtin_isfinite(pp.clip_eps_high) || !__builtin_isfinite(pp.kl_coef) ||
        !__builtin_isfinite(pp.inv_temperature))
        return LEAP_ERR_INVALID_ARG;
    if (pp.kl_type != LEAP_KL_K3 && pp.kl_type != LEAP_KL_K1 && pp.kl_type != LEAP_KL_K2)
        return LEAP_ERR_UNSUPPORTED;
    if (H % 64 != 0) return LEAP_ERR_UNSUPPORTED;  // the GEMM core takes k-tiles of 64
    const Dims d = dims_of(N, V, H);
    if (!shapes_fit(d)) return LEAP_ERR_UNSUPPORTED;
    if (N > 0) {
        if (!hidden_bf16 || !weight_bf16 || !token_ids || !old_logp || !ref_logp || !adv_tok ||
            !w_tok)
            return LEAP_ERR_INVALID_ARG;
        if (!aligned16(hidden_bf16) || !aligned16(weight_bf16)) return LEAP_ERR_MISALIGNED;
    }
    if (!aligned16(dhidden) || !aligned16(dweight) || !aligned16(weight_t_bf16))
        return LEAP_ERR_MISALIGNED;
    const Layout L = layout_of(d);
    // a caller's transposed weight stands in for the last region
    const bool own_wt = dhidden && !weight_t_bf16;
    if (!workspace || ws_bytes < (own_wt ? L.total : L.wt)) return LEAP_ERR_WORKSPACE;
    if (!aligned16(workspace)) return LEAP_ERR_MISALIGNED;

    const leap::LaunchCheck lc;
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    uint16_t* ht = reinterpret_cast<uint16_t*>(ws + L.ht);
    uint16_t* hc = reinterpret_cast<uint16_t*>(ws + L.hc);
    const uint16_t* wt = own_wt ? reinterpret_cast<const uint16_t*>(ws + L.wt)
                                : static_cast<const uint16_t*>(weight_t_bf16);
    float2* part = reinterpret_cast<float2*>(ws + L.part);
    float* lse2 = reinterpret_cast<float*>(ws + L.lse2);
    float* g = reinterpret_cast<float*>(ws + L.g);
    float* dzy = reinterpret_cast<float*>(ws + L.dzy);
    float* row_loss = reinterpret_cast<float*>(ws + L.row_loss);
    uint16_t* dz = reinterpret_cast<uint16_t*>(ws + L.dz);
    int32_t* rows = reinterpret_cast<int32_t*>(ws + L.rows);
    int32_t* seg = reinterpret_cast<int32_t*>(ws + L.seg);
    int32_t* n_live = reinterpret_cast<int32_t*>(ws + L.n_live);
    const uint16_t* Hm = static_cast<const uint16_t*>(hidden_bf16);
    const uint16_t* Wm = static_cast<const uint16_t*>(weight_bf16);
    leap_status st;

    if (N == 0) {
        if (dweight && !accumulate_dweight) {
            hipLaunchKernelGGL(fill_zero_f32_kernel, dim3(1024), dim3(256), 0, stream, dweight,
                               static_cast<int64_t>(V) * H);
            if ((st = lc.status()) != LEAP_OK) return st;
        }
        hipLaunchKernelGGL(obj::loss_reduce_kernel, dim3(1), dim3(obj::kReduceBlock), 0, stream,
                           row_loss, int64_t{0}, loss_out);
        return lc.status();
    }

    const Params p{pp.clip_eps_low, pp.clip_eps_high, pp.kl_coef, pp.inv_temperature, pp.kl_type};
    const float c2 = obj::kLog2e * pp.inv_temperature;
    const uint64_t hc_bytes = static_cast<uint64_t>(d.N_pad) * H * 2;
    const uint64_t w_bytes = static_cast<uint64_t>(V) * H * 2;
    // M of the stats and dH passes (no tile without a live row), of the dZ
    // pass (at least one tile, so that dZ holds zeros for an empty list), K
    // of the dW pass (at least one k-tile of those rows)
    const gemm::DynDim dyn_m{n_live, 0, 0};
    const gemm::DynDim dyn_m_dz{n_live, 0, 1};
    const gemm::DynDim dyn_k{n_live, 1, 1};

    // 0. the live rows, in order; the excluded rows' outputs
    hipLaunchKernelGGL(live_count_kernel, dim3(d.n_seg), dim3(kSegThreads), 0, stream, w_tok, N, seg);
    if ((st = lc.status()) != LEAP_OK) return st;
    hipLaunchKernelGGL(compact_rows_kernel, dim3(d.n_seg), dim3(kSegThreads), 0, stream, w_tok, N,
                       d.N_pad, seg, d.n_seg, rows, n_live, logp_out, tok_loss_out, row_loss);
    if ((st = lc.status()) != LEAP_OK) return st;

    // 1. gathered and transposed operands
    hipLaunchKernelGGL(transpose_pad_kernel, dim3(static_cast<unsigned>(d.N_pad / kTr), (H + kTr - 1) / kTr),
                       dim3(256), 0, stream, Hm, d.N_pad, H, static_cast<int64_t>(H), rows,
                       dweight ? ht : nullptr, d.N_pad, hc, static_cast<int64_t>(H));
    if ((st = lc.status()) != LEAP_OK) return st;
    if (own_wt) {
        hipLaunchKernelGGL(transpose_pad_kernel, dim3(static_cast<unsigned>(d.V_pad / kTr), (H + kTr - 1) / kTr),
                           dim3(256), 0, stream, Wm, static_cast<int64_t>(V), H, static_cast<int64_t>(H),
                           nullptr, reinterpret_cast<uint16_t*>(ws + L.wt), static_cast<int64_t>(d.V_pad),
                           nullptr, int64_t{0});
        if ((st = lc.status()) != LEAP_OK) return st;
    }

    // 2. row statistics of the live rows
    {
        const StatsEpi epi{part, d.N_pad, V, d.tiles_v, c2};
        if ((st = gemm_nt(hc, H, hc_bytes, Wm, H, w_bytes, H, d.N_pad, V, epi, dyn_m, stream, lc)) !=
            LEAP_OK)
            return st;
    }
    // 3. per-token objective
    hipLaunchKernelGGL(lm_combine_kernel, dim3(static_cast<unsigned>(d.N_pad / 4)), dim3(256), 0,
                       stream, part, d.tiles_v, Hm, Wm, H, rows, d.N_pad, V, token_ids, old_logp,
                       ref_logp, adv_tok, w_tok, p, logp_out, tok_loss_out, row_loss, g, lse2, dzy,
                       dev_err);
    if ((st = lc.status()) != LEAP_OK) return st;
    hipLaunchKernelGGL(obj::loss_reduce_kernel, dim3(1), dim3(obj::kReduceBlock), 0, stream,
                       row_loss, N, loss_out);
    if ((st = lc.status()) != LEAP_OK) return st;
    if (!dhidden && !dweight) return LEAP_OK;

    // 4. gradients, one vocabulary chunk at a time
    const uint64_t dz_bytes = static_cast<uint64_t>(d.N_pad) * d.Vc * 2;
    for (int c0 = 0; c0 < V; c0 += d.Vc) {
        const int vl = (d.V_pad - c0) < d.Vc ? (d.V_pad - c0) : d.Vc;  // multiple of 256
        {
            const DzEpi epi{token_ids, rows, lse2, g, dzy, dz, d.Vc, d.N_pad, V, c0, c2};
            const uint64_t wb = static_cast<uint64_t>(V - c0) * H * 2;
            if ((st = gemm_nt(hc, H, hc_bytes, Wm + static_cast<int64_t>(c0) * H, H, wb, H, d.N_pad, vl,
                              epi, dyn_m_dz, stream, lc)) != LEAP_OK)
                return st;
        }
        if (dweight) {
            // dW[chunk] = dZ^T Hc: A = dZ read k-major ([N_pad][Vc], the
            // chunk's vl columns), K = the live rows
            const int64_t vrows = (V - c0) < vl ? (V - c0) : vl;
            float* C = dweight + static_cast<int64_t>(c0) * H;
            const uint64_t bb = static_cast<uint64_t>(H) * d.N_pad * 2;
            const int K = static_cast<int>(d.N_pad);
            st = accumulate_dweight
                     ? gemm_nt<true>(dz, d.Vc, dz_bytes, ht, d.N_pad, bb, K, vl, H,
                                     StoreF32Epi<true>{C, H, vrows, H, nullptr}, dyn_k, stream, lc)
                     : gemm_nt<true>(dz, d.Vc, dz_bytes, ht, d.N_pad, bb, K, vl, H,
                                     StoreF32Epi<false>{C, H, vrows, H, nullptr}, dyn_k, stream, lc);
            if (st != LEAP_OK) return st;
        }
        if (dhidden) {
            // dH (+)= dZ Wt[:, c0 .. c0 + vl) (B rows of V_pad, the chunk's
            // columns), each result row written to its live row's place
            const uint64_t bb = (static_cast<uint64_t>(H) * d.V_pad - c0) * 2;
            st = c0 > 0 ? gemm_nt(dz, d.Vc, dz_bytes, wt + c0, d.V_pad, bb, vl, d.N_pad, H,
                                  StoreF32Epi<true>{dhidden, H, d.N_pad, H, rows}, dyn_m, stream, lc)
                        : gemm_nt(dz, d.Vc, dz_bytes, wt + c0, d.V_pad, bb, vl, d.N_pad, H,
                                  StoreF32Epi<false>{dhidden, H, d.N_pad, H, rows}, dyn_m, stream, lc);
            if (st != LEAP_OK) return st;
        }
    }
    if (dhidden) {
        const int64_t blocks = N < 8192 ? N : 8192;
        hipLaunchKernelGGL(zero_excluded_rows_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                           stream, dhidden, H, w_tok, N);
        if ((st = lc.status()) != LEAP_OK) return st;
    }
    return LEAP_OK;
}
