// Fused per-token GRPO objective and logits gradient (Sec. 3.1, Eq. 3 per
// token), over bf16 [rows x vocab] logits.
//
// Design (gfx950, wave64):
//  * One workgroup holds one row at a time.  For V up to 196608 the whole row is held in
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
//  * From 55296 to 155648 columns (one workgroup per compute unit) the kernel
//    is persistent: a grid of one workgroup per CU takes rows from a row queue
//    (a counter in the workspace) and issues the next row's loads right
//    behind the current row's stores, so each CU's reads overlap its writes
//    instead of waiting for a new workgroup to be dispatched after each row,
//    and CUs that stream faster take more rows.
//  * Up to 270336 columns the part of the row past 196608 columns is held in
//    LDS (the hybrid kernel); larger vocabularies use a streaming variant
//    that re-reads the row.
// The per-row weighted losses go to a workspace and a single-workgroup
// kernel sums them in a fixed order (bitwise reproducible).
// Optional output: each row's entropy H = -sum_v p_v ln p_v (nats), from a
// third accumulator t = sum 2^d * d beside the sum-exp (the ENT variants;
// without it the kernels are unchanged).
#include <mutex>

#include "objective.h"
#include "row_common.h"

namespace leap {
namespace {

using namespace row;
using namespace obj;

// Zero the dlogits row of an excluded token: 16-byte non-temporal stores
// through a buffer descriptor over the row's whole chunks, the partial last
// chunk element by element.
template <int BLOCK>
__device__ __forceinline__ void zero_row(uint16_t* drow, int V, int tid) {
    const int nfull = V >> 3;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, nfull * 16);
    const u32x4 z = u32x4_of(0u, 0u, 0u, 0u);
    for (int c = tid; c < nfull; c += BLOCK)
        __builtin_amdgcn_raw_buffer_store_b128(z, rd, c * 16, 0, kStorePolicy);
    for (int e = (nfull << 3) + tid; e < V; e += BLOCK) drow[e] = 0;
}

// Row outputs of an excluded row (weight 0, or counted as a data error) and
// its zero-filled dlogits row.
template <int BLOCK, bool ENT>
__device__ __forceinline__ void excluded_row(int64_t row, uint16_t* drow, int V, bool count,
                                             float* logp_out, float* tok_loss_out,
                                             float* entropy_out, float* row_loss,
                                             int32_t* dev_err, int tid) {
    if (tid == 0) {
        if (count) count_error(dev_err);
        write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
        if (ENT) entropy_out[row] = 0.0f;
    }
    zero_row<BLOCK>(drow, V, tid);
}

// LDS of one block-wide (max, sum[, t]) merge.
template <int BLOCK, bool ENT>
struct RowLds {
    float m[BLOCK / kWave];
    float s[BLOCK / kWave];
    float t[ENT ? BLOCK / kWave : 1];
};

// Pass B over the register-resident chunks: e = 2^(x c - mc) summed into s
// (and e * d into t with ENT) in fp32, the values re-packed as fp16 in place.
// Chunk j's inputs are tied to chunk j-1's output so about one chunk of fp32
// temporaries is live at once.
template <int CH, bool ENT>
__device__ __forceinline__ void exp_pass_vgpr(u32x4 (&x)[CH], float c2, float mc, float& s,
                                              float& t) {
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (j > 0) asm volatile("" : "+v"(x[j]) : "v"(x[j - 1]));
        uint32_t wv[4] = {x[j].x, x[j].y, x[j].z, x[j].w};
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
                wv[q] = pack_f16(a, b);
            } else {
                const float a = __builtin_amdgcn_exp2f(fmaf(bf_lo(wv[q]), c2, -mc));
                const float b = __builtin_amdgcn_exp2f(fmaf(bf_hi(wv[q]), c2, -mc));
                s += a;
                s += b;
                wv[q] = pack_f16(a, b);
            }
        }
        x[j] = u32x4_of(wv[0], wv[1], wv[2], wv[3]);
    }
}

// Pass C over the register-resident chunks (fp16 e from pass B):
// dlogits = sc * e, the token's own column dy, bf16 (RNE), 16-byte stores;
// the partial last chunk (V % 8 columns) element by element.
template <int BLOCK, int CH, int SAFE>
__device__ __forceinline__ void dlogits_pass_vgpr(u32x4 (&x)[CH], float sc, float dy, int y,
                                                  uint16_t* drow, int V, int tid) {
    const int lane16 = tid * 16;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
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
}

// Passes A-C of one live row whose loads into x have been issued: the
// lane maximum, the exponentials (kept as fp16 in x), the block merge, the
// scalar epilogue, the dlogits stores and the row's outputs.  A row whose
// logits are all -inf is counted and zero-filled instead.  One barrier
// (inside the block merge) in every call.  With tk_slot set, thread 0
// stores *tk there after pass A, so the value is in LDS for every thread
// once the merge's barrier has passed (*tk is read in thread 0 only).
template <int BLOCK, int CH, int SAFE, bool ENT>
__device__ __forceinline__ void fused_row(u32x4 (&x)[CH], float xy, int64_t row, uint16_t* drow,
                                          int V, int y, float w, const float* __restrict__ old_logp,
                                          const float* __restrict__ ref_logp,
                                          const float* __restrict__ adv_tok, const Params& p,
                                          float* __restrict__ logp_out,
                                          float* __restrict__ tok_loss_out,
                                          float* __restrict__ entropy_out,
                                          float* __restrict__ row_loss, int32_t* __restrict__ dev_err,
                                          RowLds<BLOCK, ENT>& lds, int tid, int* tk_slot = nullptr,
                                          const int* tk = nullptr) {
    mask_row_tail<BLOCK, CH, SAFE>(x, V, tid);

    // Pass A: lane maximum over the raw bf16 words.
    const float m = row_lane_max<CH>(x);
    if (tk_slot && tid == 0) *tk_slot = *tk;

    // Keep the bf16 words as the only live copy of the row.
#pragma unroll
    for (int j = 0; j < CH; ++j) asm volatile("" : "+v"(x[j]));

    // Pass B: e = 2^(x c - m c) summed in fp32 and kept as fp16 in place.
    const float c2 = kLog2e * p.inv_temp;
    const float mc = (m == -INFINITY) ? 0.0f : m * c2;
    float s = 0.0f;
    float t = 0.0f;  // ENT: sum of 2^d * d
    exp_pass_vgpr<CH, ENT>(x, c2, mc, s, t);

    float M = (m == -INFINITY) ? -INFINITY : mc;
    float S = s;
    float T = t;
    if constexpr (ENT)
        block_mst_reduce<BLOCK>(M, S, T, lds.m, lds.s, lds.t, tid);
    else
        block_ms_reduce<BLOCK>(M, S, lds.m, lds.s, tid);
    if (M == -INFINITY) {  // every logit of the row is -inf
        excluded_row<BLOCK, ENT>(row, drow, V, true, logp_out, tok_loss_out, entropy_out, row_loss,
                                 dev_err, tid);
        return;
    }
    const float lse2 = M + __builtin_amdgcn_logf(S);
    const RowOut o = row_epilogue(lse2, xy, old_logp[row], ref_logp[row], adv_tok[row], w, p);

    // Pass C: dlogits = -g * p_v = sc * e_v; the token's column gets g (1 - p_y).
    const float sc = -o.g * __builtin_amdgcn_exp2f(mc - lse2);
    const float dy = o.g * (1.0f - hw_exp(o.logp));
    dlogits_pass_vgpr<BLOCK, CH, SAFE>(x, sc, dy, y, drow, V, tid);
    if (tid == 0) {
        write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
        if (ENT) entropy_out[row] = entropy_of(S, T);
    }
}

// One workgroup per row.
template <int BLOCK, int CH, int SAFE, bool ENT>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void
grpo_rows_resident(const uint16_t* logits, int64_t ld, int V, int64_t N,
                   const int32_t* __restrict__ token_ids, const float* __restrict__ old_logp,
                   const float* __restrict__ ref_logp, const float* __restrict__ adv_tok,
                   const float* __restrict__ w_tok, Params p, float* __restrict__ logp_out,
                   float* __restrict__ tok_loss_out, float* __restrict__ entropy_out,
                   float* __restrict__ row_loss, uint16_t* dlogits, int32_t* __restrict__ dev_err,
                   int32_t* /*queue: the persistent form's only*/) {
    __shared__ RowLds<BLOCK, ENT> lds;
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    (void)N;
    const uint16_t* xrow = logits + row * ld;
    uint16_t* drow = dlogits + row * ld;
    const float w = w_tok[row];
    const int y = token_ids[row];
    if (!row_live(w, y, V)) {  // excluded; a weighted row with a bad token id is counted
        excluded_row<BLOCK, ENT>(row, drow, V, w != 0.0f, logp_out, tok_loss_out, entropy_out,
                                 row_loss, dev_err, tid);
        return;
    }
    // The whole row into registers: one read of HBM.
    u32x4 x[CH];
    load_row<BLOCK, CH, SAFE>(x, xrow, (V + 7) >> 3, tid * 16);
    const float xy = __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
    fused_row<BLOCK, CH, SAFE, ENT>(x, xy, row, drow, V, y, w, old_logp, ref_logp, adv_tok, p,
                                    logp_out, tok_loss_out, entropy_out, row_loss, dev_err, lds,
                                    tid);
}

// Fetch-and-add of k on the row queue, from one lane.  The pointer passes
// through an empty asm so that the compiler sees a per-lane address: it then
// emits one global atomic with return instead of a wave-wide aggregation,
// whose broadcast would wait for the atomic (and, the vector memory counter
// being in order, for every load and store before it) on the spot.  The
// result is waited for where it is used.
__device__ __forceinline__ int queue_take(int32_t* queue, int k) {
    int32_t* qp = queue;
    asm volatile("" : "+v"(qp));
    auto* gp = (__attribute__((address_space(1))) int32_t*)(qp);
    return __hip_atomic_fetch_add(gp, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Zero the row queue before the persistent kernel (a kernel rather than a
// memset, so that the call can be captured in a graph).
__global__ void queue_reset_kernel(int32_t* queue) {
    if (threadIdx.x == 0) *queue = 0;
}

// Persistent form: one workgroup per compute unit.  Workgroup b's first four
// rows are b, b + G, b + 2G and b + 3G (G = the grid); after them it takes
// rows from a queue, ticket t meaning row 4G + t.  A static stride would tie
// the call's end to the slowest compute units: measured with per-workgroup
// timestamps on the MI355X, the workgroups of half of the eight XCDs finish
// their equal shares ~8% of the call later than the others.
//
// The queue is read ahead so that its atomic never stalls the row: the
// workgroup knows its next three rows.  A live row takes as many tickets as
// make it three again (one atomic by thread 0 at the top of the row; it
// returns behind the row's own loads, which pass A waits for anyway),
// publishes the first ticket in LDS after pass A, and every thread reads it
// after the block merge's barrier.  An excluded row takes none, so three
// excluded rows in a row use the known rows up; only then does the
// workgroup fetch three tickets and wait for them at a barrier of its own.
// Every row a workgroup takes is larger than its previous one, so it stops
// at the first row >= N, and tickets it holds then are past N as well.
//
// The next row's token id and weight are fetched while the current row is
// processed, and its logits loads are issued as soon as the current row's
// registers are free: after the dlogits stores of a live row, before the
// zero fill of an excluded one.  On each compute unit the next row's reads
// thus overlap the current row's writes draining to HBM.  The token's
// logit is kept as raw bits until the epilogue, so that nothing waits for
// its load early.  The block merges of consecutive rows alternate between
// two LDS areas, and so do the published tickets: a wave that runs ahead
// into the next row cannot overwrite values a slower wave has yet to read.
// Which workgroup processes a row depends on timing, but every row's outputs
// are computed the same way wherever it runs, so results stay bitwise
// reproducible.
template <int BLOCK, int CH, int SAFE, bool ENT>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(4))) void
grpo_rows_persist(const uint16_t* logits, int64_t ld, int V, int64_t N,
                  const int32_t* __restrict__ token_ids, const float* __restrict__ old_logp,
                  const float* __restrict__ ref_logp, const float* __restrict__ adv_tok,
                  const float* __restrict__ w_tok, Params p, float* __restrict__ logp_out,
                  float* __restrict__ tok_loss_out, float* __restrict__ entropy_out,
                  float* __restrict__ row_loss, uint16_t* dlogits, int32_t* __restrict__ dev_err,
                  int32_t* queue) {
    __shared__ RowLds<BLOCK, ENT> lds[2];
    __shared__ int tks[2];
    constexpr int64_t kUnknown = -1;
    const int tid = threadIdx.x;
    const int nchunks = (V + 7) >> 3;
    const int64_t G = gridDim.x;
    const int64_t base = 4 * G;
    int64_t row = blockIdx.x;
    if (row >= N) return;
    // the next three rows; unknown ones (kUnknown) are always the last
    int64_t q1 = row + G, q2 = row + 2 * G, q3 = row + 3 * G;
    u32x4 x[CH];
    uint32_t xyb = 0;  // the token's bf16 logit
    // Issue the loads of row r (live) into x; its token logit into xyb.
    auto issue_row = [&](int64_t r, int yr) {
        const uint16_t* xrow = logits + r * ld;
        load_row<BLOCK, CH, SAFE>(x, xrow, nchunks, tid * 16);
        xyb = xrow[yr];
    };
    float w = w_tok[row];
    int y = token_ids[row];
    bool live = row_live(w, y, V);
    if (live) issue_row(row, y);
    int parity = 0;
    int tp = 0;
    while (true) {
        if (q1 == kUnknown) {
            if (tid == 0) tks[tp] = queue_take(queue, 3);
            __syncthreads();
            const int64_t t = base + __builtin_amdgcn_readfirstlane(tks[tp]);
            tp ^= 1;
            q1 = t;
            q2 = t + 1;
            q3 = t + 2;
        }
        const bool more = q1 < N;
        const int k = 1 + (q2 == kUnknown) + (q3 == kUnknown);
        int tk;  // set, and read through fused_row's pointer, in thread 0 of a live row only
        if (live && tid == 0) tk = queue_take(queue, k);
        const float w_next = more ? w_tok[q1] : 0.0f;
        const int y_next = more ? token_ids[q1] : 0;
        const bool live_next = more && row_live(w_next, y_next, V);
        uint16_t* drow = dlogits + row * ld;
        if (live) {
            fused_row<BLOCK, CH, SAFE, ENT>(x, __uint_as_float(xyb << 16), row, drow, V, y, w,
                                            old_logp, ref_logp, adv_tok, p, logp_out,
                                            tok_loss_out, entropy_out, row_loss, dev_err,
                                            lds[parity], tid, &tks[tp], &tk);
            parity ^= 1;
        }
        if (live_next) issue_row(q1, y_next);
        if (!live)
            excluded_row<BLOCK, ENT>(row, drow, V, w != 0.0f, logp_out, tok_loss_out, entropy_out,
                                     row_loss, dev_err, tid);
        if (!more) break;
        int64_t q4 = kUnknown;
        if (live) {  // the k new rows t, t + 1, ... fill the unknown places
            const int64_t t = base + __builtin_amdgcn_readfirstlane(tks[tp]);
            tp ^= 1;
            if (q2 == kUnknown) {
                q2 = t;
                q3 = t + 1;
                q4 = t + 2;
            } else if (q3 == kUnknown) {
                q3 = t;
                q4 = t + 1;
            } else {
                q4 = t;
            }
        }
        row = q1;
        q1 = q2;
        q2 = q3;
        q3 = q4;
        w = w_next;
        y = y_next;
        live = live_next;
    }
}

// Rows wider than the register file holds (196608 < V <= 270336): the first
// 24 chunks per lane stay in VGPRs as in the resident kernel, and the rest
// of the row -- up to 9 more chunks per lane, 144 KiB -- goes into LDS by
// LDS-DMA loads, so the row is still read from HBM once.  The LDS part keeps
// the bf16 logits: pass A takes its lane maximum, pass B sums its
// exponentials without storing them, and pass C recomputes each one from
// the row's log-sum-exp.  Each lane reads back only the chunks its own wave
// wrote, so the DMA needs no workgroup barrier, only the wave's own wait.
constexpr int kHybridCH = 24;
constexpr int kHybridLdsSlots = 9;
constexpr int64_t kHybridMaxV = static_cast<int64_t>(kHybridCH + kHybridLdsSlots) * 1024 * 8;

// LDS of the hybrid kernel: the row's LDS part and one block merge.
template <bool ENT>
struct HybridLds {
    __attribute__((aligned(16))) u32x4 xs[kHybridLdsSlots * 1024];
    RowLds<1024, ENT> red;
};

// Issue the loads of a live row: kHybridCH chunks per lane into x (all of
// them inside the row, V > 196608) and the rest into this wave's 1 KiB of
// each LDS slot (LDS-DMA); returns the token logit.
__device__ __forceinline__ float hybrid_issue(u32x4 (&x)[kHybridCH], u32x4* xs,
                                              const uint16_t* xrow, int V, int y, int tid) {
    constexpr int BLOCK = 1024;
    constexpr int CH = kHybridCH;
    const int wave = tid / kWave;
    const int nchunks = (V + 7) >> 3;
    const int nl = (nchunks - CH * BLOCK + BLOCK - 1) / BLOCK;  // LDS slots in use, 1..9
    load_row<BLOCK, CH, CH>(x, xrow, nchunks, tid * 16);
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(xrow, nchunks * 16);
    for (int k = 0; k < nl; ++k)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void*)(&xs[k * BLOCK + wave * kWave]), 16,
            tid * 16 + (CH + k) * BLOCK * 16, 0, 0, kLoadPolicy);
    return __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
}

// Passes A-C of a live row whose loads hybrid_issue has issued, and its
// outputs; a row whose logits are all -inf is counted and zero-filled.
template <bool ENT>
__device__ __forceinline__ void hybrid_row(u32x4 (&x)[kHybridCH], const u32x4* xs, float xy,
                                           int64_t row, uint16_t* drow, int V, int y, float w,
                                           const float* __restrict__ old_logp,
                                           const float* __restrict__ ref_logp,
                                           const float* __restrict__ adv_tok, const Params& p,
                                           float* __restrict__ logp_out,
                                           float* __restrict__ tok_loss_out,
                                           float* __restrict__ entropy_out,
                                           float* __restrict__ row_loss,
                                           int32_t* __restrict__ dev_err, RowLds<1024, ENT>& red,
                                           int tid) {
    constexpr int BLOCK = 1024;
    constexpr int CH = kHybridCH;
    const int nchunks = (V + 7) >> 3;
    const int nfull = V >> 3;
    const int nl = (nchunks - CH * BLOCK + BLOCK - 1) / BLOCK;

    // LDS chunk k of this lane, columns past V as -inf.
    auto lds_chunk = [&](int k) -> u32x4 {
        const int c = (CH + k) * BLOCK + tid;
        const u32x4 v = xs[k * BLOCK + tid];
        if (c >= nchunks) return u32x4_of(kNegInfPair, kNegInfPair, kNegInfPair, kNegInfPair);
        return c == nfull ? mask_tail(v, V & 7) : v;
    };

    // Pass A: lane maximum over both parts; the register part first, so its
    // waits follow its loads one by one, then the wait for the DMA.
    float m = row_lane_max<CH>(x);
    // this wave's loads, LDS-DMA included, have landed (tied to m so that it
    // is not scheduled ahead of the register part's maximum)
    asm volatile("s_waitcnt vmcnt(0)" : "+v"(m) : : "memory");
    {
        uint32_t mh = kNegInfPair;
        for (int k = 0; k < nl; ++k) {
            const u32x4 v = lds_chunk(k);
            mh = pk_max_f16(pk_max_f16(mh, v.x), pk_max_f16(v.y, pk_max_f16(v.z, v.w)));
        }
        m = fmaxf(m, fmaxf(max_half_to_f32(mh), max_half_to_f32(mh >> 16)));
    }
#pragma unroll
    for (int j = 0; j < CH; ++j) asm volatile("" : "+v"(x[j]));

    // Pass B: the register part as in the resident kernel, then the LDS part.
    const float c2 = kLog2e * p.inv_temp;
    const float mc = (m == -INFINITY) ? 0.0f : m * c2;
    float s = 0.0f;
    float t = 0.0f;
    exp_pass_vgpr<CH, ENT>(x, c2, mc, s, t);
    for (int k = 0; k < nl; ++k) {
        const u32x4 v = lds_chunk(k);
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float lo = bf_lo(wv[q]);
            const float hi = bf_hi(wv[q]);
            if constexpr (ENT) {
                const float da = vmax(fmaf(lo, c2, -mc), kMinExp2Arg);
                const float db = vmax(fmaf(hi, c2, -mc), kMinExp2Arg);
                const float a = __builtin_amdgcn_exp2f(da);
                const float b = __builtin_amdgcn_exp2f(db);
                s += a;
                s += b;
                t = fmaf(a, da, t);
                t = fmaf(b, db, t);
            } else {
                s += __builtin_amdgcn_exp2f(fmaf(lo, c2, -mc));
                s += __builtin_amdgcn_exp2f(fmaf(hi, c2, -mc));
            }
        }
    }

    float M = (m == -INFINITY) ? -INFINITY : mc;
    float S = s;
    float T = t;
    if constexpr (ENT)
        block_mst_reduce<BLOCK>(M, S, T, red.m, red.s, red.t, tid);
    else
        block_ms_reduce<BLOCK>(M, S, red.m, red.s, tid);
    if (M == -INFINITY) {
        excluded_row<BLOCK, ENT>(row, drow, V, true, logp_out, tok_loss_out, entropy_out, row_loss,
                                 dev_err, tid);
        return;
    }
    const float lse2 = M + __builtin_amdgcn_logf(S);
    const RowOut o = row_epilogue(lse2, xy, old_logp[row], ref_logp[row], adv_tok[row], w, p);

    // Pass C: the register part, then the LDS part with each probability
    // recomputed as 2^(x c - lse2).
    const float dy = o.g * (1.0f - hw_exp(o.logp));
    dlogits_pass_vgpr<BLOCK, CH, CH>(x, -o.g * __builtin_amdgcn_exp2f(mc - lse2), dy, y, drow, V,
                                     tid);
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, nfull * 16);
    const int cy = y >> 3;
    const int ey = y & 7;
    for (int k = 0; k < nl; ++k) {
        const int c = (CH + k) * BLOCK + tid;
        if (c >= nchunks) continue;
        const u32x4 v = xs[k * BLOCK + tid];
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
        float d[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            d[2 * q] = -o.g * __builtin_amdgcn_exp2f(fmaf(bf_lo(wv[q]), c2, -lse2));
            d[2 * q + 1] = -o.g * __builtin_amdgcn_exp2f(fmaf(bf_hi(wv[q]), c2, -lse2));
        }
        if (c == cy) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e == ey) d[e] = dy;
        }
        if (c < nfull) {
            const u32x4 out = u32x4_of(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]),
                                       pack_bf16(d[4], d[5]), pack_bf16(d[6], d[7]));
            __builtin_amdgcn_raw_buffer_store_b128(out, rd, c * 16, 0, kStorePolicy);
        } else {  // partial last chunk
            const int rem = V & 7;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (e < rem)
                    drow[(c << 3) + e] = static_cast<uint16_t>(pack_bf16(d[e], 0.0f) & 0xffffu);
        }
    }
    if (tid == 0) {
        write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
        if (ENT) entropy_out[row] = entropy_of(S, T);
    }
}

// One workgroup per row.
template <bool ENT>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(4))) void
grpo_rows_hybrid(const uint16_t* logits, int64_t ld, int V, int64_t N,
                 const int32_t* __restrict__ token_ids, const float* __restrict__ old_logp,
                 const float* __restrict__ ref_logp, const float* __restrict__ adv_tok,
                 const float* __restrict__ w_tok, Params p, float* __restrict__ logp_out,
                 float* __restrict__ tok_loss_out, float* __restrict__ entropy_out,
                 float* __restrict__ row_loss, uint16_t* dlogits, int32_t* __restrict__ dev_err,
                   int32_t* /*queue: the persistent form's only*/) {
    __shared__ HybridLds<ENT> lds;
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    (void)N;
    const uint16_t* xrow = logits + row * ld;
    uint16_t* drow = dlogits + row * ld;
    const float w = w_tok[row];
    const int y = token_ids[row];
    if (!row_live(w, y, V)) {
        excluded_row<1024, ENT>(row, drow, V, w != 0.0f, logp_out, tok_loss_out, entropy_out,
                                row_loss, dev_err, tid);
        return;
    }
    u32x4 x[kHybridCH];
    const float xy = hybrid_issue(x, lds.xs, xrow, V, y, tid);
    hybrid_row<ENT>(x, lds.xs, xy, row, drow, V, y, w, old_logp, ref_logp, adv_tok, p, logp_out,
                    tok_loss_out, entropy_out, row_loss, dev_err, lds.red, tid);
}

// ---------------------------------------------------------------------------
// Streaming variant for any V: online (max, sum) over the row, then a second
// read to form dlogits.  Each chunk is read and written by one thread only,
// so in-place use is safe.
// ---------------------------------------------------------------------------
template <int BLOCK, bool ENT>
__global__ __launch_bounds__(BLOCK) void grpo_rows_stream(
    const uint16_t* logits, int64_t ld, int V, int64_t N, const int32_t* __restrict__ token_ids,
    const float* __restrict__ old_logp, const float* __restrict__ ref_logp,
    const float* __restrict__ adv_tok, const float* __restrict__ w_tok, Params p,
    float* __restrict__ logp_out, float* __restrict__ tok_loss_out,
    float* __restrict__ entropy_out, float* __restrict__ row_loss, uint16_t* dlogits,
    int32_t* __restrict__ dev_err, int32_t* /*queue: the persistent form's only*/) {
    __shared__ float s_m[BLOCK / kWave];
    __shared__ float s_s[BLOCK / kWave];
    __shared__ float s_t[ENT ? BLOCK / kWave : 1];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    (void)N;
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
        if (tid == 0) {
            write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
            if (ENT) entropy_out[row] = 0.0f;
        }
        return;
    }
    const float xy = __uint_as_float(static_cast<uint32_t>(xrow[y]) << 16);
    const float c2 = kLog2e * p.inv_temp;
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
                    t = (t + dm * s) * exp2f(dm);
                }
            }
            s = (m == -INFINITY) ? 0.0f : s * exp2f(m - cm);
            m = cm;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if constexpr (ENT) {
                const float d = vmax(f[e] - m, kMinExp2Arg);
                const float a = exp2f(d);
                s += a;
                t = fmaf(a, d, t);
            } else {
                s += exp2f(f[e] - m);
            }
        }
    }
    float M = m, S = s, T = t;
    if constexpr (ENT)
        block_mst_reduce<BLOCK>(M, S, T, s_m, s_s, s_t, tid);
    else
        block_ms_reduce<BLOCK>(M, S, s_m, s_s, tid);
    if (M == -INFINITY) {
        if (tid == 0) count_error(dev_err);
        zero_row<BLOCK>(drow, V, tid);
        if (tid == 0) {
            write_row_outputs(row, 0.0f, 0.0f, 0.0f, logp_out, tok_loss_out, row_loss);
            if (ENT) entropy_out[row] = 0.0f;
        }
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
    if (tid == 0) {
        write_row_outputs(row, o.logp, o.loss, w, logp_out, tok_loss_out, row_loss);
        if (ENT) entropy_out[row] = entropy_of(S, T);
    }
}

// ---------------------------------------------------------------------------
// Host dispatch
// ---------------------------------------------------------------------------
using RowKernel = void (*)(const uint16_t*, int64_t, int, int64_t, const int32_t*, const float*,
                           const float*, const float*, const float*, Params, float*, float*,
                           float*, float*, uint16_t*, int32_t*, int32_t*);

struct RowConfig {
    RowKernel fn;      // without the entropy output
    RowKernel fn_ent;  // with it
    int block;
    int ch;           // 0: streaming variant
    bool persistent;  // one workgroup per compute unit, rows from a queue
};

#define LEAP_RES(B, C, S) \
    RowConfig{grpo_rows_resident<B, C, S, false>, grpo_rows_resident<B, C, S, true>, B, C, false}
#define LEAP_PER(B, C, S) \
    RowConfig{grpo_rows_persist<B, C, S, false>, grpo_rows_persist<B, C, S, true>, B, C, true}

// The kernel for V: the resident shape row::pick_resident_shape chooses, or
// the streaming variant.  From 55296 to 155648 columns (the 1024-lane shapes
// of 8, 12, 16 and 19 chunks per lane) the row kernel runs persistent with
// the row queue: measured on the MI355X with every row live it is 1.4-13.5%
// faster there than one workgroup per row (6-10% at 12 chunks; 2-3% at 16
// and 19 chunks on full lines).  Below 55296 columns the 8-chunk one-row
// kernel, which fits two workgroups per compute unit against the persistent
// loop's one, stays ahead (1-24%), and at 20 and 24 chunks the loop's live
// state would spill, so those widths keep one workgroup per row.  The row
// queue counts in 32 bits: beyond kQueueMaxRows rows (far more than any
// device holds at these widths) the one-row kernel of the same shape runs.
constexpr int64_t kQueueMaxRows = int64_t{1} << 30;
constexpr int kPersistMinV = 55297;

RowConfig pick_row_config(int V, int64_t N) {
    static const RowConfig table[] = {
        LEAP_RES(64, 1, 0),     LEAP_RES(64, 2, 1),     LEAP_RES(64, 4, 2),
        LEAP_RES(64, 8, 4),     LEAP_RES(256, 4, 0),    LEAP_RES(256, 8, 4),
        LEAP_RES(256, 12, 8),   LEAP_RES(256, 16, 12),  LEAP_RES(1024, 8, 0),
        LEAP_RES(1024, 12, 8),  LEAP_RES(1024, 16, 12), LEAP_RES(1024, 19, 16),
        LEAP_RES(1024, 20, 19), LEAP_RES(1024, 24, 20),
    };
    static const RowConfig persist[] = {
        LEAP_PER(1024, 8, 0), LEAP_PER(1024, 12, 8), LEAP_PER(1024, 16, 12),
        LEAP_PER(1024, 19, 16),
    };
    static_assert(sizeof(table) / sizeof(table[0]) == kNumResidentShapes, "shape table");
    const int i = pick_resident_shape(V);
    if (i < 0) {
        if (V <= kHybridMaxV)
            return RowConfig{grpo_rows_hybrid<false>, grpo_rows_hybrid<true>, 1024, kHybridCH,
                             false};
        return RowConfig{grpo_rows_stream<1024, false>, grpo_rows_stream<1024, true>, 1024, 0,
                         false};
    }
    if (V >= kPersistMinV && N <= kQueueMaxRows && table[i].block == 1024 && table[i].ch <= 19)
        for (const RowConfig& rc : persist)
            if (rc.ch == table[i].ch) return rc;
    return table[i];
}

#undef LEAP_RES
#undef LEAP_PER

}  // namespace
}  // namespace leap

namespace leap {
namespace {
// Workspace of the fused call: one fp32 weighted loss per row in whole
// 256-byte lines, then one line holding the persistent kernel's row queue.
size_t row_loss_bytes(int64_t N) {
    const size_t b = static_cast<size_t>(N > 0 ? N : 1) * sizeof(float);
    return (b + 255) & ~static_cast<size_t>(255);
}
constexpr size_t kQueueBytes = 256;
}  // namespace
}  // namespace leap

LEAP_API size_t leap_grpo_workspace_size(int64_t N, int32_t V) {
    (void)V;
    return leap::row_loss_bytes(N) + leap::kQueueBytes;
}

namespace leap {
namespace {

// Host-side checks of the fused call's arguments (everything but the
// workspace).
leap_status check_fused_args(const void* logits_bf16, int64_t ld, int64_t N, int32_t V,
                             const int32_t* token_ids, const float* old_logp,
                             const float* ref_logp, const float* adv_tok, const float* w_tok,
                             const leap_grpo_params* params, const float* loss_out,
                             const void* dlogits_bf16) {
    if (N < 0 || V < 1 || ld < V || !params || !loss_out) return LEAP_ERR_INVALID_ARG;
    const leap_grpo_params& pp = *params;
    if (!(pp.clip_eps_low >= 0.0f) || !(pp.clip_eps_high >= 0.0f) || !(pp.kl_coef >= 0.0f) ||
        !(pp.inv_temperature > 0.0f) || !__builtin_isfinite(pp.clip_eps_low) ||
        !__builtin_isfinite(pp.clip_eps_high) || !__builtin_isfinite(pp.kl_coef) ||
        !__builtin_isfinite(pp.inv_temperature))
        return LEAP_ERR_INVALID_ARG;
    if (pp.kl_type != LEAP_KL_K3 && pp.kl_type != LEAP_KL_K1 && pp.kl_type != LEAP_KL_K2)
        return LEAP_ERR_UNSUPPORTED;
    if (V > LEAP_MAX_V) return LEAP_ERR_UNSUPPORTED;
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
    return LEAP_OK;
}

// The row kernel, then the fixed-order loss sum, with the per-row weighted
// losses in row_loss (N floats) and the persistent kernel's row queue in
// *queue (zeroed here before that kernel).
leap_status launch_fused(const void* logits_bf16, int64_t ld, int64_t N, int32_t V,
                         const int32_t* token_ids, const float* old_logp, const float* ref_logp,
                         const float* adv_tok, const float* w_tok, const leap_grpo_params& pp,
                         float* logp_out, float* tok_loss_out, float* entropy_out, float* loss_out,
                         void* dlogits_bf16, float* row_loss, int32_t* queue, int32_t* dev_err,
                         hipStream_t stream) {
    const LaunchCheck lc;
    const Params p{pp.clip_eps_low, pp.clip_eps_high, pp.kl_coef, pp.inv_temperature, pp.kl_type};
    if (N > 0) {
        const RowConfig rc = pick_row_config(V, N);
        int64_t grid = N;
        const RowKernel fn = entropy_out ? rc.fn_ent : rc.fn;
        if (rc.persistent) {
            hipLaunchKernelGGL(queue_reset_kernel, dim3(1), dim3(kWave), 0, stream, queue);
            // as many workgroups as the device holds at once
            int dev = 0, cus = 0, per_cu = 0;
            if (hipGetDevice(&dev) != hipSuccess ||
                hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                    hipSuccess ||
                hipOccupancyMaxActiveBlocksPerMultiprocessor(
                    &per_cu, reinterpret_cast<const void*>(fn), rc.block, 0) != hipSuccess)
                return LEAP_ERR_HIP;
            const int64_t resident = static_cast<int64_t>(cus > 0 ? cus : 1) * (per_cu > 0 ? per_cu : 1);
            if (grid > resident) grid = resident;
        }
        hipLaunchKernelGGL(fn, dim3(static_cast<unsigned>(grid)),
                           dim3(rc.block), 0, stream, static_cast<const uint16_t*>(logits_bf16), ld,
                           V, N, token_ids, old_logp, ref_logp, adv_tok, w_tok, p, logp_out,
                           tok_loss_out, entropy_out, row_loss,
                           static_cast<uint16_t*>(dlogits_bf16), dev_err, queue);
        const leap_status st = lc.status();
        if (st != LEAP_OK) return st;
    }
    hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(kReduceBlock), 0, stream, row_loss, N,
                       loss_out);
    return lc.status();
}

// Scratch of the no-allocation entry point: the per-row losses, then one
// 256-byte line for the row queue; one array per device, held from the
// library's load until the process ends.  Every call on a device reuses it,
// so calls that overlap on one device (different streams without ordering)
// race on it.  Nothing needs clearing by the caller: the row kernel writes
// all N losses before the loss sum reads them, and the call zeroes the
// queue itself.
constexpr int kScratchFloats = LEAP_NOALLOC_MAX_ROWS + static_cast<int>(kQueueBytes / sizeof(float));
static __device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up once
// per device with that device current.  (The host-side name of the array is
// only a stand-in handle; kernels must receive this address.)
leap_status scratch_for_current_device(float** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return LEAP_ERR_HIP;
    if (dev >= kMaxDevices) return LEAP_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return LEAP_ERR_HIP;
        g_scratch_ptr[dev] = static_cast<float*>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return LEAP_OK;
}

}  // namespace
}  // namespace leap

LEAP_API leap_status leap_grpo_logprob_loss_fwd_bwd(
    const void* logits_bf16, int64_t ld, int64_t N, int32_t V, const int32_t* token_ids,
    const float* old_logp, const float* ref_logp, const float* adv_tok, const float* w_tok,
    const leap_grpo_params* params, float* logp_out, float* tok_loss_out, float* entropy_out,
    float* loss_out, void* dlogits_bf16, void* workspace, size_t ws_bytes, int32_t* dev_err,
    hipStream_t stream) {
    using namespace leap;
    const leap_status st = check_fused_args(logits_bf16, ld, N, V, token_ids, old_logp, ref_logp,
                                            adv_tok, w_tok, params, loss_out, dlogits_bf16);
    if (st != LEAP_OK) return st;
    if (!workspace || ws_bytes < leap_grpo_workspace_size(N, V)) return LEAP_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 3u) != 0) return LEAP_ERR_MISALIGNED;
    char* ws = static_cast<char*>(workspace);
    return launch_fused(logits_bf16, ld, N, V, token_ids, old_logp, ref_logp, adv_tok, w_tok,
                        *params, logp_out, tok_loss_out, entropy_out, loss_out, dlogits_bf16,
                        reinterpret_cast<float*>(ws),
                        reinterpret_cast<int32_t*>(ws + row_loss_bytes(N)), dev_err, stream);
}

LEAP_API leap_status leap_grpo_logprob_loss_fwd_bwd_noalloc(
    const void* logits_bf16, int64_t ld, int64_t N, int32_t V, const int32_t* token_ids,
    const float* old_logp, const float* ref_logp, const float* adv_tok, const float* w_tok,
    const leap_grpo_params* params, float* logp_out, float* tok_loss_out, float* entropy_out,
    float* loss_out, void* dlogits_bf16, int32_t* dev_err, hipStream_t stream) {
    using namespace leap;
    leap_status st = check_fused_args(logits_bf16, ld, N, V, token_ids, old_logp, ref_logp,
                                      adv_tok, w_tok, params, loss_out, dlogits_bf16);
    if (st != LEAP_OK) return st;
    if (N > LEAP_NOALLOC_MAX_ROWS) return LEAP_ERR_UNSUPPORTED;
    float* row_loss = nullptr;
    if ((st = scratch_for_current_device(&row_loss)) != LEAP_OK) return st;
    return launch_fused(logits_bf16, ld, N, V, token_ids, old_logp, ref_logp, adv_tok, w_tok,
                        *params, logp_out, tok_loss_out, entropy_out, loss_out, dlogits_bf16,
                        row_loss, reinterpret_cast<int32_t*>(row_loss + LEAP_NOALLOC_MAX_ROWS),
                        dev_err, stream);
}
