/*
 * leap.h -- C ABI of libleap, the MI355X (gfx950) hot path of the GRPO
 * training step of "LEAP: Lean Environment-Feedback via Adaptive Pruning for
 * Code RL in GPU Kernel Generation" (arXiv 2608.01804).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array pointer is a DEVICE pointer, allocated and owned by the
 *    caller.  The library never allocates or frees memory and never
 *    synchronises; each call enqueues its kernels on `stream` (0 = the null
 *    stream) and returns.
 *  - The returned leap_status reports what the host can check before
 *    launching: argument values, pointer alignment, workspace size, and a
 *    launch error from the HIP runtime (LEAP_ERR_HIP).  Every host-side check
 *    precedes the call's first launch, so on LEAP_ERR_INVALID_ARG,
 *    LEAP_ERR_MISALIGNED, LEAP_ERR_WORKSPACE and LEAP_ERR_UNSUPPORTED nothing
 *    has been enqueued.  On LEAP_ERR_HIP the kernels of the call launched
 *    before the failing one may already be enqueued (the calls made of
 *    several launches: the fused objective, the fused LM head, the
 *    vocabulary merge and the rollout statistics); the outputs are then
 *    undefined.  LEAP_ERR_HIP is returned only for an error raised by one of
 *    the call's own launches: an error the caller's earlier HIP work left
 *    pending is neither reported nor cleared.
 *  - Errors that depend on device data (a token id outside [0, V), a
 *    pass_turn outside [0, M], a rollout index out of range, a row whose
 *    logits are all -inf) add 1 per offending item to the optional device
 *    counter *dev_err (nullable; the caller zeroes it and reads it after its
 *    own synchronisation).  The offending item is treated as excluded from
 *    the objective, as described per call.
 *  - No exception crosses the ABI.  The library keeps no state between
 *    calls, is reentrant, and gives bitwise identical results for identical
 *    inputs and shapes.
 *  - Row-major layouts; "group-major" means rollout i of group g is at
 *    index g*G + i.
 */
#ifndef LEAP_H_
#define LEAP_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum leap_status {
    LEAP_OK = 0,
    LEAP_ERR_INVALID_ARG = 1, /* null required pointer, size or enum out of range */
    LEAP_ERR_MISALIGNED = 2,  /* a pointer or leading dimension breaks the alignment rule */
    LEAP_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the *_workspace_size() value */
    LEAP_ERR_UNSUPPORTED = 4, /* valid request the library does not implement */
    LEAP_ERR_HIP = 5          /* the HIP runtime reported an error at launch */
} leap_status;

/* Widest row, in columns, that the row entry points (the fused objective,
 * the forward-only log-prob and the vocabulary-shard calls) accept: every
 * per-row byte offset they form then fits in 32 bits.  Wider rows are
 * refused with LEAP_ERR_UNSUPPORTED. */
#define LEAP_MAX_V 268435456

/* Ordering key of the tournament. */
typedef enum leap_key_mode {
    /* The paper's order (Sec. 3.2, Eq. 4): first pass on an earlier turn is
     * strictly preferred; every failure ties at the bottom. */
    LEAP_KEY_TURN = 0,
    /* Extension, not in the paper: tier first, then the larger quantised
     * speedup, then the smaller generated-token count; equal tuples tie. */
    LEAP_KEY_LEX = 1
} leap_key_mode;

/* Advantage from the tournament reward ("standard GRPO formulation",
 * end of Sec. 3.2). */
typedef enum leap_adv_norm {
    LEAP_ADV_STD = 0,  /* A_i = (R_i - mean_g R) / (std_g R + eps), unbiased std */
    LEAP_ADV_NONE = 1  /* A_i = R_i */
} leap_adv_norm;

/* Aggregation weight of a token in the loss (Sec. 4.1, sample-level loss;
 * Eq. 3's 1/G sum over samples). */
typedef enum leap_loss_agg {
    LEAP_AGG_SEQ_MEAN_TOKEN_MEAN = 0, /* w = 1 / (denominator * |M_i|), denominator = sequences in the step */
    LEAP_AGG_TOKEN_MEAN = 1,          /* w = 1 / denominator, denominator = generated tokens in the step */
    LEAP_AGG_SUM = 2                  /* w = 1 */
} leap_loss_agg;

/* Estimator of the reference-KL term of Eq. 3. */
typedef enum leap_kl_type {
    LEAP_KL_K3 = 0, /* exp(r - lp) - (r - lp) - 1 (GRPO's estimator) */
    LEAP_KL_K1 = 1, /* lp - r */
    LEAP_KL_K2 = 2  /* (lp - r)^2 / 2 */
} leap_kl_type;

/* Hyper-parameters of the per-token objective (host struct, read at call). */
typedef struct leap_grpo_params {
    float clip_eps_low;    /* >= 0; ratio clipped below at 1 - clip_eps_low */
    float clip_eps_high;   /* >= 0; ratio clipped above at 1 + clip_eps_high */
    float kl_coef;         /* beta of Eq. 3, >= 0 */
    int32_t kl_type;       /* leap_kl_type */
    float inv_temperature; /* > 0; logits are multiplied by it before the softmax */
} leap_grpo_params;

/* Human-readable name of a status code (static string). */
const char *leap_status_string(leap_status s);

/* Library version, e.g. "0.1.0" (static string). */
const char *leap_version(void);

/*
 * Rank-based reward and advantage (Sec. 3.2, Eqs. 4-6).
 *
 * For every group of G rollouts: the tier r_i = 0 if pass_turn[i] == 0
 * (never passed), else M - pass_turn[i] + 1 (Eq. 4); the tournament counts
 * n_worse_i = #{j != i : key_i > key_j}, n_better_i = #{j != i : key_i <
 * key_j} (Eq. 5); the reward R_i = (n_worse_i - n_better_i) / (G - 1)
 * (Eq. 6), computed in double precision and rounded once to float; and the
 * advantage A_i per `norm` (eps is the std guard; 1e-6 is conventional).
 *
 * pass_turn  int32 [n_groups*G], group-major; 0 or 1..M.  An entry outside
 *            0..M counts in *dev_err and ranks as a failure (r = 0).
 * speedup_q  int32 [n_groups*G], LEX mode only (NULL otherwise).
 * n_tokens   int32 [n_groups*G], LEX mode only (NULL otherwise).
 * n_groups   >= 0;  G in 2..1024;  M >= 1.
 * n_worse, n_better, rank_r   int32 [n_groups*G], each nullable.
 * reward, advantage           float [n_groups*G], required.
 * Errors: LEAP_ERR_INVALID_ARG for G < 2 or > 1024, M < 1, n_groups < 0,
 * eps < 0 or not finite, an unknown key/norm, a required pointer NULL.
 */
leap_status leap_rank_advantages(const int32_t *pass_turn, const int32_t *speedup_q,
                                 const int32_t *n_tokens, int64_t n_groups, int32_t G,
                                 int32_t M, int32_t key, int32_t norm, float eps,
                                 int32_t *n_worse, int32_t *n_better, int32_t *rank_r,
                                 float *reward, float *advantage, int32_t *dev_err,
                                 hipStream_t stream);

/*
 * Difficulty-Conditioned Pruning gate (Sec. 3.1, Eqs. 1-2).
 *
 * n_fail[g] = number of rollouts of group g whose first-turn response
 * failed verification (first_turn_pass == 0; any nonzero byte is a pass);
 * gate[g] = 1 iff tau_min <= n_fail[g] <= tau_max (inclusive), else 0.
 *
 * first_turn_pass  uint8 [n_groups*G], group-major.
 * n_fail           int32 [n_groups], nullable.   gate  uint8 [n_groups].
 * Errors: LEAP_ERR_INVALID_ARG for G < 1 or > 1024, n_groups < 0,
 * tau_min > tau_max, tau_min < 0, tau_max > G, a required pointer NULL.
 */
leap_status leap_dcp_gate(const uint8_t *first_turn_pass, int64_t n_groups, int32_t G,
                          int32_t tau_min, int32_t tau_max, int32_t *n_fail,
                          uint8_t *gate, hipStream_t stream);

/*
 * Host helper (no device work): the inclusive integer bounds [tau_min,
 * tau_max] on N_fail that select exactly the groups whose first-turn pass
 * rate (G - N_fail)/G lies in the interval from lo_num/lo_den to
 * hi_num/hi_den, each end open (strict = 1) or closed (strict = 0).  The
 * conversion is exact rational arithmetic (Sec. 3.1 phrases the thresholds
 * as pass rates in its pruning study; Eq. 2 takes failure counts).
 * Errors: LEAP_ERR_INVALID_ARG for G < 1, a denominator <= 0, NULL outputs,
 * or an interval that admits no N_fail in 0..G.
 */
leap_status leap_dcp_tau_from_pass_rate(int32_t G, int32_t lo_num, int32_t lo_den,
                                        int32_t lo_strict, int32_t hi_num, int32_t hi_den,
                                        int32_t hi_strict, int32_t *tau_min,
                                        int32_t *tau_max);

/*
 * Discounted per-turn token advantage (Sec. 3.3) and aggregation weight.
 *
 * Token k belongs to rollout i = tok_rollout[k] (-1: excluded -- padding,
 * prompt or environment feedback) and generated turn t = tok_turn[k] of its
 * T_i = n_turns[i] turns.  beta_i = gamma if A_i >= 0 else 1;
 * adv_tok[k] = beta_i^(T_i - t - 1) * A_i.  w_tok[k] per `agg` with
 * |M_i| = n_gen_tokens[i] (generated tokens of rollout i over all its
 * turns).  Excluded tokens get adv = 0 and w = 0.  Computed in double and
 * rounded once to float.
 *
 * advantage     float [n_rollouts]     tok_rollout, tok_turn  int32 [N]
 * n_turns, n_gen_tokens  int32 [n_rollouts]
 * adv_tok, w_tok         float [N]
 * gamma in (0, 1];  denominator > 0 (ignored for LEAP_AGG_SUM).
 * A token with tok_rollout < -1 or >= n_rollouts, a turn outside 0..T_i-1,
 * or a rollout with T_i < 1 or n_gen_tokens < 1 counts in *dev_err and is
 * excluded.
 * Errors: LEAP_ERR_INVALID_ARG for N < 0, n_rollouts < 0, gamma or
 * denominator out of range, an unknown agg, a required pointer NULL.
 */
leap_status leap_token_advantages(const float *advantage, const int32_t *tok_rollout,
                                  const int32_t *tok_turn, const int32_t *n_turns,
                                  const int32_t *n_gen_tokens, int32_t n_rollouts, int64_t N,
                                  float gamma, int32_t agg, double denominator,
                                  float *adv_tok, float *w_tok, int32_t *dev_err,
                                  hipStream_t stream);

/* Workspace bytes leap_grpo_logprob_loss_fwd_bwd needs for N rows: the
 * per-row weighted losses (4 bytes per row, in whole 256-byte lines) and
 * one 256-byte line for the row queue of the persistent kernel. */
size_t leap_grpo_workspace_size(int64_t N, int32_t V);

/*
 * Fused per-token GRPO objective and its logits gradient over one
 * microbatch of N rows (Sec. 3.1, Eq. 3, per token; surrogate read as
 * PPO-clip, KL per params->kl_type).
 *
 * For each row k with w_tok[k] != 0, with z = inv_temperature * logits[k]:
 *   logp_k  = z[y_k] - log sum_v exp(z[v])                (y_k = token_ids[k])
 *   rho_k   = exp(logp_k - old_logp[k])
 *   surr_k  = min(rho_k * A_k, clip(rho_k, 1 - eps_lo, 1 + eps_hi) * A_k)
 *   loss_k  = -surr_k + kl_coef * KL(logp_k, ref_logp[k])
 *   g_k     = w_k * d loss_k / d logp_k * inv_temperature
 *   dlogits[k][v] = g_k * ([v == y_k] - softmax(z)[v])      (bf16, RNE)
 * where A_k = adv_tok[k] and w_k = w_tok[k].  The ratio's gradient flows
 * when A_k > 0 and rho_k <= 1 + eps_hi, or A_k < 0 and rho_k >= 1 - eps_lo.
 * A row with w_tok[k] == 0 is excluded: its logits are not read, its
 * dlogits row is written as zeros, logp_out and tok_loss_out get 0.
 * A row with w != 0 but a token id outside [0, V), or all logits -inf,
 * counts in *dev_err and is excluded the same way.
 *
 * logits_bf16  [N][ld] bf16 (row k at element k*ld; V columns used).
 * dlogits_bf16 [N][ld] bf16, written in columns 0..V-1; may equal
 *              logits_bf16 (in place), must not otherwise overlap it.
 * token_ids int32 [N]; old_logp, ref_logp, adv_tok, w_tok float [N].
 * logp_out, tok_loss_out  float [N], nullable (tok_loss is unweighted loss_k).
 * entropy_out  float [N], nullable: H_k = -sum_v p_v ln p_v of softmax(z)
 *              in nats (0 for excluded rows) -- a per-token training
 *              statistic beside Eq. 3, not a term of it; when NULL the
 *              kernels skip its extra accumulator.
 * loss_out   float [1], required: sum_k w_k * loss_k, summed in a fixed order.
 * workspace  device buffer of >= leap_grpo_workspace_size(N, V) bytes,
 *            8-byte aligned; its contents on entry do not matter and it is
 *            scratch for this call only (calls that share one workspace
 *            must be ordered on one stream).
 * Alignment: logits and dlogits 16-byte aligned, ld % 8 == 0, ld >= V.
 *            Rows whose byte stride is a multiple of 128 (ld % 64 == 0) and
 *            arrays on 128-byte boundaries write whole cache lines: with an
 *            odd vocabulary, padding ld that way makes the call 8-9% faster.
 * Finite logits are expected below 2^121 in magnitude (the row maximum is
 *            taken on an fp16 reading of the bf16 bits, exact below that).
 * Errors: LEAP_ERR_INVALID_ARG for N < 0, V < 1, ld < V, a parameter out of
 * range, a required pointer NULL; LEAP_ERR_MISALIGNED; LEAP_ERR_WORKSPACE;
 * LEAP_ERR_UNSUPPORTED for an unknown kl_type or V > LEAP_MAX_V.
 */
leap_status leap_grpo_logprob_loss_fwd_bwd(const void *logits_bf16, int64_t ld, int64_t N,
                                           int32_t V, const int32_t *token_ids,
                                           const float *old_logp, const float *ref_logp,
                                           const float *adv_tok, const float *w_tok,
                                           const leap_grpo_params *params, float *logp_out,
                                           float *tok_loss_out, float *entropy_out,
                                           float *loss_out, void *dlogits_bf16, void *workspace,
                                           size_t ws_bytes, int32_t *dev_err,
                                           hipStream_t stream);

/* Largest N that leap_grpo_logprob_loss_fwd_bwd_noalloc accepts. */
#define LEAP_NOALLOC_MAX_ROWS 1048576

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * call as leap_grpo_logprob_loss_fwd_bwd (same kernels, same results bit for
 * bit, same argument rules) without the workspace arguments.  Its scratch
 * (the per-row losses and the row queue) is a library-owned device array of
 * LEAP_NOALLOC_MAX_ROWS floats plus 256 bytes (4 MiB) per device, held until
 * the process ends; the call itself
 * allocates and frees nothing.  The first call on a device looks up that
 * device's array (the device must be current).
 * All calls on one device share its array: calls that may overlap on one
 * device (unordered streams) race and must be serialised by the caller.
 * Errors: as leap_grpo_logprob_loss_fwd_bwd, plus LEAP_ERR_UNSUPPORTED for
 * N > LEAP_NOALLOC_MAX_ROWS (or a device index of 64 or more), and
 * LEAP_ERR_HIP if the device array cannot be found.
 */
leap_status leap_grpo_logprob_loss_fwd_bwd_noalloc(const void *logits_bf16, int64_t ld,
                                                   int64_t N, int32_t V,
                                                   const int32_t *token_ids,
                                                   const float *old_logp, const float *ref_logp,
                                                   const float *adv_tok, const float *w_tok,
                                                   const leap_grpo_params *params,
                                                   float *logp_out, float *tok_loss_out,
                                                   float *entropy_out, float *loss_out,
                                                   void *dlogits_bf16, int32_t *dev_err,
                                                   hipStream_t stream);

/*
 * Forward-only log-probability of each row's token: the old-policy and
 * reference forward passes whose outputs enter the ratio and the KL term of
 * the per-token objective (Sec. 3.1, Eq. 3).
 *
 *   logp_out[k] = z[y_k] - log sum_v exp(z[v]),  z = inv_temperature * logits[k]
 *
 * logits_bf16 [N][ld] bf16, token_ids int32 [N], logp_out float [N].
 * entropy_out float [N], nullable: H_k = -sum_v p_v ln p_v of softmax(z) in
 *             nats, as in leap_grpo_logprob_loss_fwd_bwd.
 * w_tok float [N], nullable: a row with w_tok[k] == 0 is not read and gets 0
 * (log-prob and entropy).  A token id outside [0, V) or a row of all -inf
 * logits counts in *dev_err and gets NaN (log-prob and entropy).  Alignment and range rules as leap_grpo_logprob_loss_fwd_bwd;
 * no workspace.
 * Errors: LEAP_ERR_INVALID_ARG for N < 0, V < 1, ld < V, a non-positive or
 * non-finite inv_temperature, a required pointer NULL; LEAP_ERR_MISALIGNED;
 * LEAP_ERR_UNSUPPORTED for V > LEAP_MAX_V.
 */
leap_status leap_logprob_fwd(const void *logits_bf16, int64_t ld, int64_t N, int32_t V,
                             const int32_t *token_ids, const float *w_tok,
                             float inv_temperature, float *logp_out, float *entropy_out,
                             int32_t *dev_err, hipStream_t stream);

/* Workspace bytes leap_grpo_lmhead_fwd_bwd needs (0 for invalid sizes).
 * Called with a prepared transposed weight (weight_t_bf16), it needs
 * leap_lmhead_workspace_size(N, V, H) - leap_lmhead_weight_t_size(V, H)
 * bytes only. */
size_t leap_lmhead_workspace_size(int64_t N, int32_t V, int32_t H);

/* Bytes of the transposed weight leap_lmhead_transpose_weight writes:
 * H x V_pad bf16, V_pad = V rounded up to a multiple of 256 (0 for invalid
 * sizes). */
size_t leap_lmhead_weight_t_size(int32_t V, int32_t H);

/*
 * The transposed LM-head weight that leap_grpo_lmhead_fwd_bwd's dhidden
 * product reads: weight_t[h][v] = weight[v][h] for v < V, 0 for V <= v <
 * V_pad, bf16 [H][V_pad].  The weight changes only at an optimizer step, so
 * one transpose can serve every microbatch of a step (pass it as
 * weight_t_bf16); without it each call forms its own copy in the workspace.
 * weight_bf16 [V][H] and weight_t_bf16 16-byte aligned, bytes >=
 * leap_lmhead_weight_t_size(V, H), caller-owned.
 * Errors: LEAP_ERR_INVALID_ARG for V < 1, H < 1, a NULL pointer;
 * LEAP_ERR_MISALIGNED; LEAP_ERR_WORKSPACE for too few bytes;
 * LEAP_ERR_UNSUPPORTED for H % 64 != 0 or a weight of 4 GiB or more.
 */
leap_status leap_lmhead_transpose_weight(const void *weight_bf16, int32_t V, int32_t H,
                                         void *weight_t_bf16, size_t bytes, hipStream_t stream);

/*
 * Fused LM head + per-token GRPO objective (Sec. 3.1, Eq. 3, per token):
 * the same per-row objective as leap_grpo_logprob_loss_fwd_bwd, on logits
 * z = hidden * weight^T formed tile by tile on the matrix cores and never
 * written to memory, plus the gradients of L = sum_k w_k * loss_k:
 *
 *   dZ[k][v]   = g_k * ([v == y_k] - softmax(inv_temperature * z_k)[v])
 *   dhidden    = dZ * weight          [N][H]
 *   dweight    = dZ^T * hidden        [V][H]
 *
 * Products accumulate in fp32 from bf16 operands; dZ is rounded to bf16
 * (RNE) before the two gradient products.  logp, tok_loss, loss and g follow
 * the rules of leap_grpo_logprob_loss_fwd_bwd, including excluded rows
 * (w == 0: zero gradient rows, logp_out = tok_loss_out = 0) and bad token
 * ids (counted in *dev_err, excluded).  Excluded rows take no part in the
 * products: the call lists the rows with w != 0 on the device and runs its
 * GEMMs over those only, so an excluded row's hidden state is never read
 * (non-finite values there reach no output) and costs no matrix work.
 *
 * hidden_bf16 [N][H] bf16, weight_bf16 [V][H] bf16, both row-major, 16-byte
 *              aligned.  H % 64 == 0 (else LEAP_ERR_UNSUPPORTED).
 * weight_t_bf16  nullable: leap_lmhead_transpose_weight's output for this
 *              weight (16-byte aligned); the call then skips its own
 *              transpose and does not need the workspace's last
 *              leap_lmhead_weight_t_size(V, H) bytes.  Results are
 *              bitwise the same either way.
 * token_ids int32 [N]; old_logp, ref_logp, adv_tok, w_tok float [N].
 * logp_out, tok_loss_out  float [N], nullable.  loss_out float [1], required.
 * dhidden    float [N][H], 16-byte aligned, overwritten; NULL skips it.
 * dweight    float [V][H], 16-byte aligned; overwritten (accumulate_dweight = 0) or added to
 *            (accumulate_dweight = 1); NULL skips it.  With both gradients
 *            NULL only the forward outputs are computed.
 * workspace  device buffer of >= leap_lmhead_workspace_size(N, V, H) bytes,
 *            16-byte aligned, scratch for this call only (calls sharing one
 *            workspace must be ordered on one stream).  It holds the
 *            gathered and transposed operands, per-tile row statistics, the
 *            live-row list and one vocabulary chunk of dZ (bf16, row-major).
 * Limits: each operand and workspace matrix below 4 GiB (32-bit offsets in
 * the GEMM core): for H = 4096, V up to about 520000, and N up to 130816
 * once V reaches 16384 (a dZ chunk holds N_pad x 16384 bf16; chunks are
 * 32768 columns for N up to 65280); otherwise LEAP_ERR_UNSUPPORTED.
 * Errors: LEAP_ERR_INVALID_ARG for N < 0, V < 1, H < 1, accumulate_dweight
 * not 0 or 1, a parameter out of range, a required pointer NULL;
 * LEAP_ERR_MISALIGNED; LEAP_ERR_WORKSPACE; LEAP_ERR_UNSUPPORTED.
 */
leap_status leap_grpo_lmhead_fwd_bwd(const void *hidden_bf16, const void *weight_bf16,
                                     const void *weight_t_bf16, int64_t N, int32_t V, int32_t H,
                                     const int32_t *token_ids,
                                     const float *old_logp, const float *ref_logp,
                                     const float *adv_tok, const float *w_tok,
                                     const leap_grpo_params *params, float *logp_out,
                                     float *tok_loss_out, float *loss_out, float *dhidden,
                                     float *dweight, int32_t accumulate_dweight, void *workspace,
                                     size_t ws_bytes, int32_t *dev_err, hipStream_t stream);

/*
 * Vocabulary-parallel form of the per-token objective (Sec. 3.1, Eq. 3 per
 * token) for logits split by vocabulary across devices (each device holds
 * columns [vocab_start, vocab_start + V_shard) of every row).  The three
 * calls are the local halves of one exchange: every shard runs
 * leap_vocab_shard_stats, the caller gathers the partials of all shards
 * (e.g. one all-gather of N x 16 bytes per shard), every shard runs
 * leap_vocab_merge_objective on the gathered partials, then
 * leap_vocab_shard_bwd for its own slice of dlogits.  The results equal
 * leap_grpo_logprob_loss_fwd_bwd on the concatenated rows up to fp32
 * rounding of the log-sum-exp.
 *
 * leap_vocab_shard_stats: partial [N][4] float (16-byte aligned), per row
 *   (m2, s, zy, owned) with c = log2(e) * inv_temperature,
 *   m2 = c * max_v x_v, s = sum_v 2^(c x_v - m2) over the shard's columns,
 *   owned = 1 and zy = x[y - vocab_start] when the token y = token_ids[k]
 *   falls in the shard, else owned = 0, zy = 0.  A row with w_tok[k] == 0
 *   (w_tok nullable) or whose shard columns are all -inf gives m2 = -inf,
 *   s = 0 and is not read in the first case.
 *   partial_t [N] float, nullable: the entropy partial
 *   t = sum_v 2^(c x_v - m2) * (c x_v - m2) over the shard's columns (0 when
 *   m2 = -inf); needed by leap_vocab_merge_objective's entropy output.
 *   logits_bf16 [N][ld] bf16 holding the shard's V_shard columns; alignment
 *   and range rules as leap_grpo_logprob_loss_fwd_bwd; vocab_start >= 0.
 * Errors: LEAP_ERR_INVALID_ARG for N < 0, V_shard < 1, ld < V_shard,
 * vocab_start < 0, a non-positive or non-finite inv_temperature, a required
 * pointer NULL; LEAP_ERR_MISALIGNED (logits or partial not 16-byte aligned,
 * ld % 8 != 0); LEAP_ERR_UNSUPPORTED for V_shard > LEAP_MAX_V.
 */
leap_status leap_vocab_shard_stats(const void *logits_bf16, int64_t ld, int64_t N, int32_t V_shard,
                                   int32_t vocab_start, const int32_t *token_ids,
                                   const float *w_tok, float inv_temperature, float *partial,
                                   float *partial_t, hipStream_t stream);

/* Workspace bytes leap_vocab_merge_objective needs for N rows. */
size_t leap_vocab_merge_workspace_size(int64_t N);

/*
 * leap_vocab_merge_objective: partials [n_shards][N][4] float (shard-major,
 *   16-byte aligned) from leap_vocab_shard_stats of every shard; the row's
 *   log-sum-exp is merged over shards in index order, then the per-token
 *   objective of leap_grpo_logprob_loss_fwd_bwd: logp_out, tok_loss_out
 *   (nullable), loss_out (required, fixed-order sum), and row_state [N][2]
 *   float (g, lse2 = log2 sum 2^(c x); 8-byte aligned), the input of
 *   leap_vocab_shard_bwd.  An excluded row gets logp = loss = 0 and
 *   row_state (0, +inf); a token id outside [0, V_total) with w != 0, a row
 *   whose token no shard (or more than one shard) reports, or a row of all
 *   -inf logits also counts in *dev_err.
 *   entropy_out [N] float, nullable: the row's entropy as in
 *   leap_grpo_logprob_loss_fwd_bwd (0 for an excluded row), merged from
 *   partials_t [n_shards][N] float (every shard's partial_t, shard-major),
 *   which it then requires.
 * Errors: LEAP_ERR_INVALID_ARG (N < 0, n_shards < 1, V_total < 1, a
 * parameter out of range, a required pointer NULL, entropy_out without
 * partials_t), LEAP_ERR_MISALIGNED,
 * LEAP_ERR_WORKSPACE, LEAP_ERR_UNSUPPORTED (unknown kl_type).
 */
leap_status leap_vocab_merge_objective(const float *partials, const float *partials_t,
                                       int32_t n_shards, int64_t N, int32_t V_total,
                                       const int32_t *token_ids, const float *old_logp,
                                       const float *ref_logp, const float *adv_tok,
                                       const float *w_tok, const leap_grpo_params *params,
                                       float *logp_out, float *tok_loss_out, float *entropy_out,
                                       float *loss_out, float *row_state, void *workspace,
                                       size_t ws_bytes, int32_t *dev_err, hipStream_t stream);

/*
 * leap_vocab_shard_bwd: dlogits[k][v] = g_k * ([vocab_start + v == y_k] -
 *   2^(c x[k][v] - lse2_k)) in bf16 (RNE) for the shard's V_shard columns,
 *   from row_state [N][2] of leap_vocab_merge_objective; a row with g == 0 is
 *   zero-filled without reading its logits.  dlogits_bf16 [N][ld] may equal
 *   logits_bf16, must not otherwise overlap it.
 * Errors: LEAP_ERR_INVALID_ARG for N < 0, V_shard < 1, ld < V_shard,
 * vocab_start < 0, a non-positive or non-finite inv_temperature, a required
 * pointer NULL, overlapping logits and dlogits; LEAP_ERR_MISALIGNED (logits,
 * dlogits not 16-byte aligned, ld % 8 != 0, row_state not 8-byte aligned);
 * LEAP_ERR_UNSUPPORTED for V_shard > LEAP_MAX_V.
 */
leap_status leap_vocab_shard_bwd(const void *logits_bf16, int64_t ld, int64_t N, int32_t V_shard,
                                 int32_t vocab_start, const int32_t *token_ids,
                                 const float *row_state, float inv_temperature,
                                 void *dlogits_bf16, hipStream_t stream);

/*
 * Training statistics of one step's rollouts, as the paper defines them
 * (Sec. 4): the pruning-range study's activated groups (gate = 1),
 * per-rollout recovery (trajectories of activated groups whose first turn
 * failed, and of those the ones that passed on a later turn) and per-group
 * recovery (activated groups that ran at least one such trajectory, and of
 * those the ones with at least one recovery); the turn efficiency (total
 * turns of all rollouts over passed rollouts); and the rollout-composition
 * analysis: rollouts with a nonzero advantage, by the observed pass rate of
 * their group (bucket floor(n_pass * n_buckets / G), the top bucket also
 * holding n_pass = G), outcome (immediate pass, debug-assisted pass,
 * failure) and advantage sign.
 *
 * pass_turn, n_turns  int32 [n_groups*G] (0 = never passed, else the turn of
 *   first pass; T_i turns generated).  gate uint8 [n_groups].
 * advantage float [n_groups*G], nullable (no composition then).
 * counters int64 [9 + 6*n_buckets], 8-byte aligned, overwritten:
 *   [0] groups [1] rollouts [2] activated groups [3] multi-turn trajectories
 *   [4] recovered trajectories [5] debugging groups [6] recovered groups
 *   [7] total turns [8] passed rollouts, then [9 + (b*3 + o)*2 + s] for
 *   bucket b, outcome o (0 immediate, 1 debug-assisted, 2 failure), sign s
 *   (0 positive, 1 negative).  Integer counts: exact, order independent.
 * A rollout with pass_turn outside 0..M or n_turns < 1 is skipped and counts
 * in *dev_err.
 * Errors: LEAP_ERR_INVALID_ARG for n_groups < 0, G outside 1..1024, M < 1,
 * n_buckets outside 1..256, a required pointer NULL; LEAP_ERR_MISALIGNED.
 */
leap_status leap_rollout_stats(const int32_t *pass_turn, const int32_t *n_turns,
                               const uint8_t *gate, const float *advantage, int64_t n_groups,
                               int32_t G, int32_t M, int32_t n_buckets, int64_t *counters,
                               int32_t *dev_err, hipStream_t stream);

/*
 * Measurement helper, not part of the method: the achievable bf16 matrix-core
 * rate.  n_workgroups workgroups of four waves each run `iters` rounds of
 * eight independent v_mfma_f32_16x16x32_bf16 (16384 flops each) on register
 * operands, with no memory traffic in the loop: 4 * n_workgroups * iters *
 * 8 * 16384 flops in all.
 * random_operands 0: every operand is 1.0, so the multipliers' inputs never
 *   change (the lowest switching power); sink float [n_workgroups], device
 *   memory: entry g receives iters * 32 (exact for iters < 2^19) when every
 *   chain of workgroup g ran all its rounds.
 * random_operands 1: each chain's operands are hashed bf16 values of
 *   magnitude [1, 2) with random signs, different per lane and chain, so
 *   consecutive MFMAs switch about half of their input bits, as a GEMM over
 *   random data does; entry g receives a finite sum of accumulators.
 * Errors: LEAP_ERR_INVALID_ARG for iters < 1, n_workgroups < 1,
 * random_operands outside 0..1, sink NULL.
 */
leap_status leap_probe_mfma(int64_t iters, int32_t n_workgroups, int32_t random_operands,
                            float *sink, hipStream_t stream);

/*
 * Measurement helper, not part of the method: streams device memory with the
 * access shape of the fused kernel (16-byte non-temporal accesses) so the
 * achievable HBM rate of each access mix can be set beside the published
 * peak.  mode 0: dst = src over `bytes` (read + write); 1: read src only
 * (dst receives at most 16 bytes); 2: write zeros to dst.
 * bytes % 16 == 0; src (modes 0, 1) and dst 16-byte aligned, device memory.
 * Errors: LEAP_ERR_INVALID_ARG for an unknown mode, bytes % 16 != 0 or a NULL
 * pointer that the mode needs; LEAP_ERR_MISALIGNED.
 */
leap_status leap_probe_hbm(const void *src, void *dst, size_t bytes, int32_t mode,
                           hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LEAP_H_ */
