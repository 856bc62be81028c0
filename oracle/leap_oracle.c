/*
 * LEAP oracle -- plain, slow, obviously correct fp64 CPU definitions of the
 * GRPO hot path of "LEAP: Lean Environment-Feedback via Adaptive Pruning for
 * Code RL in GPU Kernel Generation" (arXiv 2608.01804).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or helper with the HIP library: the two are written
 * separately from the paper so that one can check the other.
 *
 * Every step is written in the order and notation of the paper, in double
 * precision, with no blocking or fusion:
 *   - Sec. 3.2, Eq. 4        tier r(o_i) from the turn of first pass
 *   - Sec. 3.2, Eq. 5        pairwise tournament counts N_worse, N_better
 *   - Sec. 3.2, Eq. 6        tournament reward R_i = (N_worse - N_better)/(G-1)
 *   - Sec. 3.2 (end)         "standard GRPO" advantage from R_i
 *   - Sec. 3.1, Eqs. 1-2     DCP failure count and gate
 *   - Sec. 3.3               discounted per-turn token advantage
 *   - Sec. 3.1, Eq. 3 and
 *     Sec. 4.1               per-token clipped surrogate, reference KL,
 *                            sample-level aggregation weight, and the
 *                            gradient with respect to the logits.
 *
 * Parallelism: OpenMP over independent rows / groups only; every sum that
 * crosses rows is taken afterwards, sequentially, in index order.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Keys and modes: values mirror the public enums of the library, but are
 * restated here on purpose (the oracle includes nothing from the library). */
enum { OR_KEY_TURN = 0, OR_KEY_LEX = 1 };
enum { OR_ADV_STD = 0, OR_ADV_NONE = 1 };
enum { OR_AGG_SEQ_MEAN_TOKEN_MEAN = 0, OR_AGG_TOKEN_MEAN = 1, OR_AGG_SUM = 2 };
enum { OR_KL_K3 = 0, OR_KL_K1 = 1, OR_KL_K2 = 2 };

/* ------------------------------------------------------------------------ */
/* threads                                                                  */
/* ------------------------------------------------------------------------ */
void leap_oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int leap_oracle_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.2, Eq. 4: tier of a rollout.                                      */
/* pass_turn m = 0 means the rollout never passed verification; m in 1..M   */
/* means it first passed on turn m.  A pass on turn m ranks r = M - m + 1,  */
/* a final failure ranks r = 0.  Returns -1 for an m outside 0..M.          */
/* ------------------------------------------------------------------------ */
static int tier_of(int32_t m, int32_t M)
{
    if (m < 0 || m > M) return -1;
    if (m == 0) return 0;
    return M - m + 1;
}

/* Strict preference between two outcomes.
 * TURN key: the paper's order, by tier only (Eq. 4).
 * LEX key (an extension, not in the paper): tier first, then the larger
 * quantised speedup, then the smaller generated-token count.
 * Returns +1 if a is strictly preferred, -1 if b is, 0 on a tie. */
static int compare_outcome(int key_mode, int ra, int32_t sa, int32_t na,
                           int rb, int32_t sb, int32_t nb)
{
    if (ra > rb) return 1;
    if (ra < rb) return -1;
    if (key_mode == OR_KEY_LEX) {
        if (sa > sb) return 1;
        if (sa < sb) return -1;
        if (na < nb) return 1;
        if (na > nb) return -1;
    }
    return 0;
}

/*
 * Rank-based reward and GRPO advantage, one group of G rollouts at a time.
 *
 * Eq. 5: N_worse(o_i) counts peers j != i with r(o_i) > r(o_j); N_better(o_i)
 * counts peers with r(o_i) < r(o_j); ties count for neither.
 * Eq. 6: R_i = (N_worse - N_better) / (G - 1).
 * Advantage ("standard GRPO formulation", end of Sec. 3.2), read as the
 * group-normalised form A_i = (R_i - mean R) / (std R + eps) with the
 * unbiased (G - 1) standard deviation; adv_norm = NONE gives A_i = R_i.
 *
 * Arrays are group-major: rollout i of group g sits at g*G + i.
 * speedup_q and n_tokens are read only in LEX mode.
 * Returns the number of pass_turn entries outside 0..M; such a rollout is
 * ranked as a failure (r = 0).
 */
int64_t leap_oracle_rank_tournament(const int32_t *pass_turn,
                                    const int32_t *speedup_q,
                                    const int32_t *n_tokens,
                                    int64_t n_groups, int32_t G, int32_t M,
                                    int32_t key_mode, int32_t adv_norm,
                                    double eps,
                                    int32_t *rank_r, int32_t *n_worse,
                                    int32_t *n_better, double *reward,
                                    double *advantage)
{
    int64_t bad = 0;
    int64_t g;
#pragma omp parallel for schedule(static) reduction(+ : bad)
    for (g = 0; g < n_groups; ++g) {
        const int64_t base = g * (int64_t)G;
        int i, j;
        int *r = (int *)malloc(sizeof(int) * (size_t)G);
        /* Eq. 4 */
        for (i = 0; i < G; ++i) {
            int t = tier_of(pass_turn[base + i], M);
            if (t < 0) { t = 0; bad += 1; }
            r[i] = t;
            rank_r[base + i] = t;
        }
        /* Eq. 5: a complete pairwise tournament */
        for (i = 0; i < G; ++i) {
            int32_t worse = 0, better = 0;
            for (j = 0; j < G; ++j) {
                int c;
                if (j == i) continue;
                c = compare_outcome(key_mode,
                                    r[i], key_mode == OR_KEY_LEX ? speedup_q[base + i] : 0,
                                    key_mode == OR_KEY_LEX ? n_tokens[base + i] : 0,
                                    r[j], key_mode == OR_KEY_LEX ? speedup_q[base + j] : 0,
                                    key_mode == OR_KEY_LEX ? n_tokens[base + j] : 0);
                if (c > 0) worse += 1;
                if (c < 0) better += 1;
            }
            n_worse[base + i] = worse;
            n_better[base + i] = better;
            /* Eq. 6 */
            reward[base + i] = (double)(worse - better) / (double)(G - 1);
        }
        /* GRPO advantage */
        if (adv_norm == OR_ADV_NONE) {
            for (i = 0; i < G; ++i) advantage[base + i] = reward[base + i];
        } else {
            double mean = 0.0, var = 0.0, sd;
            for (i = 0; i < G; ++i) mean += reward[base + i];
            mean /= (double)G;
            for (i = 0; i < G; ++i) {
                double d = reward[base + i] - mean;
                var += d * d;
            }
            var /= (double)(G - 1);
            sd = sqrt(var);
            for (i = 0; i < G; ++i)
                advantage[base + i] = (reward[base + i] - mean) / (sd + eps);
        }
        free(r);
    }
    return bad;
}

/*
 * Difficulty-Conditioned Pruning, Sec. 3.1.
 * Eq. 1: N_fail(q) = number of rollouts of the group whose first-turn
 * response failed verification (first_turn_pass == 0).
 * Eq. 2: gate = 1 iff tau_min <= N_fail <= tau_max, else 0.
 */
void leap_oracle_dcp_gate(const uint8_t *first_turn_pass, int64_t n_groups,
                          int32_t G, int32_t tau_min, int32_t tau_max,
                          int32_t *n_fail, uint8_t *gate)
{
    int64_t g;
#pragma omp parallel for schedule(static)
    for (g = 0; g < n_groups; ++g) {
        int32_t nf = 0;
        int i;
        for (i = 0; i < G; ++i)
            if (first_turn_pass[g * (int64_t)G + i] == 0) nf += 1;
        n_fail[g] = nf;
        gate[g] = (uint8_t)((tau_min <= nf && nf <= tau_max) ? 1 : 0);
    }
}

/*
 * Discounted per-turn token advantage, Sec. 3.3, and the aggregation weight
 * of the sample-level loss (Sec. 4.1; Eq. 3's 1/G sum over samples).
 *
 * Token k belongs to rollout i = tok_rollout[k] (-1: excluded -- padding,
 * prompt or environment feedback) and to generated turn t = tok_turn[k] of
 * that rollout's T_i = n_turns[i] generated turns.
 *   beta_i    = gamma if A_i >= 0, else 1
 *   Ahat_{ik} = beta_i^(T_i - t - 1) * A_i
 * Weight w_k:
 *   SEQ_MEAN_TOKEN_MEAN : 1 / (denom * |M_i|), |M_i| = n_gen_tokens[i],
 *                         denom = number of sequences in the step
 *   TOKEN_MEAN          : 1 / denom, denom = generated tokens in the step
 *   SUM                 : 1
 * Excluded tokens get Ahat = 0 and w = 0.  A token whose rollout index is
 * below -1 or not below n_rollouts, whose turn is outside 0..T_i-1, or whose
 * rollout has no generated tokens is counted as an error and excluded.
 * Returns the error count.
 */
int64_t leap_oracle_token_advantages(const double *A, const int32_t *tok_rollout,
                                     const int32_t *tok_turn,
                                     const int32_t *n_turns,
                                     const int32_t *n_gen_tokens,
                                     int32_t n_rollouts, int64_t N,
                                     double gamma, int32_t agg, double denom,
                                     double *adv_tok, double *w_tok)
{
    int64_t bad = 0;
    int64_t k;
#pragma omp parallel for schedule(static) reduction(+ : bad)
    for (k = 0; k < N; ++k) {
        int32_t i = tok_rollout[k];
        int32_t t, T;
        double beta, a;
        adv_tok[k] = 0.0;
        w_tok[k] = 0.0;
        if (i == -1) continue;
        if (i < -1 || i >= n_rollouts) { bad += 1; continue; }
        t = tok_turn[k];
        T = n_turns[i];
        if (T < 1 || t < 0 || t >= T || n_gen_tokens[i] < 1) { bad += 1; continue; }
        a = A[i];
        beta = (a >= 0.0) ? gamma : 1.0;
        adv_tok[k] = pow(beta, (double)(T - t - 1)) * a;
        if (agg == OR_AGG_SEQ_MEAN_TOKEN_MEAN)
            w_tok[k] = 1.0 / (denom * (double)n_gen_tokens[i]);
        else if (agg == OR_AGG_TOKEN_MEAN)
            w_tok[k] = 1.0 / denom;
        else
            w_tok[k] = 1.0;
    }
    return bad;
}

/* ------------------------------------------------------------------------ */
/* Per-token GRPO objective on one row of logits.                           */
/* ------------------------------------------------------------------------ */

/* bf16 -> double is exact: a bf16 value is the upper half of an fp32. */
static double bf16_to_double(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Log-softmax of z (length V) at y: returns log p_y and writes lse. */
static double log_softmax_at(const double *z, int32_t V, int32_t y, double *lse_out)
{
    double m = -INFINITY, s = 0.0, lse;
    int32_t v;
    for (v = 0; v < V; ++v)
        if (z[v] > m) m = z[v];
    if (m == -INFINITY) { *lse_out = -INFINITY; return NAN; }
    for (v = 0; v < V; ++v) s += exp(z[v] - m);
    lse = m + log(s);
    *lse_out = lse;
    return z[y] - lse;
}

/*
 * One row of the per-token objective (Sec. 3.1, Eq. 3, with the surrogate
 * and KL read as PPO-clip and GRPO's k3 estimator) and its gradient:
 *   logp  = z_y - logsumexp(z)
 *   rho   = exp(logp - old_logp)
 *   surr  = min(rho * Ahat, clip(rho, 1 - eps_lo, 1 + eps_hi) * Ahat)
 *   KL    = k3: exp(ref - logp) - (ref - logp) - 1
 *           k1: logp - ref          k2: (logp - ref)^2 / 2
 *   loss  = -surr + beta * KL
 *   dloss/dlogp = -Ahat * rho * [clip inactive] + beta * dKL/dlogp
 *   dlogits_v   = w * dloss/dlogp * inv_temp * ([v == y] - softmax(z)_v)
 * z = inv_temp * logits.  Returns 0 on success, 1 when the row is invalid
 * (token id out of range, or every logit is -inf); an invalid row is
 * treated as masked.
 */
static int grpo_row(const double *x, int32_t V, int32_t y, double old_lp,
                    double ref_lp, double ahat, double w, double eps_lo,
                    double eps_hi, double kl_coef, int32_t kl_type,
                    double inv_temp, double *z_scratch, double *logp_out,
                    double *loss_out, double *dlog_row)
{
    int32_t v;
    double lse, logp, rho, clipped, surr, kl, dkl, dl, g;
    int active;

    *logp_out = 0.0;
    *loss_out = 0.0;
    if (dlog_row) for (v = 0; v < V; ++v) dlog_row[v] = 0.0;
    if (w == 0.0) return 0;
    if (y < 0 || y >= V) return 1;

    for (v = 0; v < V; ++v) z_scratch[v] = inv_temp * x[v];
    logp = log_softmax_at(z_scratch, V, y, &lse);
    if (lse == -INFINITY) return 1;

    rho = exp(logp - old_lp);
    clipped = rho;
    if (clipped < 1.0 - eps_lo) clipped = 1.0 - eps_lo;
    if (clipped > 1.0 + eps_hi) clipped = 1.0 + eps_hi;
    surr = fmin(rho * ahat, clipped * ahat);

    if (kl_type == OR_KL_K1) {
        kl = logp - ref_lp;
        dkl = 1.0;
    } else if (kl_type == OR_KL_K2) {
        kl = 0.5 * (logp - ref_lp) * (logp - ref_lp);
        dkl = logp - ref_lp;
    } else {
        double d = ref_lp - logp;
        kl = exp(d) - d - 1.0;
        dkl = 1.0 - exp(d);
    }

    *logp_out = logp;
    *loss_out = -surr + kl_coef * kl;

    active = (ahat > 0.0 && rho <= 1.0 + eps_hi) || (ahat < 0.0 && rho >= 1.0 - eps_lo);
    dl = (active ? -ahat * rho : 0.0) + kl_coef * dkl;
    g = w * dl * inv_temp;
    if (dlog_row) {
        for (v = 0; v < V; ++v) {
            double p = exp(z_scratch[v] - lse);
            dlog_row[v] = g * ((v == y ? 1.0 : 0.0) - p);
        }
    }
    return 0;
}

/*
 * The fused per-token pass over a block of rows, on fp64 logits.
 * logits: [N][ld] doubles (row k at k*ld, V used).  sel_rows (nullable) lists
 * the n_sel rows to evaluate, in any order; NULL means rows 0..N-1 with
 * n_sel = N.  Outputs are indexed by position j in the selection:
 * logp[j], tok_loss[j] (unweighted per-token loss), dlogits[j*V + v]
 * (nullable).  *loss_total = sum_j w_j * loss_j, summed in selection order.
 * Returns the number of invalid rows.
 */
int64_t leap_oracle_grpo_rows_f64(const double *logits, int64_t ld, int64_t N,
                                  int32_t V, const int32_t *token_ids,
                                  const double *old_logp, const double *ref_logp,
                                  const double *adv, const double *w,
                                  double eps_lo, double eps_hi, double kl_coef,
                                  int32_t kl_type, double inv_temp,
                                  int64_t n_sel, const int64_t *sel_rows,
                                  double *logp, double *tok_loss,
                                  double *loss_total, double *dlogits)
{
    int64_t bad = 0, j;
    double total = 0.0;
    if (!sel_rows) n_sel = N;
#pragma omp parallel reduction(+ : bad)
    {
        double *zs = (double *)malloc(sizeof(double) * (size_t)(V > 0 ? V : 1));
        int64_t jj;
#pragma omp for schedule(dynamic, 4)
        for (jj = 0; jj < n_sel; ++jj) {
            int64_t k = sel_rows ? sel_rows[jj] : jj;
            bad += grpo_row(logits + k * ld, V, token_ids[k], old_logp[k],
                            ref_logp[k], adv[k], w[k], eps_lo, eps_hi, kl_coef,
                            kl_type, inv_temp, zs, &logp[jj], &tok_loss[jj],
                            dlogits ? dlogits + jj * (int64_t)V : NULL);
        }
        free(zs);
    }
    for (j = 0; j < n_sel; ++j) {
        int64_t k = sel_rows ? sel_rows[j] : j;
        total += w[k] * tok_loss[j];
    }
    *loss_total = total;
    return bad;
}

/* The same pass on bf16 logits ([N][ld] uint16 bit patterns), each row
 * converted exactly to fp64 first. */
int64_t leap_oracle_grpo_rows_bf16(const uint16_t *logits, int64_t ld, int64_t N,
                                   int32_t V, const int32_t *token_ids,
                                   const double *old_logp, const double *ref_logp,
                                   const double *adv, const double *w,
                                   double eps_lo, double eps_hi, double kl_coef,
                                   int32_t kl_type, double inv_temp,
                                   int64_t n_sel, const int64_t *sel_rows,
                                   double *logp, double *tok_loss,
                                   double *loss_total, double *dlogits)
{
    int64_t bad = 0, j;
    double total = 0.0;
    if (!sel_rows) n_sel = N;
#pragma omp parallel reduction(+ : bad)
    {
        double *xs = (double *)malloc(sizeof(double) * (size_t)(V > 0 ? V : 1));
        double *zs = (double *)malloc(sizeof(double) * (size_t)(V > 0 ? V : 1));
        int64_t jj;
        int32_t v;
#pragma omp for schedule(dynamic, 4)
        for (jj = 0; jj < n_sel; ++jj) {
            int64_t k = sel_rows ? sel_rows[jj] : jj;
            const uint16_t *row = logits + k * ld;
            for (v = 0; v < V; ++v) xs[v] = bf16_to_double(row[v]);
            bad += grpo_row(xs, V, token_ids[k], old_logp[k], ref_logp[k],
                            adv[k], w[k], eps_lo, eps_hi, kl_coef, kl_type,
                            inv_temp, zs, &logp[jj], &tok_loss[jj],
                            dlogits ? dlogits + jj * (int64_t)V : NULL);
        }
        free(xs);
        free(zs);
    }
    for (j = 0; j < n_sel; ++j) {
        int64_t k = sel_rows ? sel_rows[j] : j;
        total += w[k] * tok_loss[j];
    }
    *loss_total = total;
    return bad;
}

/*
 * Forward-only log-probability of each row's token under softmax(inv_temp *
 * logits) -- the quantity the old-policy and reference forward passes
 * produce for the ratio and the KL of Eq. 3.  Rows with an out-of-range
 * token id or all -inf logits get NaN and are counted.
 */
int64_t leap_oracle_logprob_rows_bf16(const uint16_t *logits, int64_t ld,
                                      int64_t N, int32_t V,
                                      const int32_t *token_ids, double inv_temp,
                                      double *logp)
{
    int64_t bad = 0;
#pragma omp parallel reduction(+ : bad)
    {
        double *zs = (double *)malloc(sizeof(double) * (size_t)(V > 0 ? V : 1));
        int64_t k;
        int32_t v;
#pragma omp for schedule(dynamic, 4)
        for (k = 0; k < N; ++k) {
            const uint16_t *row = logits + k * ld;
            double lse;
            int32_t y = token_ids[k];
            if (y < 0 || y >= V) { logp[k] = NAN; bad += 1; continue; }
            for (v = 0; v < V; ++v) zs[v] = inv_temp * bf16_to_double(row[v]);
            logp[k] = log_softmax_at(zs, V, y, &lse);
            if (lse == -INFINITY) { logp[k] = NAN; bad += 1; }
        }
        free(zs);
    }
    return bad;
}

/*
 * Shannon entropy, in nats, of each row's token distribution
 * p = softmax(inv_temp * logits): H = -sum_v p_v log p_v, a per-token
 * quantity training logs beside the objective of Eq. 3 (the paper itself
 * defines no entropy term).  Columns with p_v = 0 (-inf logits) contribute
 * 0.  Rows whose logits are all -inf get NaN and are counted.
 */
int64_t leap_oracle_entropy_rows_bf16(const uint16_t *logits, int64_t ld,
                                      int64_t N, int32_t V, double inv_temp,
                                      double *ent)
{
    int64_t bad = 0;
#pragma omp parallel reduction(+ : bad)
    {
        double *zs = (double *)malloc(sizeof(double) * (size_t)(V > 0 ? V : 1));
        int64_t k;
        int32_t v;
#pragma omp for schedule(dynamic, 4)
        for (k = 0; k < N; ++k) {
            const uint16_t *row = logits + k * ld;
            double lse, h = 0.0;
            for (v = 0; v < V; ++v) zs[v] = inv_temp * bf16_to_double(row[v]);
            (void)log_softmax_at(zs, V, 0, &lse);
            if (lse == -INFINITY) { ent[k] = NAN; bad += 1; continue; }
            for (v = 0; v < V; ++v) {
                const double logp = zs[v] - lse;
                const double p = exp(logp);
                if (p > 0.0) h -= p * logp;
            }
            ent[k] = h;
        }
        free(zs);
    }
    return bad;
}

/*
 * Training statistics of the method (test infrastructure like the rest).
 *
 * Definitions followed:
 *   - pruning-range study (Sec. 4, the DCP analysis): "activated groups" =
 *     groups whose gate sends them to multi-turn debugging; "per-rollout
 *     recovery" = among the trajectories that failed their first turn and
 *     entered debugging, those that later pass; "per-group recovery" = among
 *     the groups that ran debugging, those with at least one recovered
 *     trajectory;
 *   - method comparison (turn efficiency): total turns used by all samples,
 *     and passed samples (the ratio is turns per pass);
 *   - rollout-composition analysis: rollouts with a nonzero advantage,
 *     bucketed by the observed pass rate of their group, split by outcome
 *     (immediate pass, debug-assisted pass, failure) and advantage sign.
 *
 * counters[0..8]: groups, rollouts, activated groups, multi-turn
 * trajectories, recovered trajectories, debugging groups, recovered groups,
 * total turns, passed rollouts; then comp[b][o][s] (b < n_buckets, o in 0..2,
 * s: 0 positive, 1 negative) at counters[9 + (b*3 + o)*2 + s].  The bucket
 * of a group with n_pass passes is floor(n_pass * n_buckets / G), the top
 * bucket also holding n_pass = G.  A rollout with pass_turn outside 0..M or
 * n_turns < 1 is skipped everywhere and counted in the return value.
 * advantage may be NULL (no composition).
 */
int64_t leap_oracle_rollout_stats(const int32_t *pass_turn, const int32_t *n_turns,
                                  const uint8_t *gate, const double *advantage,
                                  int64_t n_groups, int32_t G, int32_t M, int32_t n_buckets,
                                  int64_t *counters)
{
    int64_t bad = 0;
    const int64_t n_counters = 9 + (int64_t)n_buckets * 6;
    for (int64_t k = 0; k < n_counters; ++k) counters[k] = 0;
    counters[0] = n_groups;
    counters[1] = n_groups * (int64_t)G;
    for (int64_t g = 0; g < n_groups; ++g) {
        const int64_t base = g * (int64_t)G;
        const int activated = gate[g] != 0;
        int64_t n_pass = 0, n_multi = 0, n_recovered = 0;
        for (int32_t i = 0; i < G; ++i) {
            const int32_t m = pass_turn[base + i];
            const int32_t T = n_turns[base + i];
            if (m < 0 || m > M || T < 1) {
                ++bad;
                continue;
            }
            counters[7] += T;
            if (m >= 1) ++n_pass;
            if (activated && m != 1) {  /* first turn failed: debugging ran */
                ++n_multi;
                if (m >= 2) ++n_recovered;
            }
        }
        counters[8] += n_pass;
        if (activated) {
            ++counters[2];
            counters[3] += n_multi;
            counters[4] += n_recovered;
            if (n_multi > 0) {
                ++counters[5];
                if (n_recovered > 0) ++counters[6];
            }
        }
        if (advantage == NULL || n_buckets < 1) continue;
        int64_t b = n_pass * (int64_t)n_buckets / G;
        if (b > n_buckets - 1) b = n_buckets - 1;
        for (int32_t i = 0; i < G; ++i) {
            const int32_t m = pass_turn[base + i];
            const int32_t T = n_turns[base + i];
            if (m < 0 || m > M || T < 1) continue;
            const double a = advantage[base + i];
            if (a == 0.0 || a != a) continue;
            const int o = (m == 1) ? 0 : (m >= 2 ? 1 : 2);
            const int s = a > 0.0 ? 0 : 1;
            ++counters[9 + (b * 3 + o) * 2 + s];
        }
    }
    return bad;
}
