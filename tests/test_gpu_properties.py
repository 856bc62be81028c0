"""GPU parity on hypothesis-generated inputs: random group sizes, turn
counts, ties and key modes for the tournament (K1) and the gate (K2), and
random masks and turn layouts for the token advantages (K3), each compared
with the oracle on the same inputs (integers and rewards bit-exact,
advantages within 1e-6, token advantages and weights within float32
rounding)."""
import numpy as np
import pytest
from hypothesis import HealthCheck, example, given, settings
from hypothesis import strategies as st

import oracle
import workloads as wl
from tests import _gpu_util as U
from tests.test_oracle_properties import groups, token_layouts

pytestmark = pytest.mark.gpu

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                           HealthCheck.function_scoped_fixture])


@SETTINGS
@given(groups(max_g=1024))
def test_tournament_matches_oracle(g):
    G, M, pt, sq, nt, lex = g
    key = oracle.KEY_LEX if lex else oracle.KEY_TURN
    gpu = U.run_rank(pt, G, M, key=key, speedup_q=sq if lex else None,
                     n_tokens=nt if lex else None)
    ora = oracle.rank_tournament(pt, G, M, key_mode=key, eps=U.EPS_ADV, speedup_q=sq,
                                 n_tokens=nt)
    U.check_rank(gpu, ora)


@SETTINGS
@given(st.integers(1, 1024), st.integers(1, 4), st.data())
def test_gate_matches_oracle(G, n_groups, data):
    p = data.draw(st.floats(0.0, 1.0))
    rng = np.random.default_rng(data.draw(st.integers(0, 2**31)))
    ftp = (rng.random(G * n_groups) < p).astype(np.uint8)
    tmin = data.draw(st.integers(0, G))
    tmax = data.draw(st.integers(tmin, G))
    nf_g, gate_g = U.run_gate(ftp, G, tmin, tmax)
    nf_o, gate_o = oracle.dcp_gate(ftp, G, tmin, tmax)
    assert np.array_equal(nf_g, nf_o) and np.array_equal(gate_g, gate_o)


@SETTINGS
@given(token_layouts(), st.sampled_from([oracle.AGG_SEQ_MEAN_TOKEN_MEAN, oracle.AGG_TOKEN_MEAN,
                                         oracle.AGG_SUM]))
# a subnormal advantage: gamma^2 A falls halfway between two subnormal floats
@example(lay=(np.array([0.0] * 5 + [9.99999935e-39] + [0.0] * 4),
              np.array([1, 1, 1, 1, 1, 3, 1, 1, 1, 1], dtype=np.int32),
              np.array([0, 1, 2, 3, 4, 5, 5, 5, 6, 7, 8, 9], dtype=np.int32),
              np.array([0, 0, 0, 0, 0, 0, 1, 2, 0, 0, 0, 0], dtype=np.int32), 0.5),
         agg=oracle.AGG_SEQ_MEAN_TOKEN_MEAN)
def test_token_advantages_match_oracle(lay, agg):
    A, T, tok_r, tok_t, gamma = lay
    A32 = A.astype(np.float32)
    g32 = float(np.float32(gamma))
    n_gen = np.bincount(tok_r[tok_r >= 0], minlength=A.size).astype(np.int32)
    denom = {oracle.AGG_SEQ_MEAN_TOKEN_MEAN: float(A.size),
             oracle.AGG_TOKEN_MEAN: float(n_gen.sum()), oracle.AGG_SUM: 1.0}[agg]
    adv_o, w_o, bad_o = oracle.token_advantages(A32.astype(np.float64), tok_r, tok_t, T, n_gen,
                                                g32, agg, denom)
    adv_g, w_g, bad_g = U.run_token_adv(A32, tok_r, tok_t, T, n_gen, gamma, agg, denom)
    assert bad_o == bad_g == 0
    U.check_f32_rounding(adv_g, adv_o, "token advantage")
    U.check_f32_rounding(w_g, w_o, "weight")


@st.composite
def objective_cases(draw):
    """One call of the fused objective: vocabulary width (every register
    shape of the kernel up to 65536 columns, odd widths included), padded
    row stride, rows, clip bounds (asymmetric), KL type and weight,
    temperature, old-policy spread, masked rows, bad token ids, -inf
    logits and the optional entropy output."""
    V = draw(st.one_of(st.integers(1, 700), st.integers(701, 40000),
                       st.sampled_from([16384, 32768, 50257, 65536])))
    ld = (V + 7) // 8 * 8 + draw(st.sampled_from([0, 8, 64]))
    return dict(
        V=V, ld=ld, N=draw(st.integers(1, 40)), seed=draw(st.integers(0, 2**31 - 1)),
        eps_lo=draw(st.floats(0.0, 0.5)), eps_hi=draw(st.floats(0.0, 0.5)),
        kl_coef=draw(st.floats(0.0, 0.5)),
        kl_type=draw(st.sampled_from([oracle.KL_K3, oracle.KL_K1, oracle.KL_K2])),
        inv_temp=draw(st.floats(0.5, 2.0)), old_sigma=draw(st.sampled_from([0.05, 0.3])),
        p_masked=draw(st.floats(0.0, 0.5)), n_bad=draw(st.integers(0, 2)),
        p_ninf=draw(st.sampled_from([0.0, 0.0, 0.01, 0.3])), entropy=draw(st.booleans()))


@settings(max_examples=40, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                 HealthCheck.function_scoped_fixture])
@given(objective_cases())
def test_fused_objective_matches_oracle(c):
    """The fused call against the oracle on random shapes and parameters:
    log-probs within 2e-3, per-token losses 2e-3 relative, the loss 1e-3
    relative, dlogits within 1e-2 of the largest entry plus 1e-6 (a
    boundary row may match either one-sided gradient), the entropy 1e-4
    relative, and the data-error count exact."""
    V, ld, N = c["V"], c["ld"], c["N"]
    rng = np.random.default_rng(c["seed"])

    def edit(lg, tok):
        if c["p_ninf"] > 0:
            keep = lg[np.arange(N), np.clip(tok, 0, V - 1)].copy()
            lg[:, :V][rng.random((N, V)) < c["p_ninf"]] = 0xFF80  # -inf
            lg[np.arange(N), np.clip(tok, 0, V - 1)] = keep  # the token's own logit stays

    lg, tok, old, ref = U.make_inputs_host(c["seed"] % 100000, N, V, ld=ld,
                                           old_sigma=c["old_sigma"], edit=edit)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = rng.uniform(0.1, 1.0, N).astype(np.float32)
    w[rng.random(N) < c["p_masked"]] = 0.0
    for k in rng.choice(N, size=min(c["n_bad"], N), replace=False):
        tok[k] = -1 if rng.random() < 0.5 else V
    kw = dict(eps_lo=c["eps_lo"], eps_hi=c["eps_hi"], kl_coef=c["kl_coef"],
              kl_type=c["kl_type"], inv_temp=c["inv_temp"])
    U.log(f"fused objective property case V={V} ld={ld} N={N} {kw}")
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, want_entropy=c["entropy"], **kw)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **kw)
    valid = (w != 0) & (tok >= 0) & (tok < V)
    assert gpu["bad"] == o["bad"] == int(((w != 0) & ~valid).sum())
    assert np.max(np.abs(gpu["logp"][valid] - o["logp"][valid]), initial=0) < 2e-3
    assert np.all(gpu["logp"][~valid] == 0) and np.all(gpu["tok_loss"][~valid] == 0)
    np.testing.assert_allclose(gpu["tok_loss"][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    assert abs(gpu["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-6
    rows = np.arange(N)
    d = U.dl_rows(gpu["dl_dev"], rows, V)
    assert np.all(d[~valid] == 0)
    # floor: the fp32 log-sum-exp leaves log-probs ~1e-7 of the logits' size
    # from the fp64 values, which shows as g * 1e-7 in entries the oracle
    # makes exactly 0 (a one-column row: p = 1, dlogits = 0)
    U.check_dlogits(d, lg, rows, tok, old, ref, adv, w, V, atol=1e-2, kw=kw, rel_to_max=True,
                    floor=1e-6)
    if c["entropy"]:
        h, _ = oracle.entropy_rows(lg, V=V, inv_temp=c["inv_temp"])
        assert np.all(gpu["entropy"][~valid] == 0)
        np.testing.assert_allclose(gpu["entropy"][valid], h[valid], rtol=1e-4, atol=2e-4)


@st.composite
def queue_cases(draw):
    """A microbatch for the persistent row-queue kernel: a width in its range
    (55297-155648 columns), more rows than the workgroups' four fixed rows
    each cover, masked runs of random lengths (long runs make workgroups
    refill the queue synchronously), random clip bounds, KL and the entropy
    output."""
    V = draw(st.integers(55297, 155648))
    N = draw(st.integers(1025, 3000))
    runs = draw(st.lists(st.tuples(st.integers(0, N - 1), st.integers(1, 1200)), max_size=4))
    return dict(V=V, N=N, runs=runs, seed=draw(st.integers(0, 2**31 - 1)),
                p_masked=draw(st.floats(0.0, 0.3)),
                eps_lo=draw(st.floats(0.0, 0.5)), eps_hi=draw(st.floats(0.0, 0.5)),
                kl_coef=draw(st.floats(0.0, 0.5)),
                kl_type=draw(st.sampled_from([oracle.KL_K3, oracle.KL_K1, oracle.KL_K2])),
                entropy=draw(st.booleans()))


@settings(max_examples=8, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                 HealthCheck.function_scoped_fixture])
@given(queue_cases())
def test_row_queue_matches_oracle(c):
    """The persistent row-queue kernel on random widths, row counts and mask
    runs against the oracle: every log-prob and per-token loss, the loss,
    the entropy, excluded rows zero-filled, and 32 sampled rows of dlogits
    (1e-2 of the largest entry)."""
    import torch
    V, N = c["V"], c["N"]
    ld = (V + 7) // 8 * 8
    rng = np.random.default_rng(c["seed"])
    U.log(f"row-queue property case V={V} N={N} runs={c['runs']}")
    lg_dev = torch.empty((N, ld), dtype=torch.bfloat16, device=U.dev())
    seed = c["seed"] % 100000
    wl.logits_device(seed, N, V, ld=ld, device=U.dev(), out=lg_dev)
    tok = wl.sample_tokens_device(lg_dev[:, :V], V, seed).cpu().numpy()
    lg = lg_dev.view(torch.int16).cpu().numpy().view(np.uint16)
    cur, _ = oracle.logprob_rows(lg, tok, V=V)
    old = (cur + rng.normal(0, 0.05, N)).astype(np.float32)
    ref = (cur + rng.normal(0, 0.1, N)).astype(np.float32)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = rng.uniform(0.1, 1.0, N).astype(np.float32)
    w[rng.random(N) < c["p_masked"]] = 0.0
    for s0, length in c["runs"]:
        w[s0:s0 + length] = 0.0
    kw = dict(eps_lo=c["eps_lo"], eps_hi=c["eps_hi"], kl_coef=c["kl_coef"],
              kl_type=c["kl_type"])
    gpu = U.run_grpo(lg_dev, V, tok, old, ref, adv, w, want_entropy=c["entropy"], **kw)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **kw)
    valid = w != 0
    assert gpu["bad"] == o["bad"] == 0
    assert np.max(np.abs(gpu["logp"][valid] - o["logp"][valid]), initial=0) < 2e-3
    assert np.all(gpu["logp"][~valid] == 0) and np.all(gpu["tok_loss"][~valid] == 0)
    np.testing.assert_allclose(gpu["tok_loss"][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    assert abs(gpu["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-6
    dead = torch.as_tensor(np.flatnonzero(~valid), device=U.dev())
    if dead.numel():
        assert int(gpu["dl_dev"].index_select(0, dead)[:, :V].view(torch.int16).abs().max()) == 0
    live = np.flatnonzero(valid)
    rows = live if live.size <= 32 else live[np.linspace(0, live.size - 1, 32).astype(int)]
    U.check_dlogits(U.dl_rows(gpu["dl_dev"], rows, V), lg, rows, tok, old, ref, adv, w, V,
                    atol=1e-2, kw=kw, rel_to_max=True, floor=1e-6)
    if c["entropy"]:
        h, _ = oracle.entropy_rows(lg, V=V)
        assert np.all(gpu["entropy"][~valid] == 0)
        np.testing.assert_allclose(gpu["entropy"][valid], h[valid], rtol=1e-4, atol=2e-4)


@st.composite
def shard_cases(draw):
    """A vocabulary split into 1-8 shards of random widths (one column
    upwards), with the objective's parameters drawn as for the fused call
    (temperature up to 1.5 and advantages within [-2, 2], so that bf16
    rounding of the largest gradient entries stays inside 2e-2)."""
    n = draw(st.integers(1, 8))
    widths = draw(st.lists(st.one_of(st.integers(1, 64), st.integers(65, 12000)), min_size=n,
                           max_size=n))
    return dict(widths=widths, V=sum(widths), N=draw(st.integers(1, 24)),
                seed=draw(st.integers(0, 2**31 - 1)),
                eps_lo=draw(st.floats(0.0, 0.5)), eps_hi=draw(st.floats(0.0, 0.5)),
                kl_coef=draw(st.floats(0.0, 0.5)),
                kl_type=draw(st.sampled_from([oracle.KL_K3, oracle.KL_K1, oracle.KL_K2])),
                inv_temp=draw(st.floats(0.5, 1.5)), p_masked=draw(st.floats(0.0, 0.5)),
                inplace=draw(st.booleans()))


@settings(max_examples=30, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                 HealthCheck.function_scoped_fixture])
@given(shard_cases())
def test_vocab_shards_match_unsharded_oracle(c):
    """Any split of the vocabulary: each shard's partial against the shard
    oracle, the merged objective against the unsharded oracle (log-probs
    2e-3, per-token losses 2e-3 relative, the loss 1e-3 relative) and the
    concatenated dlogits within 2e-2 of it (a row at a clip boundary may
    match either one-sided gradient)."""
    from tests import test_gpu_vocab_shard as S
    V, N = c["V"], c["N"]
    rng = np.random.default_rng(c["seed"])
    lg = wl.logits_host(c["seed"] % 100000, N, V)
    tok = wl.sample_tokens_host(lg, V, c["seed"] % 100000)
    cur, _ = oracle.logprob_rows(lg, tok, V=V)
    old = (cur + rng.normal(0, 0.2, N)).astype(np.float32)
    ref = (cur + rng.normal(0, 0.1, N)).astype(np.float32)
    adv = np.clip(rng.normal(0, 1, N), -2, 2).astype(np.float32)
    w = np.ones(N, np.float32)
    w[rng.random(N) < c["p_masked"]] = 0.0
    kw = dict(eps_lo=c["eps_lo"], eps_hi=c["eps_hi"], kl_coef=c["kl_coef"],
              kl_type=c["kl_type"], inv_temp=c["inv_temp"])
    shards = S._shards(V, c["widths"])
    U.log(f"vocab shard property case widths={c['widths']} N={N} {kw}")
    gpu = S._run(lg, V, tok, old, ref, adv, w, shards, kw, inplace=c["inplace"])
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **kw)
    valid = w != 0
    assert gpu["bad"] == o["bad"] == 0
    assert np.max(np.abs(gpu["logp"][valid] - o["logp"][valid]), initial=0) < 2e-3
    assert np.all(gpu["logp"][~valid] == 0) and np.all(gpu["tok_loss"][~valid] == 0)
    np.testing.assert_allclose(gpu["tok_loss"][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    assert abs(gpu["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-6
    d = U.bf16_f64(gpu["dl"])
    assert np.all(d[~valid] == 0)
    U.check_dlogits(d, lg, np.arange(N), tok, old, ref, adv, w, V, atol=2e-2, kw=kw)
    for k, (a, width) in enumerate(shards):
        m2, s, zy, owned = oracle.vocab_shard_stats(lg[:, a:a + width], a, tok, w=w,
                                                    inv_temp=kw["inv_temp"])
        q = gpu["parts"][k]
        np.testing.assert_array_equal(q[:, 3], owned)
        np.testing.assert_array_equal(q[:, 2], np.where(owned == 1, zy, 0))
        live = np.isfinite(m2)
        assert np.all(q[~live, 0] == -np.inf) and np.all(q[~live, 1] == 0)
        np.testing.assert_allclose(q[live, 0], m2[live], rtol=1e-6, atol=1e-6)
        np.testing.assert_allclose(q[live, 1], s[live], rtol=2e-5)


@settings(max_examples=30, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                 HealthCheck.function_scoped_fixture])
@given(st.one_of(st.integers(1, 700), st.integers(701, 70000)), st.sampled_from([0, 8, 64]),
       st.integers(1, 32), st.integers(0, 2**31 - 1), st.floats(0.5, 2.0),
       st.sampled_from([0.0, 0.01, 0.3]), st.booleans())
def test_logprob_fwd_matches_oracle(V, pad, N, seed, inv_temp, p_ninf, masked):
    """The forward-only pass on random widths, strides, temperatures, -inf
    logits and weight masks: log-probs within 2e-3 and entropies 1e-4
    relative of the oracle's; masked rows 0."""
    from tests import test_gpu_logprob_fwd as F
    rng = np.random.default_rng(seed)
    ld = (V + 7) // 8 * 8 + pad
    lg = wl.logits_host(seed % 100000, N, V, ld)
    tok = wl.sample_tokens_host(lg, V, seed % 100000)
    if p_ninf > 0:
        keep = lg[np.arange(N), tok].copy()
        lg[:, :V][rng.random((N, V)) < p_ninf] = 0xFF80
        lg[np.arange(N), tok] = keep
    w = (rng.random(N) >= 0.3).astype(np.float32) if masked else None
    U.log(f"logprob_fwd property case V={V} ld={ld} N={N} T^-1={inv_temp}")
    got, err, ent = F._run(U.bf16_device(lg), V, tok, w=w, inv_temp=inv_temp, want_entropy=True)
    want, bad = oracle.logprob_rows(lg, tok, V=V, inv_temp=inv_temp)
    h, _ = oracle.entropy_rows(lg, V=V, inv_temp=inv_temp)
    assert err == bad == 0
    live = np.ones(N, bool) if w is None else w != 0
    assert np.all(got[~live] == 0) and np.all(ent[~live] == 0)
    assert np.max(np.abs(got[live] - want[live]), initial=0) < 2e-3
    np.testing.assert_allclose(ent[live], h[live], rtol=1e-4, atol=2e-4)


@st.composite
def lmhead_cases(draw):
    """Small fused LM-head problems the fp64 oracle scores in well under a
    second: hidden width a multiple of the 64-deep k-tile, ragged rows and
    vocabularies (one to two 32768-column chunks), every KL estimator,
    temperatures, symmetric and clip-higher bounds, any share of excluded
    rows, either gradient left out, and the weight transposed beforehand or
    by the call."""
    H = draw(st.sampled_from([64, 128, 192, 320]))
    V = draw(st.one_of(st.integers(1, 700), st.integers(701, 40000)))
    N = draw(st.integers(1, max(1, min(600, int(6e7 // (V * H))))))
    return dict(N=N, V=V, H=H, seed=draw(st.integers(0, 2**16)),
                inv_temp=draw(st.sampled_from([1.0, 0.7, 1.3])),
                kl_type=draw(st.sampled_from([0, 1, 2])),
                eps=draw(st.sampled_from([(0.2, 0.2), (0.2, 0.28)])),
                mask_frac=draw(st.sampled_from([0.0, 0.05, 0.5, 1.0])),
                want=draw(st.sampled_from([(True, True), (True, False), (False, True)])),
                prepared=draw(st.booleans()))


@settings(max_examples=40, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                 HealthCheck.function_scoped_fixture])
@given(lmhead_cases())
def test_lmhead_matches_oracle(c):
    """The fused LM-head call against oracle.lmhead on random shapes and
    options, to the LM-head parity bars (log-prob 2e-3, loss 1e-3 relative,
    gradients under the |dZ|-scaled bound, excluded rows zero)."""
    N, V, H = c["N"], c["V"], c["H"]
    U.log(f"lmhead property case N={N} V={V} H={H} seed={c['seed']} T^-1={c['inv_temp']} "
          f"kl={c['kl_type']} eps={c['eps']} masked={c['mask_frac']} grads={c['want']} "
          f"prepared={c['prepared']}")
    inp = U.lmhead_inputs(c["seed"], N, V, H, mask_frac=c["mask_frac"], inv_temp=c["inv_temp"])
    kw = dict(eps_lo=c["eps"][0], eps_hi=c["eps"][1], kl_coef=0.05, kl_type=c["kl_type"],
              inv_temp=c["inv_temp"])
    gpu = U.run_lmhead(inp, want_dH=c["want"][0], want_dW=c["want"][1], prepared=c["prepared"],
                       **kw)
    assert (gpu["dH"] is None) != c["want"][0] and (gpu["dW"] is None) != c["want"][1]
    U.compare_lmhead(inp, gpu, kw, what=f"N={N} V={V} H={H}")


@st.composite
def stats_cases(draw):
    """Rollout statistics inputs: group sizes 1-1024, 1-6 turns, any gate,
    passes on any turn, advantages with ties and zeros (or none), bucket
    counts 1-256, and a few malformed rollouts."""
    G = draw(st.one_of(st.integers(1, 16), st.integers(17, 1024)))
    n_groups = draw(st.integers(1, max(1, min(64, 20000 // G))))
    return dict(G=G, n_groups=n_groups, M=draw(st.integers(1, 6)),
                nb=draw(st.one_of(st.integers(1, 16), st.integers(17, 256))),
                seed=draw(st.integers(0, 2**31 - 1)), with_adv=draw(st.booleans()),
                p_bad=draw(st.sampled_from([0.0, 0.0, 0.01])))


@settings(max_examples=40, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                 HealthCheck.function_scoped_fixture])
@given(stats_cases())
def test_rollout_stats_match_oracle(c):
    """Every counter of leap_rollout_stats bit-exact against the oracle on
    random groups, turn counts, gates, advantages and bucket counts."""
    from tests import test_gpu_rollout_stats as S
    G, M, n, nb = c["G"], c["M"], c["n_groups"], c["nb"]
    rng = np.random.default_rng(c["seed"])
    gate = rng.integers(0, 2, n).astype(np.uint8)
    p_pass = rng.random(n).repeat(G)
    pt = np.where(rng.random(n * G) < p_pass, rng.integers(1, M + 1, n * G), 0).astype(np.int32)
    single = np.repeat(gate == 0, G)
    pt[single & (pt > 1)] = 0  # groups without expansion stop after the first turn
    nt = np.where(pt >= 1, pt, np.where(single, 1, M)).astype(np.int32)
    bad = rng.random(n * G) < c["p_bad"]
    pt[bad & (rng.random(n * G) < 0.5)] = M + 1
    nt[bad & (pt <= M)] = 0
    adv = None
    if c["with_adv"]:
        adv = np.round(rng.normal(0, 1, n * G), 1)
        adv[rng.random(n * G) < 0.2] = 0.0
    U.log(f"rollout stats property case {n} x {G}, M={M}, buckets={nb}, "
          f"adv={c['with_adv']}, bad={int(bad.sum())}")
    got, gbad = S._gpu(pt, nt, gate, adv, G, M, nb)
    want, wbad = S._expect(pt, nt, gate, adv, G, M, nb)
    np.testing.assert_array_equal(got, want)
    assert gbad == wbad
