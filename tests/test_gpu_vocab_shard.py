"""Parity of the vocabulary-parallel entry points (leap_vocab_shard_stats,
leap_vocab_merge_objective, leap_vocab_shard_bwd) with the oracle: each
shard's partial against ``oracle.vocab_shard_stats``; the merged per-token
objective and the concatenated per-shard dlogits against the unsharded
oracle (``oracle.grpo_rows`` on the whole rows), with the tolerances of the
unsharded kernel (log-prob 2e-3 absolute, loss 1e-3 relative, dlogits 2e-2
absolute with unit weights)."""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu

KW = dict(eps_lo=0.2, eps_hi=0.2, kl_coef=0.01, kl_type=0, inv_temp=1.0)


def _shards(V, widths):
    starts = np.concatenate([[0], np.cumsum(widths)[:-1]]).astype(int)
    assert sum(widths) <= V
    return list(zip(starts.tolist(), list(widths)))


def _run(lg, V, tok, old, ref, adv, w, shards, kw, inplace=False, want_entropy=False):
    """lg: host bf16 bit patterns [N, ld]; returns partials (n_shards, N, 4),
    merged outputs and the concatenated dlogits [N, V] (uint16)."""
    import torch
    from paper_2608_01804_amd import leap as L
    N = lg.shape[0]
    dev = U.dev()
    parts = torch.full((len(shards), max(N, 1), 4), float("nan"), dtype=torch.float32, device=dev)
    parts_t = (torch.full((len(shards), max(N, 1)), float("nan"), dtype=torch.float32, device=dev)
               if want_entropy else None)
    shard_dev = []
    tok_d, w_d = U.T(np.asarray(tok, np.int32)), U.T(np.asarray(w, np.float32))
    for k, (a, width) in enumerate(shards):
        ld = (width + 7) // 8 * 8
        buf = np.zeros((N, ld), np.uint16)
        buf[:, :width] = lg[:, a:a + width]
        t = torch.from_numpy(buf.view(np.int16)).to(dev).view(torch.bfloat16)
        shard_dev.append((t, ld))
        L.leap_vocab_shard_stats(t, ld, N, width, a, tok_d, w_d, kw["inv_temp"], parts[k],
                                 partial_t=parts_t[k] if want_entropy else None)
    p = L.leap_grpo_params(kw["eps_lo"], kw["eps_hi"], kw["kl_coef"], kw["kl_type"], kw["inv_temp"])
    lp = torch.full((max(N, 1),), float("nan"), dtype=torch.float32, device=dev)
    tl = torch.full_like(lp, float("nan"))
    loss = torch.full((1,), float("nan"), dtype=torch.float32, device=dev)
    state = torch.full((max(N, 1), 2), float("nan"), dtype=torch.float32, device=dev)
    ws_bytes = L.leap_vocab_merge_workspace_size(N)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    err = U.zeros_i32(1)
    ent = torch.full_like(lp, float("nan")) if want_entropy else None
    L.leap_vocab_merge_objective(parts, len(shards), N, V, tok_d, U.T(np.asarray(old, np.float32)),
                                 U.T(np.asarray(ref, np.float32)), U.T(np.asarray(adv, np.float32)),
                                 w_d, p, lp, tl, loss, state, ws, ws_bytes, err,
                                 partials_t=parts_t, entropy_out=ent)
    out = np.zeros((N, V), np.uint16)
    for (a, width), (t, ld) in zip(shards, shard_dev):
        d = t if inplace else torch.full_like(t, float("nan"))
        L.leap_vocab_shard_bwd(t, ld, N, width, a, tok_d, state, kw["inv_temp"], d)
        out[:, a:a + width] = d.view(torch.int16).cpu().numpy().view(np.uint16)[:, :width]
    torch.cuda.synchronize()
    return {"parts": parts.cpu().numpy()[:, :N], "logp": lp.cpu().numpy()[:N],
            "tok_loss": tl.cpu().numpy()[:N], "loss": float(loss.item()),
            "state": state.cpu().numpy()[:N], "bad": int(err.item()), "dl": out,
            "entropy": ent.cpu().numpy()[:N] if want_entropy else None}


def _check(lg, V, tok, old, ref, adv, w, shards, gpu, kw, atol_dl=2e-2, bad=0):
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, **kw)
    valid = (w != 0) & (tok >= 0) & (tok < V)
    assert gpu["bad"] == bad, gpu["bad"]
    err = np.max(np.abs(gpu["logp"][valid] - o["logp"][valid]), initial=0)
    U.log(f"  logp max err {err:.3e}")
    assert err < 2e-3
    assert np.all(gpu["logp"][~valid] == 0) and np.all(gpu["tok_loss"][~valid] == 0)
    np.testing.assert_allclose(gpu["tok_loss"][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    assert abs(gpu["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-7
    dl = U.bf16_f64(gpu["dl"])
    derr = np.max(np.abs(dl[valid] - o["dlogits"][valid]), initial=0)
    U.log(f"  dlogits max err {derr:.3e}")
    assert derr <= atol_dl
    assert np.all(gpu["dl"][~valid] == 0)
    # each shard's partial against the shard oracle
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


@pytest.mark.parametrize("widths", [[18992] * 8, [10000, 10000, 12768]])
def test_shards_match_unsharded_oracle(widths):
    V = sum(widths)
    N = 512
    U.log(f"vocab shards {widths[:2]}.. x{len(widths)} V={V} N={N}")
    lg = wl.logits_host(3101, N, V)
    tok = wl.sample_tokens_host(lg, V, 3101)
    cur, _ = oracle.logprob_rows(lg, tok, V=V)
    n_old, n_ref = wl.logp_noise(3101, N)
    old, ref = (cur + n_old).astype(np.float32), (cur + n_ref).astype(np.float32)
    rng = np.random.default_rng(3101)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = np.ones(N, np.float32)
    w[rng.random(N) < 0.05] = 0.0
    shards = _shards(V, widths)
    gpu = _run(lg, V, tok, old, ref, adv, w, shards, KW)
    _check(lg, V, tok, old, ref, adv, w, shards, gpu, KW)


def test_shards_temperature_kl_and_in_place():
    V, widths = 5000, [1000, 1500, 2500]
    N = 300
    kw = dict(eps_lo=0.2, eps_hi=0.28, kl_coef=0.05, kl_type=2, inv_temp=0.7)
    U.log(f"vocab shards {widths} N={N} T^-1=0.7 kl=k2 in place")
    lg = wl.logits_host(3102, N, V)
    tok = wl.sample_tokens_host(lg, V, 3102)
    cur, _ = oracle.logprob_rows(lg, tok, V=V, inv_temp=0.7)
    n_old, n_ref = wl.logp_noise(3102, N)
    old, ref = (cur + n_old).astype(np.float32), (cur + n_ref).astype(np.float32)
    adv = np.random.default_rng(7).normal(0, 1, N).astype(np.float32)
    w = np.ones(N, np.float32)
    shards = _shards(V, widths)
    gpu = _run(lg, V, tok, old, ref, adv, w, shards, kw, inplace=True)
    _check(lg, V, tok, old, ref, adv, w, shards, gpu, kw)


def test_merge_reports_uncovered_tokens_and_bad_ids():
    V, widths = 4000, [1500, 2400]  # the last 100 columns belong to no shard
    N = 64
    U.log("vocab shards: uncovered token, bad id")
    lg = wl.logits_host(3103, N, V)
    tok = wl.sample_tokens_host(lg, V, 3103)
    tok[3] = V - 5      # no shard holds it
    tok[7] = V + 10     # outside the vocabulary
    old = np.full(N, -8.0, np.float32)
    ref = np.full(N, -8.0, np.float32)
    adv = np.ones(N, np.float32)
    w = np.ones(N, np.float32)
    gpu = _run(lg, V, tok, old, ref, adv, w, _shards(V, widths), KW)
    assert gpu["bad"] == 2
    for r in (3, 7):
        assert gpu["logp"][r] == 0 and np.all(gpu["dl"][r] == 0)
        assert gpu["state"][r, 0] == 0 and gpu["state"][r, 1] == np.inf


def test_merge_on_oracle_partials():
    """The merge alone, fed the oracle's partials rounded to fp32."""
    import torch
    from paper_2608_01804_amd import leap as L
    V, widths, N = 3000, [1000, 1000, 1000], 128
    U.log("vocab merge on oracle partials")
    lg = wl.logits_host(3104, N, V)
    tok = wl.sample_tokens_host(lg, V, 3104)
    cur, _ = oracle.logprob_rows(lg, tok, V=V)
    old = (cur - 0.02).astype(np.float32)
    ref = (cur + 0.05).astype(np.float32)
    adv = np.linspace(-1, 1, N).astype(np.float32)
    w = np.full(N, 1.0 / N, np.float32)
    parts = np.stack([np.stack(oracle.vocab_shard_stats(lg[:, a:a + b], a, tok), axis=1)
                      for a, b in _shards(V, widths)]).astype(np.float32)
    dev = U.dev()
    p = L.leap_grpo_params(0.2, 0.2, 0.01, 0, 1.0)
    lp = torch.empty(N, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    state = torch.empty((N, 2), dtype=torch.float32, device=dev)
    ws_bytes = L.leap_vocab_merge_workspace_size(N)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    L.leap_vocab_merge_objective(U.T(parts), len(widths), N, V, U.T(tok.astype(np.int32)), U.T(old),
                                 U.T(ref), U.T(adv), U.T(w), p, lp, None, loss, state, ws, ws_bytes)
    torch.cuda.synchronize()
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V)
    assert np.max(np.abs(lp.cpu().numpy() - o["logp"])) < 2e-4
    assert abs(loss.item() - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-7


@pytest.mark.parametrize("widths,inv_temp", [([18992] * 8, 1.0), ([1000, 7, 40000, 12289], 0.9)])
def test_shards_entropy(widths, inv_temp):
    """The merged entropy against the oracle's on the whole rows; asking for
    it changes no other output."""
    V = sum(widths)
    N = 48
    kw = dict(KW, inv_temp=inv_temp)
    U.log(f"vocab shards entropy {widths[:2]}.. x{len(widths)} V={V} T^-1={inv_temp}")
    lg = wl.logits_host(3103, N, V)
    tok = wl.sample_tokens_host(lg, V, 3103)
    lg[1, ::3] = 0xFF80  # -inf columns
    lg[2, :1007] = 0xFF80  # the first two shards all -inf in the second case
    tok[1], tok[2] = 1, V - 1
    cur, _ = oracle.logprob_rows(lg, tok, V=V, inv_temp=inv_temp)
    n_old, n_ref = wl.logp_noise(3103, N)
    old, ref = (cur + n_old).astype(np.float32), (cur + n_ref).astype(np.float32)
    rng = np.random.default_rng(3103)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = np.ones(N, np.float32)
    w[[5, 17]] = 0.0
    shards = _shards(V, widths)
    a = _run(lg, V, tok, old, ref, adv, w, shards, kw, want_entropy=True)
    b = _run(lg, V, tok, old, ref, adv, w, shards, kw)
    assert a["bad"] == b["bad"] == 0
    assert np.array_equal(a["parts"], b["parts"], equal_nan=True)
    assert np.array_equal(a["logp"], b["logp"]) and a["loss"] == b["loss"]
    assert np.array_equal(a["dl"], b["dl"])
    h, bad = oracle.entropy_rows(lg, V=V, inv_temp=inv_temp)
    assert bad == 0
    valid = w != 0
    assert np.all(a["entropy"][~valid] == 0)
    np.testing.assert_allclose(a["entropy"][valid], h[valid], rtol=1e-4, atol=2e-4)


# Shard widths at both ends of every entry of the stats kernel's shape table
# (chunks of 8 columns: one past the previous entry's cover, and the entry's
# own cover, the latter with a partial last chunk), plus the streaming form.
_STATS_COVERS = [64, 128, 256, 512, 1024, 2048, 2560, 3072, 4096, 5120, 6144, 8192, 9728, 12288,
                 16384, 19456, 20480, 24576]
_STATS_WIDTHS = sorted({w for lo, hi in zip([0] + _STATS_COVERS[:-1], _STATS_COVERS)
                        for w in (8 * lo + 1, 8 * hi - 3)} | {8 * 24576 + 8})


@pytest.mark.parametrize("width", _STATS_WIDTHS)
def test_stats_every_shape(width):
    """Each shape of the shard stats kernel against ``oracle.vocab_shard_stats``,
    and its entropy partial t against the whole-row entropy, which for a
    single shard is ln 2 (log2 s - t / s)."""
    import torch
    from paper_2608_01804_amd import leap as L
    N = 24
    U.log(f"shard stats width {width}")
    lg = wl.logits_host(3105 + width % 1000, N, width)
    tok = wl.sample_tokens_host(lg, width, 3105)
    lg[1, ::5] = 0xFF80  # -inf columns
    lg[2, :] = 0xFF80  # an all -inf row
    tok[3] = width - 1  # the last column, inside the partial chunk when there is one
    w = np.ones(N, np.float32)
    w[4] = 0.0
    ld = (width + 7) // 8 * 8
    buf = np.zeros((N, ld), np.uint16)
    buf[:, :width] = lg
    t = torch.from_numpy(buf.view(np.int16)).to(U.dev()).view(torch.bfloat16)
    tok_d, w_d = U.T(tok.astype(np.int32)), U.T(w)
    inv_temp = 0.8
    parts = torch.full((N, 4), float("nan"), dtype=torch.float32, device=U.dev())
    parts_t = torch.full((N,), float("nan"), dtype=torch.float32, device=U.dev())
    L.leap_vocab_shard_stats(t, ld, N, width, 0, tok_d, w_d, inv_temp, parts, partial_t=parts_t)
    q, qt = parts.cpu().numpy(), parts_t.cpu().numpy()
    m2, s, zy, owned = oracle.vocab_shard_stats(lg, 0, tok, w=w, inv_temp=inv_temp)
    np.testing.assert_array_equal(q[:, 3], owned)
    np.testing.assert_array_equal(q[:, 2], np.where(owned == 1, zy, 0))
    live = np.isfinite(m2)
    assert not live[2] and not live[4]
    assert np.all(q[~live, 0] == -np.inf) and np.all(q[~live, 1] == 0) and np.all(qt[~live] == 0)
    np.testing.assert_allclose(q[live, 0], m2[live], rtol=1e-6, atol=1e-6)
    np.testing.assert_allclose(q[live, 1], s[live], rtol=2e-5)
    h, bad = oracle.entropy_rows(lg[live], V=width, inv_temp=inv_temp)
    assert bad == 0
    got_h = np.log(2.0) * (np.log2(q[live, 1].astype(np.float64)) - qt[live] / q[live, 1])
    np.testing.assert_allclose(got_h, h, rtol=1e-4, atol=2e-4)


@pytest.mark.parametrize("widths", [[1, 1], [3, 4, 300], [18992] * 8])
def test_shards_wide_range_and_peaked_rows(widths):
    """Entry-wise relative check of the sharded dlogits on rows whose
    probabilities span many orders of magnitude (logit std 6 and 12) and on
    rows with one logit 30 above the rest (the token on the spike, so that
    p_y is within e^-30 of 1, or away from it).  The shard backward forms
    every entry in fp32 from the merged log-sum-exp and rounds it once to
    bf16 (2^-9), the token's own column as -g p_y + g in fp32: each entry is
    within 2^-8 |d| + 2^-24 |g| of the oracle, the token's column within
    2^-8 |d| + 2^-12 |g| (the fp32 log-sum-exp's error times g)."""
    V = sum(widths)
    N = 64
    seed = 3301 + V
    rng = np.random.default_rng(seed)
    lg = wl.logits_host(seed, N, V)
    x = wl.bf16_bits_to_f32(lg[:, :V]).astype(np.float32)
    x[:16] *= 3.0
    x[48:] *= 6.0
    tok = rng.integers(0, V, N).astype(np.int32)
    spike = rng.integers(0, V, N)
    for k in range(16, 48):
        x[k, spike[k]] += 30.0
        tok[k] = spike[k] if (k < 32 or V == 1) else (spike[k] + 1 + rng.integers(0, V - 1)) % V
    lg[:, :V] = wl.f32_to_bf16_bits(x)
    cur, _ = oracle.logprob_rows(lg, tok, V=V)
    n_old, n_ref = wl.logp_noise(seed, N)
    old, ref = (cur + n_old).astype(np.float32), (cur + n_ref).astype(np.float32)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = np.ones(N, np.float32)
    kw = dict(KW, kl_coef=0.05)
    U.log(f"vocab shards wide-range / peaked rows {widths[:3]} V={V}")
    gpu = _run(lg, V, tok, old, ref, adv, w, _shards(V, widths), kw)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, **kw)
    assert gpu["bad"] == o["bad"] == 0
    got, want = U.bf16_f64(gpu["dl"]), o["dlogits"]
    rho = np.exp(o["logp"] - old.astype(np.float64))
    g_max = w * (np.abs(adv) * rho + kw["kl_coef"] * np.abs(1.0 - np.exp(ref - o["logp"])))
    tol = 2.0 ** -8 * np.abs(want) + 2.0 ** -24 * g_max[:, None]
    tol[np.arange(N), tok] = 2.0 ** -8 * np.abs(want[np.arange(N), tok]) + 2.0 ** -12 * g_max
    ratio = np.abs(got - want) / tol
    k, v = np.unravel_index(np.argmax(ratio), ratio.shape)
    U.log(f"  max |err| / bound {ratio.max():.3f} at row {k}, column {v}")
    assert ratio.max() <= 1.0
