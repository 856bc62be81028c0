"""Pins of the oracle's per-token objective and logits gradient (Sec. 3.1,
Eq. 3 per token; surrogate read as PPO-clip, KL as k3 / k1 / k2).

Independent references: the closed form log p = -ln V for uniform logits,
torch.log_softmax in fp64, the gradient of torch's cross-entropy (the
ratio-one, KL-free special case), the exact KL divergence of two categorical
distributions (scipy.stats.entropy) as the expectation of the k3 and k1
estimators, and central finite differences of the oracle's own loss.
"""
import os

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))


def _rand_rows(rng, N, V, scale=2.0):
    return rng.normal(0.0, scale, (N, V))


def _logp_torch(x, y):
    t = torch.log_softmax(torch.from_numpy(x), dim=-1)
    return t[torch.arange(x.shape[0]), torch.from_numpy(np.asarray(y, np.int64))].numpy()


def test_uniform_logits_give_minus_log_v():
    for V in (16, 32768, 151936):
        lg = np.zeros((3, V), np.uint16)
        out = oracle.grpo_rows(lg, [0, V // 2, V - 1], [0, 0, 0], [0, 0, 0], [0, 0, 0], [1, 1, 1],
                               want_dlogits=False)
        np.testing.assert_allclose(out["logp"], -np.log(V), rtol=0, atol=1e-12)
    assert -np.log(151936) == pytest.approx(-11.931214658529285, abs=1e-12)


def test_logp_matches_torch_log_softmax():
    rng = np.random.default_rng(0)
    x = _rand_rows(rng, 40, 1000)
    y = rng.integers(0, 1000, 40)
    out = oracle.grpo_rows(x, y, np.zeros(40), np.zeros(40), np.zeros(40), np.ones(40),
                           want_dlogits=False)
    np.testing.assert_allclose(out["logp"], _logp_torch(x, y), rtol=0, atol=1e-12)
    # the forward-only entry point on bf16 inputs
    lg = wl.f32_to_bf16_bits(x.astype(np.float32))
    lp, bad = oracle.logprob_rows(lg, y)
    xb = wl.bf16_bits_to_f32(lg).astype(np.float64)
    assert bad == 0
    np.testing.assert_allclose(lp, _logp_torch(xb, y), rtol=0, atol=1e-12)
    for inv_temp in (0.5, 1.7):  # softmax of the scaled logits
        lp_t, bad = oracle.logprob_rows(lg, y, inv_temp=inv_temp)
        assert bad == 0
        np.testing.assert_allclose(lp_t, _logp_torch(inv_temp * xb, y), rtol=0, atol=1e-12)


def test_large_logits_are_shift_invariant():
    rng = np.random.default_rng(1)
    x = _rand_rows(rng, 8, 300)
    y = rng.integers(0, 300, 8)
    args = (y, rng.normal(-5, 0.1, 8), rng.normal(-5, 0.1, 8), rng.normal(0, 1, 8), np.ones(8))
    a = oracle.grpo_rows(x, *args)
    b = oracle.grpo_rows(x + 800.0, *args)  # exp(800) overflows double without the max shift
    np.testing.assert_allclose(b["logp"], a["logp"], atol=1e-10)
    np.testing.assert_allclose(b["dlogits"], a["dlogits"], atol=1e-12)


def test_ratio_one_no_kl_is_weighted_cross_entropy_gradient():
    """old = logp (ratio 1) and beta = 0: loss = -sum_k w_k A_k and the
    gradient is w_k A_k times the cross-entropy gradient softmax - onehot."""
    rng = np.random.default_rng(2)
    N, V = 24, 257
    x = _rand_rows(rng, N, V)
    y = rng.integers(0, V, N)
    A = rng.normal(0, 1, N)
    w = rng.uniform(0.1, 2.0, N)
    old = _logp_torch(x, y)
    out = oracle.grpo_rows(x, y, old, np.zeros(N), A, w, kl_coef=0.0)
    assert out["loss"] == pytest.approx(-(w * A).sum(), rel=1e-12)
    xt = torch.from_numpy(x).requires_grad_(True)
    ce = torch.nn.functional.cross_entropy(xt, torch.from_numpy(y), reduction="none")
    (ce * torch.from_numpy(w * A)).sum().backward()
    np.testing.assert_allclose(out["dlogits"], xt.grad.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("kl_type", [oracle.KL_K3, oracle.KL_K1])
def test_kl_estimator_expectation_is_exact_kl(kl_type):
    """Sum over every token y of pi_theta(y) * KL_est(y) = KL(pi_theta || pi_ref)
    for the k3 and k1 estimators: one row per token id, weight pi_theta(y),
    zero advantage, beta = 1."""
    rng = np.random.default_rng(3)
    V = 50
    z = rng.normal(0, 1.5, V)
    zr = rng.normal(0, 1.5, V)
    p = np.exp(z - np.logaddexp.reduce(z))
    q = np.exp(zr - np.logaddexp.reduce(zr))
    x = np.tile(z, (V, 1))
    y = np.arange(V)
    out = oracle.grpo_rows(x, y, np.log(p), np.log(q), np.zeros(V), p, kl_coef=1.0,
                           kl_type=kl_type, want_dlogits=False)
    assert out["loss"] == pytest.approx(stats.entropy(p, q), rel=1e-10)


def test_k2_is_half_squared_log_ratio_mean():
    rng = np.random.default_rng(4)
    V = 40
    z = rng.normal(0, 1.0, V)
    p = np.exp(z - np.logaddexp.reduce(z))
    ref = np.log(p) + rng.normal(0, 0.3, V)
    out = oracle.grpo_rows(np.tile(z, (V, 1)), np.arange(V), np.log(p), ref, np.zeros(V), p,
                           kl_coef=1.0, kl_type=oracle.KL_K2, want_dlogits=False)
    # k2 = (log p - log q)^2 / 2 in expectation under p
    assert out["loss"] == pytest.approx(float(np.sum(p * 0.5 * (np.log(p) - ref) ** 2)), rel=1e-10)


# Ratio placements: well inside the clip window, above and below it, and --
# for the asymmetric bounds (0.2, 0.28) -- inside the windows 1.2 < rho < 1.28
# and 0.72 < rho < 0.8 that only the correct assignment of the two bounds
# treats as it should (unclipped above 1.2, clipped below 0.8).
RHO = {"inside": 1.05, "above": 1.6, "below": 0.5, "hi_window": 1.25, "lo_window": 0.76}


def _fd_case(seed, kl_type, inv_temp, branch):
    rng = np.random.default_rng(seed)
    N, V = 4, 12
    x = _rand_rows(rng, N, V, 1.5)
    y = rng.integers(0, V, N)
    lp = _logp_torch(x * inv_temp, y)
    # place rho = exp(lp - old) at the branch's value (within 1 %)
    old = lp - np.log(RHO[branch]) + rng.normal(0, 0.003, N)
    ref = lp + rng.normal(0, 0.3, N)
    A = np.array([-1.3, 0.8, -0.6, 1.1])
    w = rng.uniform(0.5, 2.0, N)
    return x, y, old, ref, A, w


FD_CASES = [(b, (0.2, 0.2)) for b in ("inside", "above", "below")] + \
           [(b, (0.2, 0.28)) for b in ("inside", "above", "below", "hi_window", "lo_window")]


@pytest.mark.parametrize("kl_type", [oracle.KL_K3, oracle.KL_K1, oracle.KL_K2])
@pytest.mark.parametrize("inv_temp", [1.0, 0.7])
@pytest.mark.parametrize("branch,eps", FD_CASES, ids=[f"{b}-{e[0]}-{e[1]}" for b, e in FD_CASES])
def test_gradient_matches_central_differences(kl_type, inv_temp, branch, eps):
    x, y, old, ref, A, w = _fd_case(11, kl_type, inv_temp, branch)
    kw = dict(eps_lo=eps[0], eps_hi=eps[1], kl_coef=0.05, kl_type=kl_type, inv_temp=inv_temp)
    out = oracle.grpo_rows(x, y, old, ref, A, w, **kw)
    h = 1e-6
    fd = np.zeros_like(x)
    for k in range(x.shape[0]):
        for v in range(x.shape[1]):
            xp = x.copy()
            xm = x.copy()
            xp[k, v] += h
            xm[k, v] -= h
            lp = oracle.grpo_rows(xp, y, old, ref, A, w, want_dlogits=False, **kw)["loss"]
            lm = oracle.grpo_rows(xm, y, old, ref, A, w, want_dlogits=False, **kw)["loss"]
            fd[k, v] = (lp - lm) / (2 * h)
    np.testing.assert_allclose(out["dlogits"], fd, rtol=0, atol=2e-8)


def test_clipped_ratio_passes_no_surrogate_gradient():
    """A > 0 with rho above 1 + eps (or A < 0 below 1 - eps): the surrogate is
    the constant clipped value, so with beta = 0 the gradient vanishes."""
    rng = np.random.default_rng(6)
    x = _rand_rows(rng, 2, 64)
    y = np.array([3, 9])
    lp = _logp_torch(x, y)
    old = lp - np.log(np.array([1.5, 0.6]))  # rho = 1.5 and 0.6
    A = np.array([2.0, -2.0])
    out = oracle.grpo_rows(x, y, old, np.zeros(2), A, np.ones(2), kl_coef=0.0)
    assert np.all(out["dlogits"] == 0.0)
    np.testing.assert_allclose(out["tok_loss"], [-(1.2 * 2.0), -(0.8 * -2.0)], rtol=1e-12)


def _clip_higher_rows():
    rows = []
    for line in open(os.path.join(HERE, "golden", "clip_higher_examples.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            rows.append(tuple(float(v) for v in line.split()))
    return rows


@pytest.mark.parametrize("row", _clip_higher_rows())
def test_clip_higher_golden(row):
    """Hand-worked loss and gradient of the surrogate with eps_lo != eps_hi
    (tests/golden/clip_higher_examples.txt): one row of 4 equal logits."""
    eps_lo, eps_hi, beta, A, rho, q, loss, dl, d_tok, d_other = row
    V = 4
    lp = -np.log(4.0)
    out = oracle.grpo_rows(np.zeros((1, V)), [0], [lp - np.log(rho)], [lp + np.log(q)], [A], [1.0],
                           eps_lo=eps_lo, eps_hi=eps_hi, kl_coef=beta, kl_type=oracle.KL_K3)
    assert out["logp"][0] == pytest.approx(lp, abs=1e-15)
    assert out["tok_loss"][0] == pytest.approx(loss, rel=1e-12, abs=1e-13)
    assert out["loss"] == pytest.approx(loss, rel=1e-12, abs=1e-13)
    d = out["dlogits"][0]
    assert d[0] == pytest.approx(d_tok, rel=1e-12, abs=1e-14)
    np.testing.assert_allclose(d[1:], d_other, rtol=1e-12, atol=1e-14)
    # the gradient with respect to logp is the token column over (1 - 1/4)
    assert d[0] / 0.75 == pytest.approx(dl, rel=1e-12, abs=1e-14)


def test_clip_bounds_are_not_interchangeable():
    """The two bounds act on opposite sides: with (eps_lo, eps_hi) = (0.2,
    0.28) a ratio of 1.25 with A > 0 is unclipped and 0.78 with A < 0 is
    clipped; swapping the two bounds reverses both decisions."""
    lp = -np.log(4.0)
    args = lambda rho, A: (np.zeros((1, 4)), [0], [lp - np.log(rho)], [lp], [A], [1.0])  # noqa: E731
    a = oracle.grpo_rows(*args(1.25, 1.5), eps_lo=0.2, eps_hi=0.28, kl_coef=0.0)
    b = oracle.grpo_rows(*args(1.25, 1.5), eps_lo=0.28, eps_hi=0.2, kl_coef=0.0)
    assert a["tok_loss"][0] == pytest.approx(-1.875, rel=1e-13)
    assert b["tok_loss"][0] == pytest.approx(-1.8, rel=1e-13)
    assert np.any(a["dlogits"] != 0) and np.all(b["dlogits"] == 0)
    c = oracle.grpo_rows(*args(0.78, -1.5), eps_lo=0.2, eps_hi=0.28, kl_coef=0.0)
    d = oracle.grpo_rows(*args(0.78, -1.5), eps_lo=0.28, eps_hi=0.2, kl_coef=0.0)
    assert c["tok_loss"][0] == pytest.approx(1.2, rel=1e-13)
    assert d["tok_loss"][0] == pytest.approx(1.17, rel=1e-13)
    assert np.all(c["dlogits"] == 0) and np.any(d["dlogits"] != 0)


def test_bf16_entry_equals_f64_entry_on_representable_values():
    rng = np.random.default_rng(7)
    N, V = 16, 333
    lg = wl.f32_to_bf16_bits(rng.normal(0, 2, (N, V)).astype(np.float32))
    xf = wl.bf16_bits_to_f32(lg).astype(np.float64)
    y = rng.integers(0, V, N)
    args = (y, rng.normal(-6, 0.2, N), rng.normal(-6, 0.2, N), rng.normal(0, 1, N),
            rng.uniform(0, 1, N))
    a = oracle.grpo_rows(lg, *args, inv_temp=0.5)
    b = oracle.grpo_rows(xf, *args, inv_temp=0.5)
    np.testing.assert_array_equal(a["logp"], b["logp"])
    np.testing.assert_array_equal(a["dlogits"], b["dlogits"])
    assert a["loss"] == b["loss"]


def test_masked_and_invalid_rows():
    rng = np.random.default_rng(8)
    V = 20
    x = _rand_rows(rng, 4, V)
    x[3, :] = -np.inf
    y = np.array([1, V, 2, 0])  # row 1: id out of range; row 3: all -inf
    w = np.array([0.0, 1.0, 1.0, 1.0])
    out = oracle.grpo_rows(x, y, np.zeros(4), np.zeros(4), np.ones(4), w)
    assert out["bad"] == 2
    for k in (0, 1, 3):
        assert np.all(out["dlogits"][k] == 0) and out["logp"][k] == 0 and out["tok_loss"][k] == 0
    assert np.any(out["dlogits"][2] != 0)


def test_minus_inf_columns_get_zero_probability():
    rng = np.random.default_rng(9)
    V = 30
    x = _rand_rows(rng, 1, V)
    x[0, ::3] = -np.inf
    y = np.array([1])
    out = oracle.grpo_rows(x, y, [-3.0], [-3.0], [1.0], [1.0])
    finite = np.isfinite(x[0])
    np.testing.assert_allclose(out["logp"][0], _logp_torch(np.where(finite, x, -1e300), y)[0],
                               atol=1e-12)
    assert np.all(out["dlogits"][0][~finite] == 0)


# ----------------------------------------------------------------------------
# Per-token entropy of softmax(inv_temp * logits), the optional output of the
# fused call: H = -sum_v p_v log p_v in nats.
# ----------------------------------------------------------------------------
NEG_INF = 0xFF80


def test_entropy_closed_forms():
    # uniform logits: ln V; a point mass: 0; two finite columns: the binary
    # entropy of p = 1 / (1 + e^b)
    V = 4096
    def bits(v):  # one bf16 bit pattern
        return int(wl.f32_to_bf16_bits(np.float32(v))[0])

    lg = np.full((4, V), NEG_INF, np.uint16)
    lg[0, :] = bits(1.5)
    lg[1, 17] = bits(-3.0)
    b = 1.25  # exact in bf16
    lg[2, 3] = bits(0.0)
    lg[2, 4000] = bits(b)
    lg[3, :] = bits(0.0)
    lg[3, 0] = NEG_INF  # V - 1 equal columns
    h, bad = oracle.entropy_rows(lg)
    assert bad == 0
    p = 1.0 / (1.0 + np.exp(b))
    want = [np.log(V), 0.0, -p * np.log(p) - (1 - p) * np.log1p(-p), np.log(V - 1)]
    np.testing.assert_allclose(h, want, rtol=1e-12, atol=1e-15)


def test_entropy_matches_scipy_and_temperature():
    rng = np.random.default_rng(11)
    N, V = 6, 1000
    lg = wl.f32_to_bf16_bits(rng.normal(0, 2.0, (N, V)).astype(np.float32))
    x = wl.bf16_bits_to_f32(lg).astype(np.float64)
    for inv_temp in (1.0, 0.5, 1.7):
        h, bad = oracle.entropy_rows(lg, inv_temp=inv_temp)
        assert bad == 0
        z = inv_temp * x
        p = np.exp(z - z.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        np.testing.assert_allclose(h, stats.entropy(p, axis=1), rtol=1e-12)
        assert np.all(h >= 0) and np.all(h <= np.log(V))


def test_entropy_shift_invariant_and_uses_first_v_columns():
    rng = np.random.default_rng(12)
    N, V, ld = 4, 300, 304
    ints = rng.integers(-20, 20, (N, ld)).astype(np.float32)  # exact in bf16, also + 7
    a = wl.f32_to_bf16_bits(ints)
    b = wl.f32_to_bf16_bits(ints + 7.0)
    b[:, V:] = wl.f32_to_bf16_bits(np.float32(100.0))  # padding past V is ignored
    ha, _ = oracle.entropy_rows(a, V=V)
    hb, _ = oracle.entropy_rows(b, V=V)
    np.testing.assert_allclose(ha, hb, rtol=1e-13)


def test_entropy_all_minus_inf_row_is_counted():
    lg = np.full((2, 64), NEG_INF, np.uint16)
    lg[1, :] = 0
    h, bad = oracle.entropy_rows(lg)
    assert bad == 1 and np.isnan(h[0]) and abs(h[1] - np.log(64)) < 1e-13
