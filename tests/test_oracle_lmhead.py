"""Pins of the fused LM-head oracle (``oracle.lmhead``) against what the
mathematics fixes, independently of its own code path:

* central finite differences of the fp64 loss give dH and dW (catches a
  transposed or swapped operand, a dropped temperature factor, a wrong sign);
* with W = I the logits are H itself, so every output reduces to the per-row
  objective oracle (itself pinned elsewhere) and dH to its dlogits;
* a subset of rows gives the same per-row outputs as the full evaluation;
* bf16 bit-pattern inputs convert exactly.
"""
import numpy as np
import pytest

import oracle

KL = [oracle.KL_K3, oracle.KL_K1, oracle.KL_K2]


def _case(seed=7, N=5, H=6, V=7, inv_temp=0.7):
    rng = np.random.default_rng(seed)
    Hm = rng.normal(0.0, 1.0, (N, H))
    Wm = rng.normal(0.0, 0.5, (V, H))
    y = rng.integers(0, V, N).astype(np.int32)
    cur = oracle.lmhead(Hm, Wm, y, np.zeros(N), np.zeros(N), np.zeros(N), np.ones(N),
                        inv_temp=inv_temp, want_grads=False)["logp"]
    # ratios e^(cur - old): inside the clip window (rows 0, 1), clipped below
    # and above (rows 2, 3), and one excluded row (w = 0)
    old = cur + np.array([0.05, -0.05, 0.5, -0.5, 0.0])[:N]
    ref = cur + np.array([0.1, -0.2, 0.05, 0.3, 0.0])[:N]
    adv = np.array([1.0, -0.7, 0.8, -1.2, 0.4])[:N]
    w = np.array([0.25, 0.5, 1.0, 0.75, 0.0])[:N]
    return Hm, Wm, y, old, ref, adv, w


@pytest.mark.parametrize("kl_type", KL)
def test_gradients_match_central_differences(kl_type):
    inv_temp = 0.7
    Hm, Wm, y, old, ref, adv, w = _case(inv_temp=inv_temp)
    kw = dict(eps_lo=0.2, eps_hi=0.2, kl_coef=0.05, kl_type=kl_type, inv_temp=inv_temp)
    r = oracle.lmhead(Hm, Wm, y, old, ref, adv, w, v_block=4, **kw)  # two vocabulary blocks
    assert r["bad"] == 0

    def loss(Hx, Wx):
        return oracle.lmhead(Hx, Wx, y, old, ref, adv, w, want_grads=False, **kw)["loss"]

    h = 1e-6
    fd_H = np.zeros_like(Hm)
    for idx in np.ndindex(*Hm.shape):
        a, b = Hm.copy(), Hm.copy()
        a[idx] += h
        b[idx] -= h
        fd_H[idx] = (loss(a, Wm) - loss(b, Wm)) / (2 * h)
    fd_W = np.zeros_like(Wm)
    for idx in np.ndindex(*Wm.shape):
        a, b = Wm.copy(), Wm.copy()
        a[idx] += h
        b[idx] -= h
        fd_W[idx] = (loss(Hm, a) - loss(Hm, b)) / (2 * h)
    np.testing.assert_allclose(r["dH"], fd_H, rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(r["dW"], fd_W, rtol=1e-6, atol=1e-8)
    # the excluded row has no gradient
    assert np.all(r["dH"][4] == 0.0)


def test_identity_weight_reduces_to_row_objective():
    rng = np.random.default_rng(3)
    N, H = 6, 8
    Hm = rng.normal(0.0, 2.0, (N, H))
    y = rng.integers(0, H, N).astype(np.int32)
    old = rng.normal(-2.0, 0.3, N)
    ref = rng.normal(-2.0, 0.3, N)
    adv = rng.normal(0.0, 1.0, N)
    w = np.full(N, 1.0 / N)
    kw = dict(kl_coef=0.02, inv_temp=1.3)
    r = oracle.lmhead(Hm, np.eye(H), y, old, ref, adv, w, **kw)
    q = oracle.grpo_rows(Hm, y, old, ref, adv, w, **kw)
    np.testing.assert_array_equal(r["logp"], q["logp"])
    np.testing.assert_array_equal(r["tok_loss"], q["tok_loss"])
    assert r["loss"] == q["loss"]
    np.testing.assert_array_equal(r["dH"], q["dlogits"])


def test_row_subset_matches_full():
    Hm, Wm, y, old, ref, adv, w = _case(seed=11, N=5, H=6, V=9)
    full = oracle.lmhead(Hm, Wm, y, old, ref, adv, w)
    rows = np.array([3, 0, 2])
    sub = oracle.lmhead(Hm, Wm, y, old, ref, adv, w, rows=rows)
    np.testing.assert_allclose(sub["logp"], full["logp"][rows], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(sub["tok_loss"], full["tok_loss"][rows], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(sub["dH"], full["dH"][rows], rtol=1e-12, atol=1e-14)
    assert sub["dW"] is None


def test_bad_token_is_excluded_and_counted():
    Hm, Wm, y, old, ref, adv, w = _case(seed=5)
    y = y.copy()
    y[1] = Wm.shape[0]  # out of range with w != 0
    r = oracle.lmhead(Hm, Wm, y, old, ref, adv, w)
    assert r["bad"] == 1
    assert r["logp"][1] == 0.0 and np.all(r["dH"][1] == 0.0)


def test_bf16_patterns_convert_exactly():
    rng = np.random.default_rng(2)
    N, H, V = 4, 8, 5
    Hf = rng.normal(0, 1, (N, H)).astype(np.float32)
    Wf = rng.normal(0, 1, (V, H)).astype(np.float32)
    # truncate to bf16-representable values, then compare the two input forms
    Hb = (Hf.view(np.uint32) >> 16).astype(np.uint16)
    Wb = (Wf.view(np.uint32) >> 16).astype(np.uint16)
    H64 = (Hb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    W64 = (Wb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    y = np.array([0, 4, 2, 1], np.int32)
    z = np.zeros(N)
    a = oracle.lmhead(Hb, Wb, y, z, z, np.ones(N), np.ones(N))
    b = oracle.lmhead(H64, W64, y, z, z, np.ones(N), np.ones(N))
    np.testing.assert_array_equal(a["logp"], b["logp"])
    np.testing.assert_array_equal(a["dW"], b["dW"])
