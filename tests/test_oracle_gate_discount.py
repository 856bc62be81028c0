"""Pins of the oracle's pruning gate (Sec. 3.1, Eqs. 1-2) and discounted
per-turn token advantage (Sec. 3.3) with its aggregation weights.

Gate: hand-worked pass-rate windows (golden), the easy / hopeless / learning
zone classification the paper states, and the activated-group fraction
against the binomial law (scipy.stats.binom).  Discount: hand-worked values
(golden), the properties the paper states (last turn keeps A, negative A is
uniform, gamma = 1 is uniform, ratio gamma between consecutive turns) and the
sum of the aggregation weights.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle

HERE = os.path.dirname(__file__)


def _gate_rows():
    rows = []
    for line in open(os.path.join(HERE, "golden", "gate_presets.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            name, *v = line.split()
            rows.append((name, *map(int, v)))
    return rows


@pytest.mark.parametrize("row", _gate_rows(), ids=lambda r: f"{r[0]}_G{r[1]}")
def test_gate_presets_oracle_conversion(row):
    name, G, ln, ld, ls, hn, hd, hs, tmin, tmax = row
    got = oracle.tau_from_pass_rate(G, Fraction(ln, ld), bool(ls), Fraction(hn, hd), bool(hs))
    assert got == (tmin, tmax)


@pytest.mark.parametrize("G", [1, 2, 8, 16, 64, 1000])
def test_gate_zones(G):
    """Groups with N_fail below tau_min (easy) and above tau_max (hopeless)
    skip multi-turn; those inside the window enter it (Sec. 3.1)."""
    tmin, tmax = max(0, G // 4), max(0, G - 1)
    # one group per possible failure count: the first N_fail rollouts fail
    ftp = np.ones((G + 1, G), np.uint8)
    for nf in range(G + 1):
        ftp[nf, :nf] = 0
    nf_out, gate = oracle.dcp_gate(ftp, G, tmin, tmax)
    assert nf_out.tolist() == list(range(G + 1))
    for nf in range(G + 1):
        if nf < tmin:
            assert gate[nf] == 0, "easy group entered multi-turn"
        elif nf > tmax:
            assert gate[nf] == 0, "hopeless group entered multi-turn"
        else:
            assert gate[nf] == 1


def test_gate_counts_failures_not_passes():
    G = 8
    ftp = np.array([[1, 1, 1, 1, 1, 1, 1, 0], [0, 0, 0, 0, 0, 0, 0, 1]], np.uint8)
    nf, gate = oracle.dcp_gate(ftp, G, 3, 7)
    assert nf.tolist() == [1, 7]
    assert gate.tolist() == [0, 1]
    # any nonzero byte is a pass
    nf2, _ = oracle.dcp_gate(np.array([[2, 255, 0, 1]], np.uint8), 4, 0, 4)
    assert nf2.tolist() == [1]


def test_gate_activation_fraction_matches_binomial():
    """With i.i.d. first-turn passes of probability p, N_fail ~ Binomial(G,
    1 - p): the gated fraction must match the binomial mass of the window."""
    rng = np.random.default_rng(17)
    G, p, n_groups = 16, 0.55, 200_000
    tmin, tmax = 5, 15
    ftp = (rng.random((n_groups, G)) < p).astype(np.uint8)
    _, gate = oracle.dcp_gate(ftp, G, tmin, tmax)
    want = stats.binom.cdf(tmax, G, 1 - p) - stats.binom.cdf(tmin - 1, G, 1 - p)
    se = np.sqrt(want * (1 - want) / n_groups)
    assert abs(gate.mean() - want) < 5 * se


def _discount_rows():
    rows = []
    for line in open(os.path.join(HERE, "golden", "discount_examples.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            g, a, T, t, e = line.split()
            rows.append((float(g), float(a), int(T), int(t), float(e)))
    return rows


@pytest.mark.parametrize("row", _discount_rows())
def test_discount_golden(row):
    gamma, A, T, t, expected = row
    adv, w, bad = oracle.token_advantages([A], [0], [t], [T], [5], gamma, oracle.AGG_SUM)
    assert bad == 0 and w[0] == 1.0
    assert adv[0] == pytest.approx(expected, rel=1e-15, abs=0)


def test_discount_properties():
    rng = np.random.default_rng(2)
    n = 400
    A = rng.normal(0, 1.5, n)
    A[::17] = 0.0
    T = rng.integers(1, 5, n).astype(np.int32)
    gamma = 0.87
    tok_r = np.concatenate([np.full(T[i], i) for i in range(n)]).astype(np.int32)
    tok_t = np.concatenate([np.arange(T[i]) for i in range(n)]).astype(np.int32)
    adv, _, bad = oracle.token_advantages(A, tok_r, tok_t, T, np.maximum(T, 1), gamma,
                                          oracle.AGG_SUM)
    assert bad == 0
    for i in range(n):
        a = adv[tok_r == i]
        assert a[-1] == A[i]  # last generated turn keeps A_i
        if A[i] < 0:
            assert np.all(a == A[i])  # negative: uniform penalty
        elif T[i] > 1 and A[i] > 0:
            np.testing.assert_allclose(a[:-1] / a[1:], gamma, rtol=1e-14)
            assert np.all(np.abs(a[:-1]) < np.abs(a[1:]))
    adv1, _, _ = oracle.token_advantages(A, tok_r, tok_t, T, T, 1.0, oracle.AGG_SUM)
    assert np.array_equal(adv1, A[tok_r])  # gamma = 1: broadcast


def test_aggregation_weights_and_exclusion():
    # 3 rollouts: 4, 2 and 6 generated tokens; padding and feedback rows excluded
    tok_r = np.array([0, 0, -1, 0, 0, 1, -1, -1, 1, 2, 2, 2, 2, 2, 2, -1], np.int32)
    tok_t = np.array([0, 0, 0, 1, 1, 0, 0, 0, 0, 0, 0, 0, 1, 1, 1, 0], np.int32)
    n_turns = np.array([2, 1, 2], np.int32)
    n_gen = np.array([4, 2, 6], np.int32)
    A = np.array([1.0, -2.0, 0.5])
    adv, w, bad = oracle.token_advantages(A, tok_r, tok_t, n_turns, n_gen, 0.9,
                                          oracle.AGG_SEQ_MEAN_TOKEN_MEAN, 3.0)
    assert bad == 0
    ex = tok_r < 0
    assert np.all(adv[ex] == 0) and np.all(w[ex] == 0)
    for i in range(3):  # each sequence carries 1/N_seq of the total weight
        assert w[tok_r == i].sum() == pytest.approx(1.0 / 3.0, rel=1e-15)
    assert w.sum() == pytest.approx(1.0, rel=1e-15)
    _, w2, _ = oracle.token_advantages(A, tok_r, tok_t, n_turns, n_gen, 0.9,
                                       oracle.AGG_TOKEN_MEAN, 12.0)
    assert np.all(w2[~ex] == 1.0 / 12.0) and w2.sum() == pytest.approx(1.0, rel=1e-15)


def test_invalid_token_rows_are_counted_and_excluded():
    A = np.array([1.0, 1.0])
    tok_r = np.array([0, 2, -2, 1, 1], np.int32)  # rollout 2 and -2 do not exist
    tok_t = np.array([0, 0, 0, 3, 0], np.int32)  # turn 3 >= T
    adv, w, bad = oracle.token_advantages(A, tok_r, tok_t, [1, 2], [1, 1], 0.9, oracle.AGG_SUM)
    assert bad == 3
    assert adv.tolist() == [1.0, 0.0, 0.0, 0.0, 0.9]
    assert w.tolist() == [1.0, 0.0, 0.0, 0.0, 1.0]
