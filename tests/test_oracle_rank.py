"""Pins of the oracle's rank-based reward and advantage (Sec. 3.2, Eqs. 4-11).

Each check comes from outside the oracle's own code: hand-worked fixtures,
the paper's closed forms for the three-tier case, the +/-1 extremes and the
regime signs it states, an identity with average ranks computed by
scipy.stats.rankdata, and the reduction of the single-turn case to the
z-score of binary rewards (scipy.stats.zscore).
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rank_worked_examples.txt")
EPS = float(np.float32(1e-6))


def _read_examples():
    blocks, cur = [], None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, *rest = line.split()
        if head == "example":
            cur = {"name": rest[0]}
            blocks.append(cur)
        elif head == "G":
            cur["G"], cur["M"], cur["key"] = int(rest[0]), int(rest[2]), rest[4]
        elif head == "A":
            cur["A"] = [float(v) for v in rest]
        else:
            cur[head] = [int(v) for v in rest]
    return blocks


@pytest.mark.parametrize("ex", _read_examples(), ids=lambda e: e["name"])
def test_hand_worked_examples(ex):
    key = oracle.KEY_LEX if ex["key"] == "lex" else oracle.KEY_TURN
    out = oracle.rank_tournament(ex["pass_turn"], ex["G"], ex["M"], key_mode=key, eps=EPS,
                                 speedup_q=ex.get("speedup_q"), n_tokens=ex.get("n_tokens"))
    assert out["n_worse"].tolist() == ex["n_worse"]
    assert out["n_better"].tolist() == ex["n_better"]
    G = ex["G"]
    assert np.array_equal(out["R"], np.array(ex["R_num"], dtype=np.float64) / (G - 1))
    if "A" in ex:
        np.testing.assert_allclose(out["A"], ex["A"], rtol=3e-6, atol=1e-9)


@pytest.mark.parametrize("G", [2, 3, 4, 5, 8, 11, 16])
def test_three_tier_closed_forms(G):
    """Eqs. 7-9 for every split N1 + N2 + N3 = G with M = 2."""
    for N1 in range(G + 1):
        for N2 in range(G + 1 - N1):
            N3 = G - N1 - N2
            pt = [1] * N1 + [2] * N2 + [0] * N3
            out = oracle.rank_tournament(pt, G, 2, eps=EPS)
            d = out["n_worse"] - out["n_better"]
            want = [N2 + N3] * N1 + [N3 - N1] * N2 + [-(N1 + N2)] * N3
            assert d.tolist() == want, (N1, N2, N3)
            # Eq. 8 regime signs (Eqs. 10-11): R(O2) < 0 iff N1 > N3.
            if N2:
                r2 = out["R"][N1]
                assert (r2 < 0) == (N1 > N3) and (r2 > 0) == (N3 > N1)


def test_o2_monotone_in_failures_and_first_passes():
    """dR(O2)/dN3 > 0 and dR(O2)/dN1 < 0 (end of Sec. 3.2): moving one
    rollout from O1 to O3 raises the reward of an O2 rollout by 2/(G-1)."""
    G = 10
    for N1 in range(1, G):
        N2 = 1
        N3 = G - N1 - N2
        if N3 < 0:
            continue
        a = oracle.rank_tournament([1] * N1 + [2] * N2 + [0] * N3, G, 2)["R"][N1]
        b = oracle.rank_tournament([1] * (N1 - 1) + [2] * N2 + [0] * (N3 + 1), G, 2)["R"][N1 - 1]
        assert b - a == pytest.approx(2.0 / (G - 1), abs=1e-15)


@pytest.mark.parametrize("G", [2, 7, 64, 1024])
def test_outright_winner_and_loser(G):
    """An absolute winner gets exactly +1, an absolute loser exactly -1 (Eq. 6)."""
    pt = [1] + [2] * (G - 2) + [0] if G > 2 else [1, 0]
    out = oracle.rank_tournament(pt, G, 2)
    assert out["R"][0] == 1.0 and out["R"][-1] == -1.0
    assert np.all(np.abs(out["R"]) <= 1.0)


def test_average_rank_identity():
    """R_i = (2 * avgrank_i - G - 1) / (G - 1) with average ranks of the keys
    (scipy.stats.rankdata, method='average'), for random groups with ties."""
    rng = np.random.default_rng(123)
    for _ in range(300):
        G = int(rng.integers(2, 40))
        M = int(rng.integers(1, 5))
        pt = rng.integers(0, M + 1, size=G)
        out = oracle.rank_tournament(pt, G, M)
        tier = np.where(pt == 0, 0, M - pt + 1)
        ar = stats.rankdata(tier, method="average")
        want = (2 * ar - G - 1) / (G - 1)
        np.testing.assert_allclose(out["R"], want, rtol=0, atol=1e-14)


def test_average_rank_identity_lex():
    rng = np.random.default_rng(5)
    for _ in range(200):
        G = int(rng.integers(2, 30))
        pt = rng.integers(0, 3, size=G)
        sq = np.where(pt > 0, rng.integers(0, 4, size=G), 0)
        nt = rng.integers(1, 4, size=G)
        out = oracle.rank_tournament(pt, G, 2, key_mode=oracle.KEY_LEX, speedup_q=sq, n_tokens=nt)
        tier = np.where(pt == 0, 0, 3 - pt)
        # lexicographic key mapped to one integer: tier, then speedup, then fewer tokens
        code = tier * 10_000 + sq * 100 + (99 - nt)
        ar = stats.rankdata(code, method="average")
        np.testing.assert_allclose(out["R"], (2 * ar - G - 1) / (G - 1), rtol=0, atol=1e-14)


def test_sum_zero_and_permutation_invariance():
    rng = np.random.default_rng(9)
    G, M = 16, 3
    pt = rng.integers(0, M + 1, size=(50, G))
    out = oracle.rank_tournament(pt, G, M)
    d = (out["n_worse"] - out["n_better"]).reshape(50, G)
    assert np.all(d.sum(axis=1) == 0)
    for g in range(50):
        perm = rng.permutation(G)
        o2 = oracle.rank_tournament(pt[g][perm], G, M)
        assert np.array_equal(o2["n_worse"], out["n_worse"].reshape(50, G)[g][perm])
        np.testing.assert_array_equal(o2["R"], out["R"].reshape(50, G)[g][perm])


def test_equal_outcomes_give_zero_advantage():
    for G in (2, 8, 64):
        for m in (0, 1, 2):
            out = oracle.rank_tournament([m] * G, G, 2)
            assert np.all(out["R"] == 0) and np.all(out["A"] == 0)


def test_single_turn_reduces_to_binary_grpo():
    """With one turn, R_i = G/(G-1) (b_i - mean b) for binary pass b, so the
    group-normalised advantage is the z-score of b with the unbiased std."""
    rng = np.random.default_rng(3)
    for _ in range(100):
        G = int(rng.integers(2, 65))
        b = rng.integers(0, 2, size=G)
        if b.min() == b.max():
            continue
        out = oracle.rank_tournament(b, G, 1, eps=0.0)
        z = stats.zscore(b.astype(np.float64), ddof=1)
        np.testing.assert_allclose(out["A"], z, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(out["R"], G / (G - 1) * (b - b.mean()), atol=1e-14)


def test_brute_force_tiny_groups():
    """Every outcome assignment for G <= 5, M = 2, against counts taken from
    pairwise comparisons of Python Fractions of the tier order."""
    for G in range(2, 6):
        for pt in itertools.product(range(3), repeat=G):
            out = oracle.rank_tournament(list(pt), G, 2)
            tiers = [Fraction(0) if m == 0 else Fraction(3 - m) for m in pt]
            for i in range(G):
                w = sum(1 for j in range(G) if j != i and tiers[i] > tiers[j])
                b = sum(1 for j in range(G) if j != i and tiers[i] < tiers[j])
                assert out["n_worse"][i] == w and out["n_better"][i] == b
                assert out["R"][i] == float(Fraction(w - b, G - 1))


def test_invalid_pass_turn_counts_and_ranks_as_failure():
    out = oracle.rank_tournament([1, 5, -1, 0], 4, 2)
    assert out["bad"] == 2
    assert out["r"].tolist() == [2, 0, 0, 0]


def test_adv_none_returns_reward():
    out = oracle.rank_tournament([1, 2, 0, 0], 4, 2, adv_norm=oracle.ADV_NONE)
    assert np.array_equal(out["A"], out["R"])
