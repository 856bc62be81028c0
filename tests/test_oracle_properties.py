"""Property tests of the oracle with hypothesis: random group sizes, turn
counts, ties and key modes for the tournament and the gate, random masks and
turn layouts for the token advantages.

The properties come from the definitions, not from the oracle's code:
every strict pair of the tournament adds +1 to one side and -1 to the other
(so the rewards of a group sum to zero and lie in [-1, 1]); the reward is a
function of the multiset of outcomes (permutation invariance); in the
paper's order it equals (2 avgrank - G - 1) / (G - 1) with average ranks of
the tiers (scipy.stats.rankdata); the gate is membership of the failure
count in the inclusive window (Sec. 3.1, Eq. 2); the token advantage of a
rollout's last turn is its advantage, earlier turns are multiplied by gamma
per turn when A >= 0 and unchanged when A < 0 (Sec. 3.3); excluded rows get
zero advantage and weight.
"""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st
from scipy import stats

import oracle

EPS = float(np.float32(1e-6))
SETTINGS = settings(max_examples=150, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])


@st.composite
def groups(draw, max_g=64):
    G = draw(st.integers(2, max_g))
    M = draw(st.integers(1, 4))
    n_groups = draw(st.integers(1, 4))
    n = n_groups * G
    # few distinct values, so ties are common
    pass_turn = np.array(draw(st.lists(st.integers(0, M), min_size=n, max_size=n)), np.int32)
    sq = np.array(draw(st.lists(st.integers(0, 3), min_size=n, max_size=n)), np.int32)
    nt = np.array(draw(st.lists(st.integers(1, 4), min_size=n, max_size=n)), np.int32)
    lex = draw(st.booleans())
    return G, M, pass_turn, sq, nt, lex


@SETTINGS
@given(groups())
def test_tournament_sums_bounds_and_counts(g):
    G, M, pt, sq, nt, lex = g
    key = oracle.KEY_LEX if lex else oracle.KEY_TURN
    out = oracle.rank_tournament(pt, G, M, key_mode=key, eps=EPS, speedup_q=sq, n_tokens=nt)
    assert out["bad"] == 0
    R = out["R"].reshape(-1, G)
    assert np.all(np.abs(R.sum(axis=1)) < 1e-12)
    assert np.all((R >= -1.0) & (R <= 1.0))
    nw, nb = out["n_worse"].reshape(-1, G), out["n_better"].reshape(-1, G)
    assert np.all(nw + nb <= G - 1)
    assert np.array_equal(nw.sum(axis=1), nb.sum(axis=1))  # each strict pair counted once per side
    np.testing.assert_array_equal(R, (nw - nb) / (G - 1))


@SETTINGS
@given(groups(), st.randoms(use_true_random=False))
def test_tournament_permutation_invariance(g, rnd):
    G, M, pt, sq, nt, lex = g
    key = oracle.KEY_LEX if lex else oracle.KEY_TURN
    a = oracle.rank_tournament(pt, G, M, key_mode=key, eps=EPS, speedup_q=sq, n_tokens=nt)
    perm = np.concatenate([g0 * G + np.array(rnd.sample(range(G), G))
                           for g0 in range(pt.size // G)])
    b = oracle.rank_tournament(pt[perm], G, M, key_mode=key, eps=EPS, speedup_q=sq[perm],
                               n_tokens=nt[perm])
    for k in ("n_worse", "n_better", "R"):
        np.testing.assert_array_equal(b[k], a[k][perm])
    np.testing.assert_allclose(b["A"], a["A"][perm], rtol=1e-12, atol=1e-15)


@SETTINGS
@given(groups())
def test_turn_order_reward_is_average_rank(g):
    G, M, pt, _, _, _ = g
    out = oracle.rank_tournament(pt, G, M, eps=EPS)
    tier = np.where(pt == 0, 0, M - pt + 1).reshape(-1, G)
    ranks = stats.rankdata(tier, method="average", axis=1)
    np.testing.assert_allclose(out["R"].reshape(-1, G), (2 * ranks - G - 1) / (G - 1),
                               rtol=0, atol=1e-12)


@SETTINGS
@given(st.integers(1, 64), st.integers(1, 5), st.data())
def test_gate_is_window_membership(G, n_groups, data):
    ftp = np.array(data.draw(st.lists(st.integers(0, 1), min_size=G * n_groups,
                                      max_size=G * n_groups)), np.uint8)
    tmin = data.draw(st.integers(0, G))
    tmax = data.draw(st.integers(tmin, G))
    nf, gate = oracle.dcp_gate(ftp, G, tmin, tmax)
    want_nf = (ftp.reshape(-1, G) == 0).sum(axis=1)
    np.testing.assert_array_equal(nf, want_nf)
    np.testing.assert_array_equal(gate, ((want_nf >= tmin) & (want_nf <= tmax)).astype(np.uint8))


@st.composite
def token_layouts(draw):
    n_roll = draw(st.integers(1, 12))
    T = np.array(draw(st.lists(st.integers(1, 4), min_size=n_roll, max_size=n_roll)), np.int32)
    A = np.array(draw(st.lists(st.floats(-3, 3, allow_nan=False, width=32), min_size=n_roll,
                               max_size=n_roll)), np.float64)
    rows_r, rows_t = [], []
    for i in range(n_roll):
        for t in range(int(T[i])):
            k = draw(st.integers(1, 5))
            rows_r += [i] * k
            rows_t += [t] * k
    rows_r = np.array(rows_r, np.int32)
    rows_t = np.array(rows_t, np.int32)
    # random excluded rows (padding / feedback) inserted anywhere
    n_ex = draw(st.integers(0, 10))
    pos = np.array(draw(st.lists(st.integers(0, rows_r.size), min_size=n_ex, max_size=n_ex)),
                   np.int64)
    tok_r = np.insert(rows_r, pos, -1)
    tok_t = np.insert(rows_t, pos, 0)
    order = draw(st.permutations(range(tok_r.size)))
    tok_r, tok_t = tok_r[list(order)], tok_t[list(order)]
    gamma = draw(st.sampled_from([1.0, 0.9, 0.5, 0.25]))
    return A, T, tok_r, tok_t, gamma


@SETTINGS
@given(token_layouts())
def test_token_advantage_discount_and_masks(lay):
    A, T, tok_r, tok_t, gamma = lay
    n_gen = np.bincount(tok_r[tok_r >= 0], minlength=A.size).astype(np.int32)
    adv, w, bad = oracle.token_advantages(A, tok_r, tok_t, T, n_gen, gamma,
                                          oracle.AGG_SEQ_MEAN_TOKEN_MEAN, float(A.size))
    assert bad == 0
    ex = tok_r < 0
    assert np.all(adv[ex] == 0) and np.all(w[ex] == 0)
    for k in np.flatnonzero(~ex):
        i, t = tok_r[k], tok_t[k]
        if t == T[i] - 1 or A[i] < 0 or gamma == 1.0:
            assert adv[k] == A[i]
        else:
            np.testing.assert_allclose(adv[k], gamma ** (T[i] - 1 - t) * A[i], rtol=1e-14,
                                       atol=0)
        np.testing.assert_allclose(w[k], 1.0 / (A.size * n_gen[i]), rtol=1e-15)
    # every rollout's weights sum to 1 / N_seq, all weights to 1
    np.testing.assert_allclose(w.sum(), 1.0, rtol=1e-12)
