"""GPU parity on hypothesis-generated inputs: random group sizes, turn
counts, ties and key modes for the tournament (K1) and the gate (K2), and
random masks and turn layouts for the token advantages (K3), each compared
with the oracle on the same inputs (integers and rewards bit-exact,
advantages within 1e-6, token advantages and weights within float32
rounding)."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from tests import _gpu_util as U
from tests.test_oracle_properties import groups, token_layouts

pytestmark = pytest.mark.gpu

SETTINGS = settings(max_examples=60, deadline=None,
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
    np.testing.assert_allclose(adv_g, adv_o, rtol=1.2e-7, atol=0)
    np.testing.assert_allclose(w_g, w_o, rtol=1.2e-7, atol=0)
