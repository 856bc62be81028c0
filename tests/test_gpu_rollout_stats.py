"""Parity of leap_rollout_stats with ``oracle.rollout_stats``: every counter
bit-exact (integer counts), on the workloads' simulated rollouts (gate and
advantages from the oracle), on the tournament-stress workload, with bad
items, and without advantages."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads as wl
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu


def _gpu(pt, nt, gate, adv, G, M, nb):
    import torch
    from paper_2608_01804_amd import leap as L
    n_groups = gate.size
    cnt = torch.full((9 + 6 * nb,), -7, dtype=torch.int64, device=U.dev())
    err = U.zeros_i32(1)
    L.leap_rollout_stats(U.T(pt.astype(np.int32)), U.T(nt.astype(np.int32)),
                         U.T(gate.astype(np.uint8)),
                         None if adv is None else U.T(adv.astype(np.float32)), n_groups, G, M, nb,
                         cnt, err)
    torch.cuda.synchronize()
    return cnt.cpu().numpy(), int(err.item())


def _expect(pt, nt, gate, adv, G, M, nb):
    o = oracle.rollout_stats(pt, nt, gate, G, M,
                             advantage=None if adv is None else adv.astype(np.float32).astype(np.float64),
                             n_buckets=nb)
    head = np.array([o[k] for k in oracle.STAT_FIELDS], np.int64)
    return np.concatenate([head, o["composition"].reshape(-1)]), o["bad"]


@pytest.mark.parametrize("name", ["tiny", "mid", "full"])
def test_workload_step(name):
    lat = wl.draw_latent(name)
    U.log(f"rollout stats on the {name} workload: {lat.n_groups} groups x {lat.G}")
    tmin, tmax = oracle.tau_from_pass_rate(lat.G, Fraction(0), True, Fraction(3, 4), True)
    _, gate = oracle.dcp_gate(lat.first_turn_pass, lat.G, tmin, tmax)
    gate = np.asarray(gate, np.uint8)
    ro = wl.realize(lat, gate)
    rk = oracle.rank_tournament(ro.pass_turn, lat.G, lat.M)
    for nb in (1, 10, 16):
        got, bad = _gpu(ro.pass_turn, ro.n_turns, gate, rk["A"], lat.G, lat.M, nb)
        want, wbad = _expect(ro.pass_turn, ro.n_turns, gate, rk["A"], lat.G, lat.M, nb)
        np.testing.assert_array_equal(got, want)
        assert bad == wbad == 0


def test_stress_workload_and_bad_items():
    lat = wl.draw_latent("stress")
    U.log(f"rollout stats on the stress workload with bad items: {lat.n_groups} x {lat.G}")
    rng = np.random.default_rng(4)
    gate = rng.integers(0, 2, lat.n_groups).astype(np.uint8)
    ro = wl.realize(lat, gate)
    pt = np.array(ro.pass_turn, np.int32)
    nt = np.array(ro.n_turns, np.int32)
    adv = rng.normal(0, 1, pt.size)
    adv[rng.random(pt.size) < 0.1] = 0.0
    bad_idx = rng.choice(pt.size, 37, replace=False)
    pt[bad_idx[:20]] = lat.M + 1
    nt[bad_idx[20:]] = 0
    got, bad = _gpu(pt, nt, gate, adv, lat.G, lat.M, 10)
    want, wbad = _expect(pt, nt, gate, adv, lat.G, lat.M, 10)
    np.testing.assert_array_equal(got, want)
    assert bad == wbad == 37


def test_without_advantages_and_large_groups():
    rng = np.random.default_rng(5)
    G, M, n_groups = 1000, 4, 37
    pt = rng.integers(0, M + 1, n_groups * G).astype(np.int32)
    nt = np.where(pt >= 1, pt, M).astype(np.int32)
    gate = rng.integers(0, 2, n_groups).astype(np.uint8)
    got, bad = _gpu(pt, nt, gate, None, G, M, 4)
    want, _ = _expect(pt, nt, gate, None, G, M, 4)
    np.testing.assert_array_equal(got, want)
    assert np.all(got[9:] == 0) and bad == 0


def test_empty_step():
    got, bad = _gpu(np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.uint8), None, 8, 2, 3)
    assert np.all(got == 0) and bad == 0
