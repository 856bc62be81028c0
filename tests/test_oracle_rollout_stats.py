"""Pins of ``oracle.rollout_stats`` (training statistics of the pruning-range
study, turns per pass, and the advantage-sign composition of rollouts): a
hand-worked fixture, identities that hold for any rollouts, and agreement
with the simulated debugging loop of the synthetic workloads."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rollout_stats_examples.txt")


def _fixture():
    gates, pts, nts, advs, want, comp = [], [], [], [], {}, {}
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        if "|" in line:
            head, pt, nt, adv = [p.strip() for p in line.split("|")]
            gates.append(int(head.split()[1]))
            pts += [int(v) for v in pt.split()]
            nts += [int(v) for v in nt.split()]
            advs += [float(v) for v in adv.split()]
        elif line.startswith("comp"):
            _, b, o, s, c = line.split()
            comp[(int(b), int(o), int(s))] = int(c)
        else:
            k, v = line.split()
            want[k] = int(v)
    return (np.array(pts, np.int32), np.array(nts, np.int32), np.array(gates, np.uint8),
            np.array(advs), want, comp)


def test_hand_worked_fixture():
    pt, nt, gate, adv, want, comp = _fixture()
    r = oracle.rollout_stats(pt, nt, gate, G=4, M=3, advantage=adv, n_buckets=4)
    assert r["bad"] == 0
    for k, v in want.items():
        assert r[k] == v, k
    expect = np.zeros((4, 3, 2), np.int64)
    for (b, o, s), c in comp.items():
        expect[b, o, s] = c
    np.testing.assert_array_equal(r["composition"], expect)
    assert Fraction(r["recovered_rollouts"], r["multi_turn_rollouts"]) == Fraction(2, 7)
    assert r["turns_per_pass"] == pytest.approx(29 / 9)
    assert r["activated_fraction"] == 0.75 and r["per_group_recovery"] == 0.5


def _random(seed, n_groups=200, G=8, M=3):
    rng = np.random.default_rng(seed)
    pt = rng.integers(0, M + 1, n_groups * G).astype(np.int32)
    nt = np.where(pt >= 1, pt, M).astype(np.int32)
    gate = rng.integers(0, 2, n_groups).astype(np.uint8)
    adv = rng.normal(0, 1, n_groups * G)
    adv[rng.random(adv.size) < 0.2] = 0.0
    return pt, nt, gate, adv


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_identities(seed):
    G, M, nb = 8, 3, 5
    pt, nt, gate, adv = _random(seed, G=G, M=M)
    r = oracle.rollout_stats(pt, nt, gate, G, M, advantage=adv, n_buckets=nb)
    comp = r["composition"]
    assert comp.sum() == np.count_nonzero(adv)
    assert comp[:, :2].sum() == np.count_nonzero(adv[pt >= 1])
    assert r["passed_rollouts"] == np.count_nonzero(pt >= 1)
    assert r["total_turns"] == nt.sum()
    assert 0 <= r["recovered_rollouts"] <= r["multi_turn_rollouts"]
    assert 0 <= r["recovered_groups"] <= r["debugging_groups"] <= r["activated_groups"]
    # per group, counted directly from the definitions
    pg = pt.reshape(-1, G)
    act = gate.astype(bool)
    multi = (pg != 1) & act[:, None]
    rec = (pg >= 2) & act[:, None]
    assert r["multi_turn_rollouts"] == multi.sum() and r["recovered_rollouts"] == rec.sum()
    assert r["debugging_groups"] == multi.any(axis=1).sum()
    assert r["recovered_groups"] == rec.any(axis=1).sum()
    # bucket of every nonzero-advantage rollout from its group's pass count
    n_pass = (pg >= 1).sum(axis=1)
    b = np.minimum(n_pass * nb // G, nb - 1)
    for bucket in range(nb):
        sel = np.repeat(b == bucket, G) & (adv != 0)
        assert comp[bucket].sum() == sel.sum()


def test_no_gate_and_full_gate():
    G, M = 8, 3
    pt, nt, gate, adv = _random(9, G=G, M=M)
    none = oracle.rollout_stats(pt, nt, np.zeros_like(gate), G, M)
    assert none["activated_groups"] == none["multi_turn_rollouts"] == 0
    assert none["debugging_groups"] == 0 and none["per_rollout_recovery"] is None
    full = oracle.rollout_stats(pt, nt, np.ones_like(gate), G, M)
    assert full["activated_fraction"] == 1.0
    assert full["multi_turn_rollouts"] == np.count_nonzero(pt != 1)


def test_bad_items_are_skipped():
    pt = np.array([1, 5, 0, 2], np.int32)  # 5 > M
    nt = np.array([1, 1, 0, 2], np.int32)  # T = 0
    r = oracle.rollout_stats(pt, nt, np.array([1], np.uint8), G=4, M=3)
    assert r["bad"] == 2
    assert r["total_turns"] == 3 and r["passed_rollouts"] == 2
    assert r["multi_turn_rollouts"] == 1 and r["recovered_rollouts"] == 1


def test_simulated_debugging_loop():
    """On the mid workload's rollouts, realised with the oracle's own gate:
    ungated rollouts use one turn, gated failures retry up to M turns, and
    the activated fraction is the gate's."""
    lat = wl.draw_latent("mid")
    tmin, tmax = oracle.tau_from_pass_rate(lat.G, Fraction(0), True, Fraction(3, 4), True)
    _, gate = oracle.dcp_gate(lat.first_turn_pass, lat.G, tmin, tmax)
    ro = wl.realize(lat, np.asarray(gate, np.uint8))
    r = oracle.rollout_stats(ro.pass_turn, ro.n_turns, gate, lat.G, lat.M)
    assert r["bad"] == 0
    assert r["activated_groups"] == int(np.sum(gate))
    g = np.repeat(np.asarray(gate, bool), lat.G)
    assert np.all(ro.n_turns[~g] == 1)
    assert r["multi_turn_rollouts"] == np.count_nonzero(g & (ro.pass_turn != 1))
    assert r["turns_per_pass"] >= 1.0
