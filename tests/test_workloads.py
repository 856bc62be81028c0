"""The seeded synthetic workloads that both the oracle and the GPU path draw
from: determinism, the sizes the measurements quote, and the layout
invariants the kernels rely on (rows of a rollout in turn order, feedback and
padding rows excluded, a rollout that passes stops)."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads as wl


def _gated(name):
    lat = wl.draw_latent(name)
    tmin, tmax = oracle.tau_from_pass_rate(lat.G, Fraction(0), True, Fraction(3, 4), True)
    _, gate = oracle.dcp_gate(lat.first_turn_pass, lat.G, tmin, tmax)
    return lat, gate, wl.realize(lat, gate)


@pytest.mark.parametrize("name", ["tiny", "mid", "full", "stress", "lmhead"])
def test_latent_is_deterministic(name):
    a, b = wl.draw_latent(name), wl.draw_latent(name)
    for f in ("p", "turn_pass", "speedup_q", "turn_len", "fb_len"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    assert a.turn_pass.shape == (a.n_groups * a.G, a.M)
    # the speedup is recorded only on a pass; feedback never precedes turn 0
    assert np.all(a.speedup_q[a.turn_pass == 0] == 0)
    assert np.all(a.fb_len[:, 0] == 0)
    cfg = a.cfg
    assert a.turn_len.min() >= cfg["len_lo"] and a.turn_len.max() <= cfg["len_hi"]


def test_tiny_is_one_full_microbatch():
    lat, gate, ro = _gated("tiny")
    mbs = wl.pack(ro, lat.cfg["rows_per_mb"])
    assert ro.n_rollouts == 16 and np.all(ro.n_turns == 1)
    assert len(mbs) == 1 and mbs[0].n_valid == 2048
    assert np.all(mbs[0].tok_turn == 0)


def test_mid_step_sizes():
    # the step every measurement of the logits-resident path runs on
    lat, gate, ro = _gated("mid")
    mbs = wl.pack(ro, lat.cfg["rows_per_mb"])
    assert ro.n_rollouts == 256
    assert len(mbs) == 38 and len(mbs) * lat.cfg["rows_per_mb"] == 311296
    assert sum(m.n_valid for m in mbs) == int(ro.n_tokens.sum()) == 242774


@pytest.mark.parametrize("name", ["mid", "full"])
def test_rollout_and_packing_invariants(name):
    lat, gate, ro = _gated(name)
    G, M = lat.G, lat.M
    gated = np.repeat(gate != 0, G)
    # ungated groups stay single-turn; a pass ends the rollout on that turn;
    # a gated rollout that never passes uses every turn
    assert np.all(ro.n_turns[~gated] == 1)
    passed = ro.pass_turn > 0
    assert np.all(ro.n_turns[passed] == ro.pass_turn[passed])
    assert np.all(ro.n_turns[gated & ~passed] == M)
    assert np.all(ro.speedup_q[~passed] == 0)
    assert np.array_equal(ro.first_turn_pass, lat.turn_pass[:, 0])
    assert np.array_equal(ro.n_tokens, ro.turn_len.sum(axis=1))

    R = lat.cfg["rows_per_mb"]
    mbs = wl.pack(ro, R)
    tr = np.concatenate([m.tok_rollout for m in mbs])
    tt = np.concatenate([m.tok_turn for m in mbs])
    assert all(m.tok_rollout.size == R for m in mbs)
    assert tr.min() >= -1 and tr.max() < ro.n_rollouts
    assert np.all(tt[tr < 0] == 0)
    live = tr >= 0
    # every rollout's generated rows, each turn's count, contiguous per turn
    # and in turn order, within one microbatch
    counts = np.bincount(tr[live], minlength=ro.n_rollouts)
    assert np.array_equal(counts, ro.n_tokens)
    for i in range(0, ro.n_rollouts, max(1, ro.n_rollouts // 40)):
        rows = np.nonzero(tr == i)[0]
        assert rows[0] // R == rows[-1] // R
        turns = tt[rows]
        assert np.all(np.diff(turns) >= 0) and turns[-1] == ro.n_turns[i] - 1
        for t in range(int(ro.n_turns[i])):
            assert int((turns == t).sum()) == int(ro.turn_len[i, t])
        # feedback rows before a later turn are excluded rows right before it
        for t in range(1, int(ro.n_turns[i])):
            start = rows[np.searchsorted(turns, t)]
            fb = int(ro.fb_len[i, t])
            assert np.all(tr[start - fb:start] == -1)
    # rollouts are packed in order: first rows increase with the rollout index
    vals, idx = np.unique(tr[live], return_index=True)
    assert np.array_equal(vals, np.arange(ro.n_rollouts))
    assert np.all(np.diff(np.nonzero(live)[0][idx]) > 0)


def test_stress_shape_and_token_counts():
    lat = wl.draw_latent("stress")
    assert (lat.n_groups, lat.G, lat.M) == (4096, 64, 3)
    n = wl.stress_token_counts(lat)
    assert n.shape == (4096 * 64,) and n.min() >= 200 and n.max() <= 8000
    assert np.array_equal(n, wl.stress_token_counts(lat))


def test_bf16_round_trip_and_rounding():
    # values a bf16 holds exactly come back unchanged (normal extremes included)
    x = np.array([1.0, -2.5, 2.0 ** 127, 2.0 ** -126, 0.0, np.inf, -np.inf], np.float32)
    np.testing.assert_array_equal(wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(x)), x)
    # round to nearest, ties to even: 1 + 2^-8 is a tie between 1 and 1 + 2^-7
    t = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], np.float32)
    np.testing.assert_array_equal(wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(t)),
                                  np.array([1.0, 1.0 + 2.0 ** -6], np.float32))


@pytest.mark.parametrize("name", ["mid", "full"])
def test_right_padded_layout(name):
    """Right-padded microbatches hold the same generated rows as the packed
    layout, each sequence at the start of its own slot with the slot's tail
    and the microbatch's tail excluded."""
    lat, gate, ro = _gated(name)
    R = lat.cfg["rows_per_mb"]
    packed = wl.pack(ro, R)
    rp = wl.pack_right_padded(ro, R)
    seq_len = np.array([wl._sequence(ro, i)[0].size for i in range(ro.n_rollouts)])
    slot = (seq_len.max() + 63) // 64 * 64
    per_mb = R // slot
    assert len(rp) == -(-ro.n_rollouts // per_mb)
    assert sum(m.n_valid for m in rp) == sum(m.n_valid for m in packed) == int(ro.n_tokens.sum())
    for b, m in enumerate(rp):
        assert m.tok_rollout.size == R and m.first_row == b * R
        assert np.all(m.tok_rollout[per_mb * slot:] == -1)
        for j in range(per_mb):
            i = b * per_mb + j
            cell = m.tok_rollout[j * slot:(j + 1) * slot]
            if i >= ro.n_rollouts:
                assert np.all(cell == -1)
                continue
            r, t = wl._sequence(ro, i)
            np.testing.assert_array_equal(cell[:r.size], r)
            np.testing.assert_array_equal(m.tok_turn[j * slot:j * slot + r.size], t)
            assert np.all(cell[r.size:] == -1)
    if name == "mid":
        assert slot == 2304 and per_mb == 3 and len(rp) == 86
