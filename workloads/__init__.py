"""Seeded synthetic workloads shaped like the paper's RL training step.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no tiers, tournaments, gates, advantages, softmax or
loss).  Where a step of the environment depends on a decision of the method
(which groups the pruning gate lets into multi-turn debugging), the decision
is an *input* here, computed by the caller with whichever implementation it
is checking.  Both the oracle tests and the GPU path draw their inputs from
here, so identical seeds give identical inputs.

Workloads (sizes from the paper's training setup, Sec. 4.1, scaled to the
five shapes this library is measured on):

* ``tiny``   -- 2 prompts x G=8, one turn of 128 tokens (2048 rows), V=32768.
* ``mid``    -- 16 prompts x G=16, up to 2 turns of U[256,1024] tokens with
  U[64,512] masked environment-feedback rows between turns, V=151936,
  packed into 8192-row microbatches (tail padding masked); a second,
  right-padded layout puts every sequence in a fixed-length slot.
* ``full``   -- 64 prompts x G=16, up to 3 turns of U[512,4096] tokens,
  V=151936, 16384-row microbatches.
* ``stress`` -- 4096 groups x G=64, M=3, outcome tuples with many ties
  (tournament and gate only; no logits).
* ``lmhead`` -- hidden states [16384 x 4096] ~ N(0,1) and LM-head weight
  [151936 x 4096] ~ N(0, 0.02), outcomes and masks as ``full``.

Outcome model: every turn draws ``compiled ~ Bernoulli(0.8)`` and
``correct | compiled ~ Bernoulli(p)`` with a per-prompt pass probability p
(0.5 for ``tiny``; ``Beta(0.7, 0.7)`` otherwise); a rollout passes a turn
when both hold.  The speedup of a passing rollout is ``LogNormal(0, 0.5)``,
quantised to 0.1 (stored as the integer round(10 * speedup)), 0 otherwise.
Logits are bf16 of ``N(0, sigma^2)`` with sigma = 2; token ids are sampled
from softmax(logits) with the Gumbel-max trick; the old-policy and reference
log-probabilities are the current ones plus ``N(0, 0.05^2)`` and
``N(0, 0.1^2)`` noise, drawn here and added by the caller.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

CONFIGS = {
    "tiny": dict(n_prompts=2, G=8, M=1, len_lo=128, len_hi=128, fb_lo=0, fb_hi=0,
                 V=32768, rows_per_mb=2048, p_pass="fixed0.5", seed=1001, gamma=1.0),
    "mid": dict(n_prompts=16, G=16, M=2, len_lo=256, len_hi=1024, fb_lo=64, fb_hi=512,
                V=151936, rows_per_mb=8192, p_pass="beta0.7", seed=1002, gamma=0.9),
    "full": dict(n_prompts=64, G=16, M=3, len_lo=512, len_hi=4096, fb_lo=64, fb_hi=512,
                 V=151936, rows_per_mb=16384, p_pass="beta0.7", seed=1003, gamma=0.9),
    "stress": dict(n_prompts=4096, G=64, M=3, len_lo=200, len_hi=8000, fb_lo=0, fb_hi=0,
                   V=0, rows_per_mb=0, p_pass="beta0.7", seed=1004, gamma=0.9),
    "lmhead": dict(n_prompts=64, G=16, M=3, len_lo=512, len_hi=4096, fb_lo=64, fb_hi=512,
                   V=151936, H=4096, rows_per_mb=16384, p_pass="beta0.7", seed=1005, gamma=0.9),
}

LOGIT_SIGMA = 2.0
OLD_SIGMA = 0.05
REF_SIGMA = 0.1
CLIP_CASE_OLD_SIGMA = 0.3
LM_HIDDEN_SIGMA = 1.0
LM_WEIGHT_SIGMA = 0.02


@dataclass
class Latent:
    """Per-rollout latent outcomes: what each turn *would* give if attempted."""
    cfg: dict
    n_groups: int
    G: int
    M: int
    p: np.ndarray            # [n_groups] pass probability
    turn_pass: np.ndarray    # [n_rollouts, M] uint8, pass on attempt t
    speedup_q: np.ndarray    # [n_rollouts, M] int32, round(10*speedup) on a pass
    turn_len: np.ndarray     # [n_rollouts, M] int32 generated tokens per turn
    fb_len: np.ndarray       # [n_rollouts, M] int32 feedback rows before turn t (t>=1)

    @property
    def first_turn_pass(self) -> np.ndarray:
        return np.ascontiguousarray(self.turn_pass[:, 0])


@dataclass
class Rollouts:
    """Realised rollouts once the pruning gate of each group is known."""
    G: int
    M: int
    pass_turn: np.ndarray      # [n_rollouts] int32; 0 = never passed, m = first pass on turn m
    n_turns: np.ndarray        # [n_rollouts] int32 generated turns T_i
    first_turn_pass: np.ndarray  # [n_rollouts] uint8
    speedup_q: np.ndarray      # [n_rollouts] int32 (0 unless passed)
    n_tokens: np.ndarray       # [n_rollouts] int32 generated tokens over all turns
    turn_len: np.ndarray       # [n_rollouts, M] int32 (0 for turns not taken)
    fb_len: np.ndarray         # [n_rollouts, M] int32 (0 for turns not taken)

    @property
    def n_rollouts(self) -> int:
        return int(self.pass_turn.size)


@dataclass
class Microbatch:
    tok_rollout: np.ndarray    # [rows] int32, -1 = excluded row
    tok_turn: np.ndarray       # [rows] int32 (0 on excluded rows)
    first_row: int = 0         # index of this microbatch's first row in the step
    n_valid: int = 0


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([int(seed), int(stream)]))


def draw_latent(name: str, seed: int | None = None) -> Latent:
    cfg = dict(CONFIGS[name])
    seed = cfg["seed"] if seed is None else seed
    rng = _rng(seed, 1)
    n_groups, G, M = cfg["n_prompts"], cfg["G"], cfg["M"]
    n = n_groups * G
    if cfg["p_pass"] == "fixed0.5":
        p = np.full(n_groups, 0.5)
    else:
        p = rng.beta(0.7, 0.7, size=n_groups)
    p_roll = np.repeat(p, G)[:, None]
    compiled = rng.random((n, M)) < 0.8
    correct = rng.random((n, M)) < p_roll
    turn_pass = (compiled & correct).astype(np.uint8)
    speed = rng.lognormal(0.0, 0.5, size=(n, M))
    speedup_q = np.where(turn_pass == 1, np.rint(10.0 * speed), 0).astype(np.int32)
    turn_len = rng.integers(cfg["len_lo"], cfg["len_hi"] + 1, size=(n, M)).astype(np.int32)
    if cfg["fb_hi"] > 0:
        fb_len = rng.integers(cfg["fb_lo"], cfg["fb_hi"] + 1, size=(n, M)).astype(np.int32)
        fb_len[:, 0] = 0
    else:
        fb_len = np.zeros((n, M), np.int32)
    return Latent(cfg=cfg, n_groups=n_groups, G=G, M=M, p=p, turn_pass=turn_pass,
                  speedup_q=speedup_q, turn_len=turn_len, fb_len=fb_len)


def realize(lat: Latent, gate: np.ndarray) -> Rollouts:
    """Run the (simulated) debugging loop: a group whose gate is 1 lets each
    failed rollout retry, up to M turns, stopping at its first pass; a group
    whose gate is 0 stays single-turn.  ``gate`` is [n_groups] (any ints)."""
    gate = np.asarray(gate).reshape(-1)
    assert gate.size == lat.n_groups
    n, M = lat.turn_pass.shape
    g_roll = np.repeat(gate != 0, lat.G)
    pass_turn = np.zeros(n, np.int32)
    n_turns = np.ones(n, np.int32)
    speed = np.zeros(n, np.int32)
    for i in range(n):
        limit = M if g_roll[i] else 1
        taken = limit
        for t in range(limit):
            if lat.turn_pass[i, t]:
                pass_turn[i] = t + 1
                speed[i] = lat.speedup_q[i, t]
                taken = t + 1
                break
        n_turns[i] = taken
    turn_len = lat.turn_len.copy()
    fb_len = lat.fb_len.copy()
    cols = np.arange(M)[None, :]
    taken_mask = cols < n_turns[:, None]
    turn_len[~taken_mask] = 0
    fb_len[~taken_mask] = 0
    n_tokens = turn_len.sum(axis=1).astype(np.int32)
    return Rollouts(G=lat.G, M=M, pass_turn=pass_turn, n_turns=n_turns,
                    first_turn_pass=lat.first_turn_pass.astype(np.uint8),
                    speedup_q=speed, n_tokens=n_tokens, turn_len=turn_len, fb_len=fb_len)


def stress_token_counts(lat: Latent, seed: int | None = None) -> np.ndarray:
    """Token counts U{200..8000} for the tournament stress workload."""
    seed = lat.cfg["seed"] if seed is None else seed
    rng = _rng(seed, 2)
    return rng.integers(200, 8001, size=lat.turn_pass.shape[0]).astype(np.int32)


def _sequence(ro: Rollouts, i: int):
    """Rows of rollout i's sequence: turn 0, then for each later turn its
    environment-feedback rows (excluded, -1) followed by its generated rows.
    Returns (rollout index per row, turn per row)."""
    segs_r, segs_t = [], []
    for t in range(int(ro.n_turns[i])):
        fb = int(ro.fb_len[i, t])
        if fb:
            segs_r.append(np.full(fb, -1, np.int32))
            segs_t.append(np.zeros(fb, np.int32))
        ln = int(ro.turn_len[i, t])
        segs_r.append(np.full(ln, i, np.int32))
        segs_t.append(np.full(ln, t, np.int32))
    return np.concatenate(segs_r), np.concatenate(segs_t)


def pack_right_padded(ro: Rollouts, rows_per_mb: int, slot_rows: int | None = None
                      ) -> list[Microbatch]:
    """Right-padded layout: each rollout's sequence starts a slot of
    ``slot_rows`` rows (default: the step's longest sequence rounded up to a
    multiple of 64) and the rest of the slot is excluded padding; a
    microbatch of ``rows_per_mb`` rows holds floor(rows_per_mb / slot_rows)
    slots in rollout order, and its rows past the last slot are excluded
    too.  ``first_row`` is the microbatch's first row in the step."""
    seqs = [_sequence(ro, i) for i in range(ro.n_rollouts)]
    if slot_rows is None:
        longest = max((r.size for r, _ in seqs), default=1)
        slot_rows = (longest + 63) // 64 * 64
    assert 0 < slot_rows <= rows_per_mb, "slot longer than a microbatch"
    per_mb = rows_per_mb // slot_rows
    mbs: list[Microbatch] = []
    for m0 in range(0, len(seqs), per_mb):
        tr = np.full(rows_per_mb, -1, np.int32)
        tt = np.zeros(rows_per_mb, np.int32)
        for j, (r, t) in enumerate(seqs[m0:m0 + per_mb]):
            assert r.size <= slot_rows, "sequence longer than its slot"
            tr[j * slot_rows: j * slot_rows + r.size] = r
            tt[j * slot_rows: j * slot_rows + t.size] = t
        mbs.append(Microbatch(tok_rollout=tr, tok_turn=tt, first_row=len(mbs) * rows_per_mb,
                              n_valid=int((tr >= 0).sum())))
    return mbs


def pack(ro: Rollouts, rows_per_mb: int) -> list[Microbatch]:
    """Pack whole rollout sequences, in rollout order, into microbatches of
    ``rows_per_mb`` rows.  A sequence is turn 0, then for each later turn its
    environment-feedback rows (excluded) followed by its generated rows.  The
    tail of each microbatch is excluded padding."""
    mbs: list[Microbatch] = []
    cur_r: list[np.ndarray] = []
    cur_t: list[np.ndarray] = []
    used = 0
    first = 0
    step_row = 0

    def flush():
        nonlocal cur_r, cur_t, used, first
        tr = np.full(rows_per_mb, -1, np.int32)
        tt = np.zeros(rows_per_mb, np.int32)
        if cur_r:
            r = np.concatenate(cur_r)
            t = np.concatenate(cur_t)
            tr[: r.size] = r
            tt[: t.size] = t
        mbs.append(Microbatch(tok_rollout=tr, tok_turn=tt, first_row=first,
                              n_valid=int((tr >= 0).sum())))
        cur_r, cur_t, used = [], [], 0

    for i in range(ro.n_rollouts):
        seq_r, seq_t = _sequence(ro, i)
        assert seq_r.size <= rows_per_mb, "sequence longer than a microbatch"
        if used + seq_r.size > rows_per_mb:
            flush()
            first = step_row
        cur_r.append(seq_r)
        cur_t.append(seq_t)
        used += seq_r.size
        step_row += seq_r.size
    if used:
        flush()
    return mbs


# ----------------------------------------------------------------------------
# Logits, sampled tokens and log-probability noise
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = 0x7FFF + ((u >> 16) & 1)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def logits_host(seed: int, rows: int, V: int, ld: int | None = None,
                sigma: float = LOGIT_SIGMA) -> np.ndarray:
    """bf16 bit patterns [rows, ld] of N(0, sigma^2); columns >= V are zero."""
    ld = V if ld is None else ld
    rng = _rng(seed, 3)
    out = np.zeros((rows, ld), np.uint16)
    chunk = max(1, (1 << 24) // max(V, 1))
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        x = rng.standard_normal((r1 - r0, V), dtype=np.float32) * np.float32(sigma)
        out[r0:r1, :V] = f32_to_bf16_bits(x)
    return out


def sample_tokens_host(logits_u16: np.ndarray, V: int, seed: int) -> np.ndarray:
    """Gumbel-max draws y_k ~ softmax(logits_k) (an exact sampler)."""
    rng = _rng(seed, 4)
    rows = logits_u16.shape[0]
    out = np.empty(rows, np.int32)
    chunk = max(1, (1 << 22) // max(V, 1))
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        z = bf16_bits_to_f32(logits_u16[r0:r1, :V]).astype(np.float64)
        u = rng.random((r1 - r0, V))
        gum = -np.log(-np.log(np.clip(u, 1e-300, None)))
        out[r0:r1] = np.argmax(z + gum, axis=1).astype(np.int32)
    return out


def logits_device(seed: int, rows: int, V: int, ld: int | None = None,
                  sigma: float = LOGIT_SIGMA, device="cuda", out=None):
    """bf16 torch tensor [rows, ld] of N(0, sigma^2) drawn on the device with a
    seeded torch generator (columns >= V are zero)."""
    import torch
    ld = V if ld is None else ld
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 7919 + 3)
    if out is None:
        out = torch.empty((rows, ld), dtype=torch.bfloat16, device=device)
    if ld > V:
        out[:, V:].zero_()
    chunk = max(1, (1 << 26) // max(V, 1))
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        x = torch.randn((r1 - r0, V), generator=g, device=device, dtype=torch.float32)
        out[r0:r1, :V] = (x * sigma).to(torch.bfloat16)
    return out


def sample_tokens_device(logits, V: int, seed: int):
    """Gumbel-max draws on the device; returns int32 tensor [rows]."""
    import torch
    g = torch.Generator(device=logits.device)
    g.manual_seed(int(seed) * 7919 + 4)
    rows = logits.shape[0]
    out = torch.empty(rows, dtype=torch.int32, device=logits.device)
    chunk = max(1, (1 << 26) // max(V, 1))
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        u = torch.rand((r1 - r0, V), generator=g, device=logits.device, dtype=torch.float32)
        u.clamp_(min=1e-38)
        gum = -torch.log(-torch.log(u))
        out[r0:r1] = torch.argmax(logits[r0:r1, :V].float() + gum, dim=1).to(torch.int32)
    return out


def lmhead_operands_device(seed: int, N: int, V: int, H: int, device,
                           hidden_sigma: float = LM_HIDDEN_SIGMA,
                           weight_sigma: float = LM_WEIGHT_SIGMA):
    """bf16 torch tensors hidden [N, H] ~ N(0, hidden_sigma^2) and weight
    [V, H] ~ N(0, weight_sigma^2), drawn on the device."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 7919 + 11)
    hid = torch.empty((N, H), dtype=torch.bfloat16, device=device)
    wt = torch.empty((V, H), dtype=torch.bfloat16, device=device)
    chunk = max(1, (1 << 26) // max(H, 1))
    for r0 in range(0, N, chunk):
        r1 = min(N, r0 + chunk)
        hid[r0:r1] = (torch.randn((r1 - r0, H), generator=g, device=device) * hidden_sigma).to(torch.bfloat16)
    for r0 in range(0, V, chunk):
        r1 = min(V, r0 + chunk)
        wt[r0:r1] = (torch.randn((r1 - r0, H), generator=g, device=device) * weight_sigma).to(torch.bfloat16)
    return hid, wt


def lmhead_tokens_device(hidden, weight, seed: int, row_chunk: int = 256):
    """Gumbel-max draws y_k ~ softmax(hidden_k weight^T), the logits formed in
    fp32 a block of rows at a time (generation only).  int32 tensor [N]."""
    import torch
    N = hidden.shape[0]
    g = torch.Generator(device=hidden.device)
    g.manual_seed(int(seed) * 7919 + 12)
    y = torch.empty(N, dtype=torch.int32, device=hidden.device)
    wf = weight.float()
    for r0 in range(0, N, row_chunk):
        r1 = min(N, r0 + row_chunk)
        z = hidden[r0:r1].float() @ wf.T
        u = torch.rand(z.shape, generator=g, device=z.device).clamp_(min=1e-38)
        y[r0:r1] = torch.argmax(z - torch.log(-torch.log(u)), dim=1).to(torch.int32)
    return y


def logp_noise(seed: int, N: int, old_sigma: float = OLD_SIGMA,
               ref_sigma: float = REF_SIGMA):
    """(noise_old, noise_ref) float64 [N]: added by the caller to the current
    log-probabilities to form the old-policy and reference inputs."""
    rng = _rng(seed, 5)
    return rng.normal(0.0, old_sigma, N), rng.normal(0.0, ref_sigma, N)


def rollout_arrays_for_gate(lat: Latent):
    """First-turn outcomes as the gate consumes them: uint8 [n_groups*G]."""
    return lat.first_turn_pass.astype(np.uint8)
