"""Benchmark of the LEAP GRPO hot path on one MI355X.

One step = one pass of the whole hot path over one RL training step:

  leap_dcp_gate                    first-turn outcomes -> multi-turn gate
  leap_rank_advantages             final outcomes -> tournament reward, advantage
  leap_token_advantages            every row of the step -> token advantage, weight
  leap_grpo_logprob_loss_fwd_bwd   per microbatch: log-softmax, surrogate, KL,
                                   loss and bf16 dlogits

The headline workload is the "full" paper-shaped step: 64 prompts x G=16
rollouts, up to 3 turns of U[512,4096] generated tokens with masked
environment-feedback rows between turns, vocabulary 151936, 305 microbatches
of 16384 rows (about 5 GB of bf16 logits each, 1.5 TB for the step).  The
step's logits cannot all be resident, so three 16384-row logits buffers (and
three dlogits buffers) are cycled: microbatch i reads buffer i mod 3 with its
own rows' side inputs (token ids sampled from that buffer's logits, old /
reference log-probs from them plus noise, and the token advantages and
weights the step's own gate, tournament and token-advantage calls produce
for the microbatch's rows, masked rows included).  The "mid" step (16 x 16,
up to 2 turns, 38 microbatches of 8192 rows) runs as a secondary leg with
every microbatch's logits resident.

Every input is resident in HBM before a timed region; dlogits go to separate
buffers, so every step sees the same inputs.  Prints one JSON line on
stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12  # MI355X HBM3E, bytes/s
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k4_grpo_rows_traffic.json")
# The fused row kernel's translation unit: the source and every header it includes.
K4_SOURCES = [os.path.join(ROOT, "paper_2608_01804_amd", "csrc", f)
              for f in ("grpo_loss.hip", "row_common.h", "objective.h", "leap_common.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def k4_source_hash() -> str:
    h = hashlib.sha256()
    for f in K4_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def settle(torch, fn, ms: float = 300.0) -> None:
    """Run fn back to back for about `ms` milliseconds before a timed region.
    After idle time or a run of short kernels the device takes tens of
    milliseconds to bring its clocks back up (the forward-only leg timed
    right after the shard leg measured 455 us against 384 us once settled),
    and a short timed region would include that ramp."""
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(4):
            fn()
        torch.cuda.synchronize()


def row_bytes(V: int, valid: bool) -> int:
    """Algorithmic HBM bytes of one row of the fused kernel.
    valid row : read 2V (logits) + 20 (token id, old, ref, adv, w)
                write 2V (dlogits) + 8 (logp, weighted row loss)
    masked row: read 8 (w, token id); write 2V (zero dlogits) + 8."""
    return 4 * V + 28 if valid else 2 * V + 16


def build_step(L, torch, dev, name, seed, n_buffers=None):
    """The step's rollouts, gate, layout and inputs.  ``n_buffers`` logits
    buffers of one microbatch each are generated (default: one per
    microbatch, all resident); microbatch i reads buffer i mod n_buffers."""
    import workloads as wl
    lat = wl.draw_latent(name)
    cfg = lat.cfg
    G, M, V, R = lat.G, lat.M, cfg["V"], cfg["rows_per_mb"]
    tmin, tmax = L.leap_dcp_tau_from_pass_rate(G, 0, 1, 1, 3, 4, 1)  # 0 < pass rate < 3/4
    ftp_d = torch.from_numpy(lat.first_turn_pass).to(dev)
    gate_d = torch.empty(lat.n_groups, dtype=torch.uint8, device=dev)
    nf_d = torch.empty(lat.n_groups, dtype=torch.int32, device=dev)
    L.leap_dcp_gate(ftp_d, lat.n_groups, G, tmin, tmax, nf_d, gate_d)
    ro = wl.realize(lat, gate_d.cpu().numpy())
    mbs = wl.pack(ro, R)
    n_mb = len(mbs)
    n_buf = n_mb if n_buffers is None else min(n_buffers, n_mb)
    rows = n_mb * R
    tok_r = np.concatenate([m.tok_rollout for m in mbs])
    tok_t = np.concatenate([m.tok_turn for m in mbs])
    valid = tok_r >= 0
    log(f"[bench] workload {name}: {ro.n_rollouts} rollouts, {n_mb} microbatches x {R} rows, "
        f"{int(valid.sum())} generated tokens, V={V}; {n_buf} resident logits buffers "
        f"({n_buf * R * V * 2 / 1e9:.1f} GB)")

    s = {"name": name, "lat": lat, "ro": ro, "mbs": mbs, "V": V, "R": R, "rows": rows,
         "n_mb": n_mb, "n_buf": n_buf, "G": G, "M": M, "tau": (tmin, tmax), "valid": valid,
         "gamma": cfg["gamma"]}
    s["ftp"] = ftp_d
    s["gate"] = gate_d
    s["n_fail"] = nf_d
    s["pass_turn"] = torch.from_numpy(ro.pass_turn).to(dev)
    s["n_turns"] = torch.from_numpy(ro.n_turns).to(dev)
    s["n_gen"] = torch.from_numpy(ro.n_tokens).to(dev)
    s["tok_r"] = torch.from_numpy(tok_r).to(dev)
    s["tok_t"] = torch.from_numpy(tok_t).to(dev)
    n = ro.n_rollouts
    s["reward"] = torch.empty(n, dtype=torch.float32, device=dev)
    s["adv_roll"] = torch.empty(n, dtype=torch.float32, device=dev)
    s["adv_tok"] = torch.empty(rows, dtype=torch.float32, device=dev)
    s["w_tok"] = torch.empty(rows, dtype=torch.float32, device=dev)

    # the logits buffers, resident; dlogits in separate buffers
    t0 = time.time()
    s["logits"] = torch.empty((n_buf * R, V), dtype=torch.bfloat16, device=dev)
    s["dlogits"] = torch.empty((n_buf * R, V), dtype=torch.bfloat16, device=dev)
    tok_buf = torch.empty(n_buf * R, dtype=torch.int32, device=dev)
    for b in range(n_buf):
        sl = slice(b * R, (b + 1) * R)
        wl.logits_device(seed + b, R, V, device=dev, out=s["logits"][sl])
        tok_buf[sl] = wl.sample_tokens_device(s["logits"][sl], V, seed + b)
    torch.cuda.synchronize()
    log(f"[bench] logits and sampled tokens ready in {time.time() - t0:.1f} s")

    # current log-probs from the library's forward-only pass, then, per row
    # of the step, old / reference = current + N(0, 0.05^2) / N(0, 0.1^2)
    cur_buf = torch.empty(n_buf * R, dtype=torch.float32, device=dev)
    L.leap_logprob_fwd(s["logits"], V, n_buf * R, V, tok_buf, None, 1.0, cur_buf)
    reps = -(-n_mb // n_buf)
    s["tok"] = tok_buf.view(n_buf, R).repeat(reps, 1)[:n_mb].reshape(-1).contiguous()
    cur = cur_buf.view(n_buf, R).repeat(reps, 1)[:n_mb].reshape(-1)
    n_old, n_ref = wl.logp_noise(seed, rows)
    s["old"] = (cur + torch.from_numpy(n_old.astype(np.float32)).to(dev)).contiguous()
    s["ref"] = (cur + torch.from_numpy(n_ref.astype(np.float32)).to(dev)).contiguous()
    del cur, cur_buf, tok_buf
    ws_bytes = L.leap_grpo_workspace_size(R, V)
    s["ws"] = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    s["ws_bytes"] = ws_bytes
    s["loss"] = torch.empty(n_mb, dtype=torch.float32, device=dev)
    s["err"] = torch.zeros(1, dtype=torch.int32, device=dev)
    s["params"] = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
    torch.cuda.synchronize()
    return s


def mb_logits(s, i):
    """(logits, dlogits) buffers microbatch i reads and writes."""
    R = s["R"]
    b = i % s["n_buf"]
    return s["logits"][b * R:(b + 1) * R], s["dlogits"][b * R:(b + 1) * R]


def run_step(L, s, events=None):
    """The whole hot path over one step.  events: list of (start, end) CUDA
    event pairs to record around each fused-kernel call, or None."""
    import torch
    G, M, R, V = s["G"], s["M"], s["R"], s["V"]
    n = s["ro"].n_rollouts
    L.leap_dcp_gate(s["ftp"], n // G, G, s["tau"][0], s["tau"][1], s["n_fail"], s["gate"])
    L.leap_rank_advantages(s["pass_turn"], None, None, n // G, G, M, L.LEAP_KEY_TURN,
                           L.LEAP_ADV_STD, 1e-6, None, None, None, s["reward"], s["adv_roll"],
                           s["err"])
    L.leap_token_advantages(s["adv_roll"], s["tok_r"], s["tok_t"], s["n_turns"], s["n_gen"], n,
                            s["rows"], s["gamma"], L.LEAP_AGG_SEQ_MEAN_TOKEN_MEAN, float(n),
                            s["adv_tok"], s["w_tok"], s["err"])
    stream = torch.cuda.current_stream()
    for i in range(s["n_mb"]):
        sl = slice(i * R, (i + 1) * R)
        lg, dl = mb_logits(s, i)
        if events is not None:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
        L.leap_grpo_logprob_loss_fwd_bwd(lg, V, R, V, s["tok"][sl], s["old"][sl],
                                         s["ref"][sl], s["adv_tok"][sl], s["w_tok"][sl],
                                         s["params"], None, None, None, s["loss"][i:i + 1],
                                         dl, s["ws"], s["ws_bytes"], s["err"])
        if events is not None:
            e1.record(stream)
            events.append((e0, e1))


COPY_PROBE_BYTES = 1 << 30


def copy_probe(torch, dev):
    """A plain elementwise kernel of known size (reads 1 GiB, writes 1 GiB):
    the reference the profiler's HBM byte counters are scaled by."""
    a = torch.ones(COPY_PROBE_BYTES // 2, dtype=torch.int16, device=dev)
    b = torch.empty_like(a)
    torch.bitwise_not(a, out=b)
    torch.cuda.synchronize()


def hbm_probe(L, torch, dev, gib: int = 4, reps: int = 5):
    """Achievable HBM rates of the device for the three access mixes, from
    the library's streaming probe (median of `reps` launches over `gib` GiB)."""
    n = gib << 30
    a = torch.ones(n // 2, dtype=torch.int16, device=dev)
    b = torch.empty_like(a)
    out = {}
    for mode, name, moved in ((0, "copy", 2 * n), (1, "read", n), (2, "write", n)):
        settle(torch, lambda: L.leap_probe_hbm(a, b, n, mode))
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            L.leap_probe_hbm(a, b, n, mode)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        out[f"{name}_GBps"] = moved / float(np.median(ts)) / 1e9
    del a, b
    torch.cuda.empty_cache()
    return out


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_rows_inputs(s, rows):
    """Host copies of the given step rows' inputs: bf16 logits (from the
    buffer each row's microbatch reads), token ids, old / reference log-probs."""
    import torch
    R, nb = s["R"], s["n_buf"]
    brow = (rows // R) % nb * R + rows % R
    dev = s["logits"].device
    lg = s["logits"].index_select(0, torch.as_tensor(brow, device=dev))
    idx = torch.as_tensor(rows, device=dev)
    return (lg.view(torch.int16).cpu().numpy().view(np.uint16), s["tok"][idx].cpu().numpy(),
            s["old"][idx].cpu().numpy(), s["ref"][idx].cpu().numpy())


def cpu_baseline(s, seconds: float, samples: int = 3):
    """The fp64 oracle (as it is) on the host cores over a bounded sample of
    the same step: the tournament, gate and token advantages over the whole
    step, then the fused objective with dlogits on generated-token rows of
    the step for about seconds / samples each, `samples` times (different
    rows each time); the whole-step time at the median per-row rate.  Then
    the same on one thread over a shorter sample."""
    import oracle
    ro, lat = s["ro"], s["lat"]
    cores = oracle.get_threads()
    tok_r = s["tok_r"].cpu().numpy()
    tok_t = s["tok_t"].cpu().numpy()

    def small_steps():
        t0 = time.perf_counter()
        oracle.dcp_gate(lat.first_turn_pass, s["G"], *s["tau"])
        rk = oracle.rank_tournament(ro.pass_turn, s["G"], s["M"], eps=float(np.float32(1e-6)))
        adv, w, _ = oracle.token_advantages(rk["A"], tok_r, tok_t, ro.n_turns, ro.n_tokens,
                                            s["gamma"], oracle.AGG_SEQ_MEAN_TOKEN_MEAN,
                                            float(ro.n_rollouts))
        return time.perf_counter() - t0, adv, w

    t_small, adv, w = small_steps()
    valid_rows = np.flatnonzero(w != 0)  # generated-token rows of the whole step
    n_valid = valid_rows.size

    def row_rate(start, budget, chunk):
        """Oracle seconds per row over rows from `start` until `budget` s
        of oracle time (device->host copies of the sample excluded)."""
        done, t = 0, 0.0
        while t < budget and start + done < n_valid:
            rows = valid_rows[start + done:start + done + chunk]
            lg, tok, old, ref = _oracle_rows_inputs(s, rows)
            tc = time.perf_counter()
            oracle.grpo_rows(lg, tok, old, ref, adv[rows], w[rows])
            t += time.perf_counter() - tc
            done += rows.size
        return t / max(done, 1), done, t

    rates = []
    start = 0
    for _ in range(samples):
        r, done, t = row_rate(start, seconds / samples, 4 * cores)
        rates.append((r, done, t))
        start += done
    per_row = float(np.median([r for r, _, _ in rates]))
    step_time = t_small + per_row * n_valid

    oracle.set_threads(1)
    try:
        t_small1, _, _ = small_steps()
        per_row1, done1, t_rows1 = row_rate(0, seconds / 4, 8)
    finally:
        oracle.set_threads(cores)
    step_time1 = t_small1 + per_row1 * n_valid
    return {"value": n_valid / step_time, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"gate+tournament+token advantages over the whole step ({t_small * 1e3:.1f} ms), "
                      f"then the fused objective with dlogits on {samples} samples of "
                      f"generated-token rows ({', '.join(f'{d} rows in {t:.1f} s' for _, d, t in rates)}); "
                      f"median per-row rate scaled to the step's {n_valid} tokens",
            "cpu_model": _cpu_model(), "nproc": os.cpu_count(),
            "value_1_thread": n_valid / step_time1,
            "sample_1_thread": f"the same on one thread: small steps {t_small1 * 1e3:.1f} ms, fused "
                               f"objective on {done1} rows ({t_rows1:.1f} s)"}


MFMA_BF16_PEAK = 2.5e15  # MI355X dense bf16 matrix-core peak, flop/s


def shard_leg(L, torch, s, n_shards: int = 8, reps: int = 20):
    """The vocabulary-parallel entry points at one shard's real shape: the
    first microbatch's rows, the first V / n_shards columns of the resident
    logits (row stride V), n_shards partials for the merge (shard 0's own and
    copies that own no token).  HIP events on the launch stream around `reps`
    back-to-back calls (as in a training step), per-call average."""
    V, R = s["V"], s["R"]
    vs = V // n_shards
    lg = s["logits"][:R]
    dl = s["dlogits"][:R]
    tok, w = s["tok"][:R], s["w_tok"][:R]
    dev = lg.device
    parts = torch.empty((n_shards, R, 4), dtype=torch.float32, device=dev)
    state = torch.empty((R, 2), dtype=torch.float32, device=dev)
    logp = torch.empty(R, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    ws_bytes = L.leap_vocab_merge_workspace_size(R)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    def timed(fn):
        settle(torch, fn)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps / 1e3

    t_stats = timed(lambda: L.leap_vocab_shard_stats(lg, V, R, vs, 0, tok, w, 1.0, parts[0]))
    parts[1:] = parts[0]
    parts[1:, :, 3] = 0.0  # copies own no token
    parts[1:, :, 2] = 0.0
    owned0 = parts[0, :, 3].clone()
    parts[0, :, 3] = 1.0  # every row's token counted once (timing only)
    t_merge = timed(lambda: L.leap_vocab_merge_objective(
        parts, n_shards, R, V, tok, s["old"][:R], s["ref"][:R], s["adv_tok"][:R], w, s["params"],
        logp, None, loss, state, ws, ws_bytes, err))
    parts[0, :, 3] = owned0
    t_bwd = timed(lambda: L.leap_vocab_shard_bwd(lg, V, R, vs, 0, tok, state, 1.0, dl))
    nv = int((w != 0).sum().item())
    stats_bytes = nv * (2 * vs + 8) + R * 24
    bwd_bytes = nv * (4 * vs + 12) + (R - nv) * (2 * vs + 12)
    log(f"[bench] vocab shard {R} x {vs}: stats {t_stats * 1e6:.1f} us "
        f"({stats_bytes / t_stats / 1e9:.0f} GB/s), merge of {n_shards} {t_merge * 1e6:.1f} us, "
        f"bwd {t_bwd * 1e6:.1f} us ({bwd_bytes / t_bwd / 1e9:.0f} GB/s)")
    return {"workload": f"one vocabulary shard: first microbatch ({R} rows, {nv} live) x "
                        f"{vs} columns (V/{n_shards}), row stride {V}",
            "stats_us": t_stats * 1e6, "stats_GBps": stats_bytes / t_stats / 1e9,
            "merge_us": t_merge * 1e6, "bwd_us": t_bwd * 1e6, "bwd_GBps": bwd_bytes / t_bwd / 1e9,
            "stats_frac": stats_bytes / t_stats / HBM_PEAK, "bwd_frac": bwd_bytes / t_bwd / HBM_PEAK}


def _us_per_call(torch, fn, reps: int) -> float:
    """Average µs per call of `reps` back-to-back calls of fn (HIP events on
    the launch stream), after a short settling run."""
    stream = torch.cuda.current_stream()
    settle(torch, fn, ms=100)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps * 1e3


def graph_leg(L, torch, s, steps: int):
    """The whole step captured once in a HIP graph and replayed `steps`
    times (host clock around the replays, synchronised on both sides):
    what launching the step's calls one by one costs against a replay."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run_step(L, s)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run_step(L, s)
    settle(torch, g.replay)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / steps
    log(f"[bench] step replayed from a HIP graph: {t * 1e3:.3f} ms")
    return {"ms_per_step": t * 1e3, "steps": steps}


def small_leg(L, torch, s, reps: int = 200):
    """Latency of the gate, the tournament and the token advantages (µs per
    call): on the measured step, and the gate and tournament on the
    tournament-stress workload (4096 groups x G=64, M=3), both outcome
    orders."""
    import workloads as wl
    G, M = s["G"], s["M"]
    n = s["ro"].n_rollouts
    mid = {
        "groups": n // G, "G": G, "rows": s["rows"],
        "gate_us": _us_per_call(torch, lambda: L.leap_dcp_gate(
            s["ftp"], n // G, G, s["tau"][0], s["tau"][1], s["n_fail"], s["gate"]), reps),
        "rank_us": _us_per_call(torch, lambda: L.leap_rank_advantages(
            s["pass_turn"], None, None, n // G, G, M, L.LEAP_KEY_TURN, L.LEAP_ADV_STD, 1e-6, None,
            None, None, s["reward"], s["adv_roll"], s["err"]), reps),
        "token_adv_us": _us_per_call(torch, lambda: L.leap_token_advantages(
            s["adv_roll"], s["tok_r"], s["tok_t"], s["n_turns"], s["n_gen"], n, s["rows"],
            s["gamma"], L.LEAP_AGG_SEQ_MEAN_TOKEN_MEAN, float(n), s["adv_tok"], s["w_tok"],
            s["err"]), reps),
    }
    dev = s["pass_turn"].device
    lat = wl.draw_latent("stress")
    Gs, Ms, ng = lat.G, lat.M, lat.n_groups
    tmin, tmax = L.leap_dcp_tau_from_pass_rate(Gs, 0, 1, 1, 3, 4, 1)
    ftp = torch.from_numpy(lat.first_turn_pass).to(dev)
    gate = torch.empty(ng, dtype=torch.uint8, device=dev)
    nf = torch.empty(ng, dtype=torch.int32, device=dev)
    L.leap_dcp_gate(ftp, ng, Gs, tmin, tmax, nf, gate)
    ro = wl.realize(lat, gate.cpu().numpy())
    pt = torch.from_numpy(ro.pass_turn).to(dev)
    sq = torch.from_numpy(ro.speedup_q).to(dev)
    nt = torch.from_numpy(wl.stress_token_counts(lat)).to(dev)
    nr = ng * Gs
    rew = torch.empty(nr, dtype=torch.float32, device=dev)
    adv = torch.empty(nr, dtype=torch.float32, device=dev)
    stress = {
        "groups": ng, "G": Gs, "rollouts": nr,
        "gate_us": _us_per_call(torch, lambda: L.leap_dcp_gate(ftp, ng, Gs, tmin, tmax, nf, gate),
                                reps),
        "rank_turn_us": _us_per_call(torch, lambda: L.leap_rank_advantages(
            pt, None, None, ng, Gs, Ms, L.LEAP_KEY_TURN, L.LEAP_ADV_STD, 1e-6, None, None, None,
            rew, adv, s["err"]), reps),
        "rank_lex_us": _us_per_call(torch, lambda: L.leap_rank_advantages(
            pt, sq, nt, ng, Gs, Ms, L.LEAP_KEY_LEX, L.LEAP_ADV_STD, 1e-6, None, None, None, rew,
            adv, s["err"]), reps),
    }
    log(f"[bench] step: gate {mid['gate_us']:.1f} us, tournament {mid['rank_us']:.1f} us, token "
        f"advantages {mid['token_adv_us']:.1f} us; stress {ng}x{Gs}: gate {stress['gate_us']:.1f} "
        f"us, tournament {stress['rank_turn_us']:.1f} us (turn), {stress['rank_lex_us']:.1f} us (lex)")
    return {"step": mid, "stress": stress}


def entropy_leg(L, torch, s, reps: int = 20):
    """The fused call on the first microbatch without and with the optional
    per-token entropy output (HIP events on the launch stream, per-call
    average of `reps` back-to-back calls each): the entropy's cost."""
    V, R = s["V"], s["R"]
    ent = torch.empty(R, dtype=torch.float32, device=s["logits"].device)
    stream = torch.cuda.current_stream()

    def timed(entropy_out):
        def call():
            L.leap_grpo_logprob_loss_fwd_bwd(s["logits"][:R], V, R, V, s["tok"][:R], s["old"][:R],
                                             s["ref"][:R], s["adv_tok"][:R], s["w_tok"][:R],
                                             s["params"], None, None, entropy_out, s["loss"][:1],
                                             s["dlogits"][:R], s["ws"], s["ws_bytes"], s["err"])

        settle(torch, call)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps / 1e3

    t, t_ent = timed(None), timed(ent)
    log(f"[bench] fused call, first microbatch: {t * 1e6:.1f} us; with entropy {t_ent * 1e6:.1f} us")
    return {"workload": f"fused call on the first microbatch ({R} x {V})", "call_us": t * 1e6,
            "call_us_with_entropy": t_ent * 1e6}


def logprob_leg(L, torch, s, reps: int = 20):
    """The forward-only log-probability (old-policy / reference passes) on the
    first microbatch of the resident logits, every row read: HIP events on the
    launch stream around `reps` back-to-back calls, per-call average; then the
    same with the optional per-row entropy output."""
    V, R = s["V"], s["R"]
    lg, tok = s["logits"][:R], s["tok"][:R]
    out = torch.empty(R, dtype=torch.float32, device=lg.device)
    ent = torch.empty(R, dtype=torch.float32, device=lg.device)
    stream = torch.cuda.current_stream()

    def timed(entropy_out):
        def call():
            L.leap_logprob_fwd(lg, V, R, V, tok, None, 1.0, out, entropy_out, s["err"])

        settle(torch, call)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps / 1e3

    t = timed(None)
    t_ent = timed(ent)
    nbytes = R * (2 * V + 8)
    log(f"[bench] forward-only log-prob {R} x {V}: {t * 1e6:.1f} us ({nbytes / t / 1e9:.0f} GB/s); "
        f"with entropy {t_ent * 1e6:.1f} us")
    return {"workload": f"forward-only log-prob: first microbatch ({R} rows, all read) x {V}",
            "call_us": t * 1e6, "GBps": nbytes / t / 1e9, "frac": nbytes / t / HBM_PEAK,
            "bytes_per_call": nbytes, "call_us_with_entropy": t_ent * 1e6}


def _token_logp_torch(torch, hidden, weight, y, row_chunk=256):
    """fp32 log-softmax of hidden weight^T at y with torch, a block of rows at
    a time: input preparation for the old / reference log-probabilities."""
    out = torch.empty(hidden.shape[0], dtype=torch.float32, device=hidden.device)
    wf = weight.float()
    yl = y.long()
    for r0 in range(0, hidden.shape[0], row_chunk):
        r1 = min(hidden.shape[0], r0 + row_chunk)
        z = hidden[r0:r1].float() @ wf.T
        out[r0:r1] = torch.log_softmax(z, dim=1).gather(1, yl[r0:r1, None])[:, 0]
    del wf
    return out


STAT_FIELDS = ("groups", "rollouts", "activated_groups", "multi_turn_rollouts",
               "recovered_rollouts", "debugging_groups", "recovered_groups", "total_turns",
               "passed_rollouts")


def stats_report(counters, n_buckets: int) -> dict:
    """The counters leap_rollout_stats wrote, named, with the rates the paper
    reports formed from them for the benchmark's record (activated fraction,
    per-rollout and per-group recovery, turns per pass)."""
    c = [int(v) for v in counters]
    out = dict(zip(STAT_FIELDS, c[:9]))
    out["composition"] = [[c[9 + (b * 3 + o) * 2: 9 + (b * 3 + o) * 2 + 2] for o in range(3)]
                          for b in range(n_buckets)]
    ratio = lambda a, b: (a / b) if b else None  # noqa: E731
    out["activated_fraction"] = ratio(out["activated_groups"], out["groups"])
    out["per_rollout_recovery"] = ratio(out["recovered_rollouts"], out["multi_turn_rollouts"])
    out["per_group_recovery"] = ratio(out["recovered_groups"], out["debugging_groups"])
    out["turns_per_pass"] = ratio(out["total_turns"], out["passed_rollouts"])
    return out


def stats_leg(L, torch, s, n_buckets: int = 10, reps: int = 20):
    """The step's training statistics (activated groups, recovery rates,
    turns per pass, advantage-sign composition) from its own gate, outcomes
    and advantages, with the call's median time."""
    ro = s["ro"]
    G, M = s["G"], s["M"]
    n_groups = ro.n_rollouts // G
    cnt = torch.empty(9 + 6 * n_buckets, dtype=torch.int64, device=s["gate"].device)
    stream = torch.cuda.current_stream()
    ms = []
    for _ in range(reps + 1):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        L.leap_rollout_stats(s["pass_turn"], s["n_turns"], s["gate"], s["adv_roll"], n_groups, G, M,
                             n_buckets, cnt, s["err"])
        e1.record(stream)
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    out = stats_report(cnt.cpu().numpy(), n_buckets)
    out["call_us"] = float(np.median(ms[1:])) * 1e3
    out["n_buckets"] = n_buckets
    log(f"[bench] rollout stats: activated {out['activated_fraction']:.3f}, per-rollout recovery "
        f"{out['per_rollout_recovery']}, per-group recovery {out['per_group_recovery']}, "
        f"turns/pass {out['turns_per_pass']:.3f} ({out['call_us']:.1f} us)")
    return out


def lmhead_leg(L, torch, dev, seed: int, reps: int):
    """The fused LM-head variant on one 16384-row microbatch of the LM-head
    workload (hidden [16384 x 4096] ~ N(0,1), weight [151936 x 4096] ~
    N(0, 0.02^2), bf16): side arrays from the step's own rank and token
    advantages, forward + dhidden + dweight per call, HIP events around each
    call on the stream it runs on."""
    import workloads as wl
    lat = wl.draw_latent("lmhead")
    cfg = lat.cfg
    G, M, V, H, R = lat.G, lat.M, cfg["V"], cfg["H"], cfg["rows_per_mb"]
    tmin, tmax = L.leap_dcp_tau_from_pass_rate(G, 0, 1, 1, 3, 4, 1)
    ftp = torch.from_numpy(lat.first_turn_pass).to(dev)
    gate = torch.empty(lat.n_groups, dtype=torch.uint8, device=dev)
    L.leap_dcp_gate(ftp, lat.n_groups, G, tmin, tmax, None, gate)
    ro = wl.realize(lat, gate.cpu().numpy())
    mb = wl.pack(ro, R)[0]
    n = ro.n_rollouts
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    reward = torch.empty(n, dtype=torch.float32, device=dev)
    adv_roll = torch.empty(n, dtype=torch.float32, device=dev)
    L.leap_rank_advantages(torch.from_numpy(ro.pass_turn).to(dev), None, None, n // G, G, M,
                           L.LEAP_KEY_TURN, L.LEAP_ADV_STD, 1e-6, None, None, None, reward,
                           adv_roll, err)
    adv_tok = torch.empty(R, dtype=torch.float32, device=dev)
    w_tok = torch.empty(R, dtype=torch.float32, device=dev)
    L.leap_token_advantages(adv_roll, torch.from_numpy(mb.tok_rollout).to(dev),
                            torch.from_numpy(mb.tok_turn).to(dev),
                            torch.from_numpy(ro.n_turns).to(dev),
                            torch.from_numpy(ro.n_tokens).to(dev), n, R, cfg["gamma"],
                            L.LEAP_AGG_SEQ_MEAN_TOKEN_MEAN, float(n), adv_tok, w_tok, err)
    hid, wt = wl.lmhead_operands_device(seed, R, V, H, dev)
    y = wl.lmhead_tokens_device(hid, wt, seed)
    cur = _token_logp_torch(torch, hid, wt, y)
    n_old, n_ref = wl.logp_noise(seed, R)
    old = cur + torch.from_numpy(n_old.astype(np.float32)).to(dev)
    ref = cur + torch.from_numpy(n_ref.astype(np.float32)).to(dev)
    logp = torch.empty(R, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dH = torch.empty((R, H), dtype=torch.float32, device=dev)
    dW = torch.empty((V, H), dtype=torch.float32, device=dev)
    ws_bytes = L.leap_lmhead_workspace_size(R, V, H)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)

    wt_bytes = L.leap_lmhead_weight_t_size(V, H)
    w_t = torch.empty(wt_bytes, dtype=torch.uint8, device=dev)

    def call(prepared=False):
        L.leap_grpo_lmhead_fwd_bwd(hid, wt, R, V, H, y, old, ref, adv_tok, w_tok, p, logp, None,
                                   loss, dH, dW, 0, ws, ws_bytes, err,
                                   weight_t=w_t if prepared else None)

    def transpose():
        L.leap_lmhead_transpose_weight(wt, V, H, w_t, wt_bytes)

    probe = mfma_probe(L, torch, dev, 0)
    probe_rnd = mfma_probe(L, torch, dev, 1)
    log(f"[bench] MFMA probe: {probe / 1e12:.0f} TFLOP/s bf16 on ones, {probe_rnd / 1e12:.0f} on "
        f"random operands ({probe / MFMA_BF16_PEAK:.3f} and {probe_rnd / MFMA_BF16_PEAK:.3f} of "
        f"the 2.5 PFLOP/s spec)")
    stream = torch.cuda.current_stream()

    def timed(fn, n):
        settle(torch, fn)
        ms = []
        for _ in range(n):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return float(np.median(ms))

    # the call as a one-off (it transposes the weight itself), then with the
    # weight transposed beforehand, as the microbatches of one optimizer step
    # share it, and the transpose alone
    t = timed(call, reps) / 1e3
    assert int(err.item()) == 0, "data errors reported by the kernels"
    assert bool(torch.isfinite(loss).item())
    t_tr = timed(transpose, max(reps, 5)) / 1e3
    t_prep = timed(lambda: call(prepared=True), reps) / 1e3
    assert int(err.item()) == 0 and bool(torch.isfinite(loss).item())
    # The call drops the excluded rows (w = 0) before its GEMMs: useful work
    # is 6 H V flops per live row; executed work counts the compacted
    # extents (256-row tiles for the stats, dZ (at least one tile) and dH
    # passes, 64-row k-tiles for dW) and the vocabulary padded to 256.
    n_live = int((w_tok != 0).sum().item())
    v_pad = (V + 255) // 256 * 256
    m256 = (n_live + 255) // 256 * 256
    k64 = max(64, (n_live + 63) // 64 * 64)
    useful = 6.0 * n_live * H * V
    executed = 2.0 * H * v_pad * (2 * m256 + max(256, m256) + k64)
    log(f"[bench] lmhead {R}x{V}x{H} ({n_live} live rows): {t * 1e3:.2f} ms/call (median of "
        f"{reps}); {useful / t / 1e12:.0f} TFLOP/s useful, {executed / t / 1e12:.0f} executed; "
        f"with the weight transposed beforehand {t_prep * 1e3:.2f} ms (the transpose "
        f"{t_tr * 1e3:.3f} ms)")
    return {"workload": f"fused LM head, one microbatch: hidden [{R} x {H}] ~ N(0,1), weight "
                        f"[{V} x {H}] ~ N(0,0.02^2), bf16; forward, dhidden and dweight (fp32); "
                        f"{n_live} live rows (w != 0), the rest excluded",
            "ms_per_call": t * 1e3, "calls": reps, "rows_per_s": R / t, "live_rows": n_live,
            "ms_per_call_prepared_weight": t_prep * 1e3, "transpose_weight_ms": t_tr * 1e3,
            "frac_prepared_weight": useful / t_prep / MFMA_BF16_PEAK,
            "tokens_per_s": mb.n_valid / t, "generated_tokens": int(mb.n_valid),
            "roofline": {"bound": "mfma", "achieved": useful / t / 1e12,
                         "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s",
                         "frac": useful / t / MFMA_BF16_PEAK, "traffic": None,
                         "kernel": "one leap_grpo_lmhead_fwd_bwd call (4 GEMM passes over the live rows)",
                         "flops_per_call_useful": useful, "flops_per_call_executed": executed,
                         "executed_TFLOPs": executed / t / 1e12,
                         "executed_frac": executed / t / MFMA_BF16_PEAK,
                         "probe_ones_TFLOPs": probe / 1e12,
                         "probe_random_TFLOPs": probe_rnd / 1e12,
                         "executed_frac_of_probe_random": executed / t / probe_rnd},
            # the target for this path: half the bf16 matrix-core peak.  On executed flops
            # (the forward product formed twice, since the logits never reach HBM) that is
            # ~65 ms per 16384-row microbatch; on useful flops (6 n_live H V) it would need
            # 0.50 / 0.75 of peak executed, beyond the random-operand probe's power-limited rate
            "target": {"mfma_frac": 0.5,
                       "executed_frac": executed / t / MFMA_BF16_PEAK,
                       "met_on_executed_flops": executed / t / MFMA_BF16_PEAK >= 0.5,
                       "useful_frac": useful / t / MFMA_BF16_PEAK,
                       "met_on_useful_flops": useful / t / MFMA_BF16_PEAK >= 0.5}}


def mfma_probe(L, torch, dev, random_operands: int = 0, iters: int = 500000, reps: int = 3):
    """Achievable bf16 matrix-core rate of the device from the library's MFMA
    probe (register operands, no memory traffic; four waves per workgroup,
    four workgroups per compute unit), median of `reps` launches of about
    0.1 s each, after 100 ms of the same launches so the clock has settled.
    random_operands=0 multiplies ones (the least switching power);
    random_operands=1 hashed random bf16, which switch the multipliers'
    inputs as a GEMM over random data does: the rate the power limit leaves
    before any memory traffic, an upper bound for such a GEMM."""
    wgs = 4 * torch.cuda.get_device_properties(dev).multi_processor_count
    sink = torch.empty(wgs, dtype=torch.float32, device=dev)
    settle(torch, lambda: L.leap_probe_mfma(iters, wgs, sink, random_operands), ms=100)
    ts = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        L.leap_probe_mfma(iters, wgs, sink, random_operands)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / 1e3)
    if random_operands:
        assert bool(torch.isfinite(sink).all().item()), "MFMA probe gave a non-finite sum"
    else:
        assert bool((sink == iters * 32).all().item()), "MFMA probe did not run every round"
    flops = 4.0 * wgs * iters * 8 * 16384
    return flops / float(np.median(ts))


def blas_reference(torch, dev, rows: int = 16384):
    """Context only, not part of the path: torch's bf16 matmul (hipBLASLt) on
    the shapes of the fused LM head's four GEMM passes over `rows` rows (the
    call's live rows), as plain products with a bf16 result and no epilogue
    work.  Median of 3 timed calls."""
    shapes = {"stats (H W^T)": (rows, 151936, 4096), "dZ chunk": (rows, 32768, 4096),
              "dW chunk": (32768, 4096, rows), "dH chunk": (rows, 4096, 32768)}
    out = {}
    for name, (m, n, k) in shapes.items():
        a = torch.randn(m, k, device=dev, dtype=torch.bfloat16)
        b = torch.randn(n, k, device=dev, dtype=torch.bfloat16) * 0.02
        c = a @ b.t()
        torch.cuda.synchronize()
        ms = []
        for _ in range(3):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            c = a @ b.t()
            e1.record()
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        t = float(np.median(ms))
        out[name] = {"M": m, "N": n, "K": k, "ms": t, "TFLOPs": 2.0 * m * n * k / (t * 1e-3) / 1e12}
        log(f"[bench] torch bf16 matmul {name} {m}x{n}x{k}: {t:.3f} ms, {out[name]['TFLOPs']:.0f} TFLOP/s")
        del a, b, c
        torch.cuda.empty_cache()
    return out


def time_step(L, torch, s, steps: int, warmup: int) -> dict:
    """`warmup` untimed steps, then exactly `steps` timed steps between two
    device synchronisations (host clock), with HIP events on the launch
    stream around every fused call.  Rates use the step's algorithmic bytes
    (row_bytes per row of each microbatch)."""
    log(f"[bench] {s['name']}: warmup {warmup} steps")
    for _ in range(warmup):
        run_step(L, s)
    torch.cuda.synchronize()
    assert int(s["err"].item()) == 0, "data errors reported by the kernels"
    events = []
    log(f"[bench] {s['name']}: timing {steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run_step(L, s, events)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    V, R = s["V"], s["R"]
    k4_ms = np.array([a.elapsed_time(b) for a, b in events])
    mb_bytes = np.array([m.n_valid * row_bytes(V, True) + (R - m.n_valid) * row_bytes(V, False)
                         for m in s["mbs"]], np.float64)
    bytes_per_launch = float(mb_bytes.mean())
    k4_avg_s = float(k4_ms.mean()) / 1e3
    achieved = bytes_per_launch / k4_avg_s
    n_valid = int(s["valid"].sum())
    out = {"value": n_valid * steps / elapsed, "ms_per_step": elapsed / steps * 1e3,
           "k4_avg_s": k4_avg_s, "k4_median_us": float(np.median(k4_ms)) * 1e3,
           "achieved": achieved, "bytes_per_launch": bytes_per_launch,
           "step_bytes": float(mb_bytes.sum()), "n_valid": n_valid,
           "masked_row_fraction": 1.0 - n_valid / s["rows"]}
    log(f"[bench] {s['name']}: {out['ms_per_step']:.3f} ms/step; fused call {k4_avg_s * 1e6:.1f} us "
        f"avg over {len(k4_ms)} launches (median {out['k4_median_us']:.1f}); "
        f"{achieved / 1e9:.0f} GB/s algorithmic = {achieved / HBM_PEAK:.3f} of 8 TB/s")
    return out


def all_live_leg(L, torch, s, reps: int = 20):
    """The fused call on microbatch 0's logits with every row live (weight
    1/R, the microbatch's own advantages): the pure 1:1 read / write pattern,
    without the write-only masked rows of the real layout."""
    V, R = s["V"], s["R"]
    lg, dl = mb_logits(s, 0)
    w = torch.full((R,), 1.0 / R, dtype=torch.float32, device=lg.device)
    stream = torch.cuda.current_stream()

    def call():
        L.leap_grpo_logprob_loss_fwd_bwd(lg, V, R, V, s["tok"][:R], s["old"][:R], s["ref"][:R],
                                         s["adv_tok"][:R], w, s["params"], None, None, None,
                                         s["loss"][:1], dl, s["ws"], s["ws_bytes"], s["err"])

    settle(torch, call)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / reps / 1e3
    nbytes = R * row_bytes(V, True)
    log(f"[bench] fused call, every row live ({R} x {V}): {t * 1e6:.1f} us, "
        f"{nbytes / t / 1e9:.0f} GB/s = {nbytes / t / HBM_PEAK:.3f} of 8 TB/s")
    return {"workload": f"fused call on microbatch 0's logits ({R} x {V}), every row live",
            "call_us": t * 1e6, "GBps": nbytes / t / 1e9, "frac": nbytes / t / HBM_PEAK,
            "bytes_per_call": nbytes}


# Vocabulary widths of the width leg, with their row strides (odd widths on
# the 128-byte grid): the one-row kernels, the persistent row-queue range
# (55297-155648 columns) and the hybrid register + LDS rows.
WIDTHS = [(32768, 32768), (50257, 50304), (65536, 65536), (100000, 100000), (128256, 128256),
          (151936, 151936), (200003, 200064), (262144, 262144)]


def width_leg(L, torch, dev, reps: int = 20, R: int = 16384):
    """The fused call across vocabulary widths: 16384 rows of synthetic
    logits per width (bf16 N(0, 2^2), tokens sampled from them), every row
    live (weight 1/R), HIP events around `reps` back-to-back calls after a
    settling run; algorithmic bytes as in the headline (4V + 28 per row).
    The forward-only log-prob call on the same rows beside it (2V + 8 bytes
    per row)."""
    import workloads as wl
    out = []
    for V, ld in WIDTHS:
        lg = torch.empty((R, ld), dtype=torch.bfloat16, device=dev)
        wl.logits_device(4000 + V, R, V, ld=ld, device=dev, out=lg)
        tok = wl.sample_tokens_device(lg[:, :V], V, 4000 + V)
        dl = torch.empty_like(lg)
        cur = torch.empty(R, dtype=torch.float32, device=dev)
        L.leap_logprob_fwd(lg, ld, R, V, tok, None, 1.0, cur)
        rng = np.random.default_rng(V)
        old = cur + torch.from_numpy(rng.normal(0, 0.05, R).astype(np.float32)).to(dev)
        adv = torch.from_numpy(rng.normal(0, 1, R).astype(np.float32)).to(dev)
        w = torch.full((R,), 1.0 / R, dtype=torch.float32, device=dev)
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        ws_bytes = L.leap_grpo_workspace_size(R, V)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
        stream = torch.cuda.current_stream()

        def call():
            L.leap_grpo_logprob_loss_fwd_bwd(lg, ld, R, V, tok, old, cur, adv, w, p, None, None,
                                             None, loss, dl, ws, ws_bytes, None)

        def timed(fn):
            settle(torch, fn, 200)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps / 1e3

        t = timed(call)
        t_fwd = timed(lambda: L.leap_logprob_fwd(lg, ld, R, V, tok, None, 1.0, cur))
        nbytes = R * row_bytes(V, True)
        fwd_bytes = R * (2 * V + 8)
        log(f"[bench] width {V} (ld {ld}): {t * 1e6:.1f} us, {nbytes / t / 1e9:.0f} GB/s = "
            f"{nbytes / t / HBM_PEAK:.3f} of 8 TB/s; forward-only {t_fwd * 1e6:.1f} us = "
            f"{fwd_bytes / t_fwd / HBM_PEAK:.3f}")
        out.append({"V": V, "ld": ld, "call_us": t * 1e6, "GBps": nbytes / t / 1e9,
                    "frac": nbytes / t / HBM_PEAK, "logprob_fwd_us": t_fwd * 1e6,
                    "logprob_fwd_frac": fwd_bytes / t_fwd / HBM_PEAK})
        del lg, dl
        torch.cuda.empty_cache()
    return {"workload": f"fused call, {R} rows per width, every row live", "widths": out}


WORKLOAD_TEXT = {
    "full": "full: 64 prompts x G=16, up to 3 turns, U[512,4096] tokens/turn with U[64,512] "
            "masked feedback rows between turns, V={V}, {n_mb} microbatches x {R} rows "
            "(3 resident 16384-row logits buffers cycled through the step's per-microbatch "
            "side inputs)",
    "mid": "mid: 16 prompts x G=16, up to 2 turns, U[256,1024] tokens/turn with U[64,512] "
           "masked feedback rows between turns, V={V}, {n_mb} microbatches x {R} rows (every "
           "microbatch's logits resident)",
}
SEEDS = {"full": 1003, "mid": 1002}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # one full step is ~0.5 s of HBM traffic: 10 timed steps
    ap.add_argument("--steps", type=int, default=10)
    # ~3 s of the real step first: a fresh device settles its clocks over the
    # first seconds of sustained traffic
    ap.add_argument("--warmup", type=int, default=6)
    ap.add_argument("--workload", default="full", choices=["full", "mid"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lmhead-reps", type=int, default=5,
                    help="timed calls of the fused LM-head variant (0 skips it)")
    ap.add_argument("--no-shard", action="store_true", help="skip the vocabulary-shard leg")
    ap.add_argument("--no-widths", action="store_true",
                    help="skip the leg across vocabulary widths")
    ap.add_argument("--no-mid", action="store_true", help="skip the secondary mid-step leg")
    ap.add_argument("--no-legs", action="store_true",
                    help="only the headline step (for profiling its kernel)")
    ap.add_argument("--lmhead-only", action="store_true",
                    help="run only the fused LM-head leg and print its JSON object")
    ap.add_argument("--blas-reference", action="store_true",
                    help="with --lmhead-only: also time torch's bf16 matmul on the same GEMM "
                         "shapes (context for the GEMM core, not part of the path)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the LEAP hot path here is built and timed on a "
              "single MI355X; run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_01804_amd import leap as L
    L.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.lmhead_only:
        out = {"lmhead": lmhead_leg(L, torch, dev, 1005, max(1, args.lmhead_reps))}
        if args.blas_reference:
            out["blas_reference"] = blas_reference(torch, dev, out["lmhead"]["live_rows"])
        print(json.dumps(out), flush=True)
        return

    probe = hbm_probe(L, torch, dev)
    log("[bench] HBM probe: " + ", ".join(f"{k} {v:.0f}" for k, v in probe.items()))
    name = args.workload
    s = build_step(L, torch, dev, name, SEEDS[name], n_buffers=3 if name == "full" else None)
    copy_probe(torch, dev)
    m = time_step(L, torch, s, args.steps, args.warmup)
    V, R = s["V"], s["R"]

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        t = json.load(open(TRAFFIC_FILE))
        if t.get("k4_source_sha256_16") == k4_source_hash() and t.get("workload") == name:
            traffic = t.get("bytes_per_launch")

    legs = {}
    cpu = None
    if not args.no_legs:
        if not args.no_cpu_baseline:
            log(f"[bench] oracle on the host ({args.cpu_seconds:.0f} s sample)")
            cpu = cpu_baseline(s, args.cpu_seconds)
        legs["all_live"] = all_live_leg(L, torch, s)
        legs["widths"] = width_leg(L, torch, dev) if not args.no_widths else None
        legs["vocab_shard"] = shard_leg(L, torch, s) if not args.no_shard else None
        legs["logprob_fwd"] = logprob_leg(L, torch, s)
        legs["entropy"] = entropy_leg(L, torch, s)
        legs["small_kernels"] = small_leg(L, torch, s)
        legs["graph_replay"] = graph_leg(L, torch, s, max(2, args.steps // 2))
        legs["rollout_stats"] = stats_leg(L, torch, s)
    meta = {k: s[k] for k in ("n_mb", "rows", "G", "M")}
    del s
    torch.cuda.empty_cache()
    if not args.no_legs and not args.no_mid and name != "mid":
        sm = build_step(L, torch, dev, "mid", SEEDS["mid"])
        mm = time_step(L, torch, sm, 20, 30)
        legs["mid_step"] = {
            "workload": WORKLOAD_TEXT["mid"].format(V=sm["V"], n_mb=sm["n_mb"], R=sm["R"]),
            "value": mm["value"], "unit": "tokens/s", "ms_per_step": mm["ms_per_step"],
            "steps": 20, "warmup": 30, "generated_tokens_per_step": mm["n_valid"],
            "masked_row_fraction": mm["masked_row_fraction"],
            "fused_call_avg_us": mm["k4_avg_s"] * 1e6, "fused_call_median_us": mm["k4_median_us"],
            "achieved_GBps": mm["achieved"] / 1e9, "frac": mm["achieved"] / HBM_PEAK}
        del sm
        torch.cuda.empty_cache()
    lm = None
    if args.lmhead_reps > 0 and not args.no_legs:
        lm = lmhead_leg(L, torch, dev, 1005, args.lmhead_reps)

    out = {
        "metric": "rollout tokens/sec for fused GRPO logprob+loss+dlogits; % of HBM roofline",
        "value": m["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[name].format(V=V, n_mb=meta["n_mb"], R=R),
                   "generated_tokens_per_step": m["n_valid"], "rows_per_step": meta["rows"],
                   "masked_row_fraction": m["masked_row_fraction"],
                   "vocab": V, "microbatch_rows": R, "G": meta["G"], "max_turns": meta["M"]},
        "roofline": {"bound": "hbm", "achieved": m["achieved"] / 1e9, "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": m["achieved"] / HBM_PEAK, "traffic": traffic,
                     "kernel": "queue_reset + grpo_rows_persist<1024,19,16,false> + loss_reduce (one fused call)",
                     "avg_launch_us": m["k4_avg_s"] * 1e6, "median_launch_us": m["k4_median_us"],
                     "bytes_per_launch": m["bytes_per_launch"], "probe_GBps": probe,
                     "frac_of_probe_copy": m["achieved"] / 1e9 / probe["copy_GBps"]},
        "cpu_baseline": cpu,
        "lmhead": lm,
    }
    out.update(legs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
