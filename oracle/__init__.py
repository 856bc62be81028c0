"""fp64 CPU oracle for the LEAP GRPO hot path (arXiv 2608.01804).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP library in ``paper_2608_01804_amd`` and imports nothing from
it; the two meet only through the seeded input generators in ``workloads``.

The arithmetic lives in ``leap_oracle.c`` (plain C, double precision, OpenMP
over independent rows and groups only).  This module is argument marshalling
over ctypes with numpy arrays.  Functions and the passages they follow:

* ``rank_tournament``  -- Sec. 3.2, Eqs. 4-6 and the closing "standard GRPO"
  sentence (advantage read as (R - mean)/(unbiased std + eps)).
* ``dcp_gate``         -- Sec. 3.1, Eqs. 1-2.
* ``token_advantages`` -- Sec. 3.3 (discounted per-turn advantage) and the
  sample-level aggregation weight of Sec. 4.1 / Eq. 3.
* ``grpo_rows``        -- Sec. 3.1 Eq. 3 per token: log-softmax, ratio,
  clipped surrogate, reference KL, loss and dlogits.
* ``logprob_rows``     -- forward-only log-probabilities (old / reference).
* ``lmhead``           -- the same per-token objective on logits z = H W^T
  (fused LM head), with dH = dZ W and dW = dZ^T H.
* ``vocab_shard_stats`` -- one vocabulary shard's share of a row's
  log-softmax normaliser (max and base-2 sum) and of its token logit.
* ``rollout_stats``    -- the training statistics of the pruning study
  (activated groups, per-rollout / per-group recovery), turns per pass, and
  the pass-rate-bucketed advantage-sign composition of rollouts.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from fractions import Fraction

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "leap_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

KEY_TURN, KEY_LEX = 0, 1
ADV_STD, ADV_NONE = 0, 1
AGG_SEQ_MEAN_TOKEN_MEAN, AGG_TOKEN_MEAN, AGG_SUM = 0, 1, 2
KL_K3, KL_K1, KL_K2 = 0, 1, 2


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (no fast-math: IEEE double throughout).
    ``src`` / ``out`` default to this package's source and library; the
    mutation check of the test suite builds altered copies elsewhere."""
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
           "-fno-fast-math", "-Wall", "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.leap_oracle_set_threads.argtypes = [ctypes.c_int]
    lib.leap_oracle_get_threads.restype = ctypes.c_int
    lib.leap_oracle_rank_tournament.restype = i64
    lib.leap_oracle_rank_tournament.argtypes = [P, P, P, i64, i32, i32, i32, i32, f64,
                                                P, P, P, P, P]
    lib.leap_oracle_dcp_gate.restype = None
    lib.leap_oracle_dcp_gate.argtypes = [P, i64, i32, i32, i32, P, P]
    lib.leap_oracle_token_advantages.restype = i64
    lib.leap_oracle_token_advantages.argtypes = [P, P, P, P, P, i32, i64, f64, i32, f64, P, P]
    row_args = [P, i64, i64, i32, P, P, P, P, P, f64, f64, f64, i32, f64, i64, P, P, P, P, P]
    lib.leap_oracle_grpo_rows_f64.restype = i64
    lib.leap_oracle_grpo_rows_f64.argtypes = row_args
    lib.leap_oracle_grpo_rows_bf16.restype = i64
    lib.leap_oracle_grpo_rows_bf16.argtypes = row_args
    lib.leap_oracle_logprob_rows_bf16.restype = i64
    lib.leap_oracle_logprob_rows_bf16.argtypes = [P, i64, i64, i32, P, f64, P]
    lib.leap_oracle_entropy_rows_bf16.restype = i64
    lib.leap_oracle_entropy_rows_bf16.argtypes = [P, i64, i64, i32, f64, P]
    lib.leap_oracle_rollout_stats.restype = i64
    lib.leap_oracle_rollout_stats.argtypes = [P, P, P, P, i64, i32, i32, i32, P]
    _lib = lib
    return lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def set_threads(n: int) -> None:
    _load().leap_oracle_set_threads(int(n))


def get_threads() -> int:
    return int(_load().leap_oracle_get_threads())


def rank_tournament(pass_turn, G, M, key_mode=KEY_TURN, adv_norm=ADV_STD, eps=1e-6,
                    speedup_q=None, n_tokens=None):
    """Eqs. 4-6 + GRPO advantage.  Returns dict of r, n_worse, n_better, R, A, bad."""
    lib = _load()
    pt = _c(pass_turn, np.int32).reshape(-1)
    assert pt.size % G == 0
    n_groups = pt.size // G
    sq = _c(speedup_q, np.int32).reshape(-1) if speedup_q is not None else None
    nt = _c(n_tokens, np.int32).reshape(-1) if n_tokens is not None else None
    if key_mode == KEY_LEX:
        assert sq is not None and nt is not None
    r = np.empty(pt.size, np.int32)
    nw = np.empty(pt.size, np.int32)
    nb = np.empty(pt.size, np.int32)
    R = np.empty(pt.size, np.float64)
    A = np.empty(pt.size, np.float64)
    bad = lib.leap_oracle_rank_tournament(_p(pt), _p(sq), _p(nt), n_groups, G, M, key_mode,
                                          adv_norm, eps, _p(r), _p(nw), _p(nb), _p(R), _p(A))
    return {"r": r, "n_worse": nw, "n_better": nb, "R": R, "A": A, "bad": int(bad)}


def dcp_gate(first_turn_pass, G, tau_min, tau_max):
    """Eqs. 1-2.  Returns (n_fail int32[n_groups], gate uint8[n_groups])."""
    lib = _load()
    ftp = _c(first_turn_pass, np.uint8).reshape(-1)
    assert ftp.size % G == 0
    n_groups = ftp.size // G
    nf = np.empty(n_groups, np.int32)
    gate = np.empty(n_groups, np.uint8)
    lib.leap_oracle_dcp_gate(_p(ftp), n_groups, G, tau_min, tau_max, _p(nf), _p(gate))
    return nf, gate


def token_advantages(A, tok_rollout, tok_turn, n_turns, n_gen_tokens, gamma,
                     agg=AGG_SEQ_MEAN_TOKEN_MEAN, denom=1.0):
    """Sec. 3.3 + aggregation weight.  Returns (adv_tok f64, w_tok f64, bad)."""
    lib = _load()
    A = _c(A, np.float64)
    tr = _c(tok_rollout, np.int32)
    tt = _c(tok_turn, np.int32)
    nt = _c(n_turns, np.int32)
    ng = _c(n_gen_tokens, np.int32)
    N = tr.size
    adv = np.empty(N, np.float64)
    w = np.empty(N, np.float64)
    bad = lib.leap_oracle_token_advantages(_p(A), _p(tr), _p(tt), _p(nt), _p(ng), A.size, N,
                                           float(gamma), int(agg), float(denom), _p(adv), _p(w))
    return adv, w, int(bad)


def grpo_rows(logits, token_ids, old_logp, ref_logp, adv, w, V=None, eps_lo=0.2,
              eps_hi=0.2, kl_coef=0.01, kl_type=KL_K3, inv_temp=1.0, rows=None,
              want_dlogits=True):
    """Per-token objective and dlogits.

    ``logits`` is either a float64 array [N, ld] or a uint16 array of bf16 bit
    patterns [N, ld].  ``rows`` selects a subset (outputs follow its order).
    Returns dict: logp, tok_loss, loss (= sum w*loss over the selection),
    dlogits [n_sel, V] or None, bad.
    """
    lib = _load()
    lg = np.ascontiguousarray(logits)
    assert lg.ndim == 2
    N, ld = lg.shape
    V = ld if V is None else int(V)
    tok = _c(token_ids, np.int32)
    old = _c(old_logp, np.float64)
    ref = _c(ref_logp, np.float64)
    a = _c(adv, np.float64)
    ww = _c(w, np.float64)
    sel = None if rows is None else _c(rows, np.int64)
    n_sel = N if sel is None else sel.size
    logp = np.empty(n_sel, np.float64)
    tl = np.empty(n_sel, np.float64)
    dl = np.empty((n_sel, V), np.float64) if want_dlogits else None
    total = ctypes.c_double(0.0)
    if lg.dtype == np.uint16:
        fn = lib.leap_oracle_grpo_rows_bf16
    else:
        assert lg.dtype == np.float64
        fn = lib.leap_oracle_grpo_rows_f64
    bad = fn(_p(lg), ld, N, V, _p(tok), _p(old), _p(ref), _p(a), _p(ww), float(eps_lo),
             float(eps_hi), float(kl_coef), int(kl_type), float(inv_temp), n_sel, _p(sel),
             _p(logp), _p(tl), ctypes.byref(total), _p(dl))
    return {"logp": logp, "tok_loss": tl, "loss": total.value, "dlogits": dl, "bad": int(bad)}


def logprob_rows(logits_bf16, token_ids, V=None, inv_temp=1.0):
    """Forward-only log p(token) per row from bf16 logits [N, ld] (uint16)."""
    lib = _load()
    lg = np.ascontiguousarray(logits_bf16)
    assert lg.dtype == np.uint16 and lg.ndim == 2
    N, ld = lg.shape
    V = ld if V is None else int(V)
    tok = _c(token_ids, np.int32)
    out = np.empty(N, np.float64)
    bad = lib.leap_oracle_logprob_rows_bf16(_p(lg), ld, N, V, _p(tok), float(inv_temp), _p(out))
    return out, int(bad)


def entropy_rows(logits_bf16, V=None, inv_temp=1.0):
    """Shannon entropy (nats) of softmax(inv_temp * logits) per row, from bf16
    logits [N, ld] (uint16): H = -sum_v p_v log p_v.  All -inf rows give NaN
    and are counted in the second return value."""
    lib = _load()
    lg = np.ascontiguousarray(logits_bf16)
    assert lg.dtype == np.uint16 and lg.ndim == 2
    N, ld = lg.shape
    V = ld if V is None else int(V)
    out = np.empty(N, np.float64)
    bad = lib.leap_oracle_entropy_rows_bf16(_p(lg), ld, N, V, float(inv_temp), _p(out))
    return out, int(bad)


def _bf16_to_f64(a):
    """bf16 bit patterns (uint16) -> exact float64; float64 arrays pass through."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert a.dtype == np.float64
    return a


def lmhead(hidden, weight, token_ids, old_logp, ref_logp, adv, w, eps_lo=0.2, eps_hi=0.2,
           kl_coef=0.01, kl_type=KL_K3, inv_temp=1.0, rows=None, want_grads=True,
           v_block=8192):
    """Fused LM head: the per-token objective of ``grpo_rows`` (Sec. 3.1, Eq. 3
    per token) on logits z = H W^T, and its gradients.

    ``hidden`` [N, H] and ``weight`` [V, H] are float64 arrays or bf16 bit
    patterns (uint16, converted exactly).  Z = H W^T is a float64 matrix
    product (formed in blocks of ``v_block`` vocabulary rows); ``grpo_rows``
    on Z gives logp, tok_loss, loss and dZ = d(sum_k w_k loss_k)/dZ; then
    dH = dZ W and dW = dZ^T H.  ``rows`` evaluates only those rows (outputs in
    its order, loss summed over them, dH for them); dW sums over every row and
    is None then.  Returns dict: logp, tok_loss, loss, dZ, dH, dW, bad.
    """
    Hm = _bf16_to_f64(hidden)
    Wm = _bf16_to_f64(weight)
    assert Hm.ndim == 2 and Wm.ndim == 2 and Hm.shape[1] == Wm.shape[1]
    V = Wm.shape[0]
    sel = np.arange(Hm.shape[0]) if rows is None else np.asarray(rows, np.int64)
    Hs = Hm[sel]
    Z = np.empty((sel.size, V), np.float64)
    for v0 in range(0, V, v_block):
        Z[:, v0:v0 + v_block] = Hs @ Wm[v0:v0 + v_block].T
    pick = lambda a: np.asarray(a)[sel]  # noqa: E731
    r = grpo_rows(Z, pick(token_ids), pick(old_logp), pick(ref_logp), pick(adv), pick(w), V=V,
                  eps_lo=eps_lo, eps_hi=eps_hi, kl_coef=kl_coef, kl_type=kl_type,
                  inv_temp=inv_temp, want_dlogits=want_grads)
    dZ = dH = dW = None
    if want_grads:
        dZ = r["dlogits"]
        dH = np.zeros_like(Hs)
        for v0 in range(0, V, v_block):
            dH += dZ[:, v0:v0 + v_block] @ Wm[v0:v0 + v_block]
        if rows is None:
            dW = dZ.T @ Hm
    return {"logp": r["logp"], "tok_loss": r["tok_loss"], "loss": r["loss"], "dZ": dZ, "dH": dH,
            "dW": dW, "bad": r["bad"]}


def vocab_shard_stats(logits, vocab_start, token_ids, w=None, inv_temp=1.0, V=None):
    """One vocabulary shard's partial of the log-softmax of Sec. 3.1 (Eq. 3):
    for each row, with c = log2(e) * inv_temp over the shard's columns
    x[0..V-1] (global ids vocab_start + j): m2 = c * max_j x_j, s = sum_j
    2^(c x_j - m2); owned = 1 and zy = x[y - vocab_start] when the row's token
    y lies in the shard, else 0.  Rows with w == 0 (if w is given) are not
    read (m2 = -inf, s = 0, zy = 0; owned still reported); all -inf rows give
    m2 = -inf, s = 0.  ``logits`` is float64 or bf16 bit patterns
    [N, ld].  Returns float64 arrays (m2, s, zy, owned)."""
    x = _bf16_to_f64(logits)
    N, ld = x.shape
    V = ld if V is None else int(V)
    x = x[:, :V]
    c = np.log2(np.e) * float(inv_temp)
    yl = np.asarray(token_ids, np.int64) - int(vocab_start)
    owned = ((yl >= 0) & (yl < V)).astype(np.float64)
    m2 = np.full(N, -np.inf)
    s = np.zeros(N)
    zy = np.zeros(N)
    for k in range(N):
        if w is not None and w[k] == 0:
            continue  # an excluded row is not read: zy stays 0
        if owned[k]:
            zy[k] = x[k, yl[k]]
        mx = np.max(x[k])
        if mx == -np.inf:
            continue
        m2[k] = c * mx
        s[k] = np.sum(np.exp2(c * x[k] - m2[k]))
    return m2, s, zy, owned


STAT_FIELDS = ("groups", "rollouts", "activated_groups", "multi_turn_rollouts",
               "recovered_rollouts", "debugging_groups", "recovered_groups", "total_turns",
               "passed_rollouts")


def rollout_stats(pass_turn, n_turns, gate, G, M, advantage=None, n_buckets=10):
    """Counters of ``leap_oracle_rollout_stats`` as a dict (STAT_FIELDS, plus
    ``composition`` int64 [n_buckets, 3, 2]: outcome immediate / debug-assisted
    / failure x advantage sign positive / negative), the derived rates
    (activated fraction, per-rollout and per-group recovery, turns per pass;
    None where the denominator is 0) and ``bad``."""
    lib = _load()
    pt = _c(pass_turn, np.int32)
    nt = _c(n_turns, np.int32)
    gt = _c(gate, np.uint8)
    n_groups = gt.size
    adv = None if advantage is None else _c(advantage, np.float64)
    cnt = np.zeros(9 + n_buckets * 6, np.int64)
    bad = lib.leap_oracle_rollout_stats(_p(pt), _p(nt), _p(gt), _p(adv), n_groups, int(G),
                                        int(M), int(n_buckets), _p(cnt))
    out = {k: int(v) for k, v in zip(STAT_FIELDS, cnt[:9])}
    out["composition"] = cnt[9:].reshape(n_buckets, 3, 2)
    ratio = lambda a, b: (a / b) if b else None  # noqa: E731
    out["activated_fraction"] = ratio(out["activated_groups"], out["groups"])
    out["per_rollout_recovery"] = ratio(out["recovered_rollouts"], out["multi_turn_rollouts"])
    out["per_group_recovery"] = ratio(out["recovered_groups"], out["debugging_groups"])
    out["turns_per_pass"] = ratio(out["total_turns"], out["passed_rollouts"])
    out["bad"] = int(bad)
    return out


def tau_from_pass_rate(G: int, lo: Fraction, lo_strict: bool, hi: Fraction, hi_strict: bool):
    """Inclusive N_fail window of Eq. 2 selecting exactly the groups whose
    first-turn pass rate (G - N_fail)/G lies between lo and hi (each end open
    or closed), by exact rational enumeration of N_fail = 0..G.  Returns
    (tau_min, tau_max), or None if no N_fail qualifies."""
    ok = []
    for n in range(G + 1):
        q = Fraction(G - n, G)
        a = (q > lo) if lo_strict else (q >= lo)
        b = (q < hi) if hi_strict else (q <= hi)
        if a and b:
            ok.append(n)
    if not ok:
        return None
    return min(ok), max(ok)
