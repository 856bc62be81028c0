"""ctypes binding of libleap (declared in include/leap.h).

Argument marshalling only: every function has the name of its C entry point,
takes torch tensors (or raw device addresses as ints, or None for nullable
pointers), checks dtype / device / contiguity, passes ``data_ptr()`` and the
stream (default: torch's current stream), and raises :class:`LeapError` when
the library returns a status other than ``LEAP_OK``.  All computation runs in
the HIP kernels of libleap; there is no fallback of any kind -- importing a
function when libleap.so is missing raises.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libleap.so")

LEAP_OK = 0
LEAP_ERR_INVALID_ARG = 1
LEAP_ERR_MISALIGNED = 2
LEAP_ERR_WORKSPACE = 3
LEAP_ERR_UNSUPPORTED = 4
LEAP_ERR_HIP = 5

LEAP_KEY_TURN, LEAP_KEY_LEX = 0, 1
LEAP_ADV_STD, LEAP_ADV_NONE = 0, 1
LEAP_AGG_SEQ_MEAN_TOKEN_MEAN, LEAP_AGG_TOKEN_MEAN, LEAP_AGG_SUM = 0, 1, 2
LEAP_KL_K3, LEAP_KL_K1, LEAP_KL_K2 = 0, 1, 2

EXPORTED = (
    "leap_status_string",
    "leap_version",
    "leap_rank_advantages",
    "leap_dcp_gate",
    "leap_dcp_tau_from_pass_rate",
    "leap_token_advantages",
    "leap_grpo_workspace_size",
    "leap_grpo_logprob_loss_fwd_bwd",
    "leap_grpo_logprob_loss_fwd_bwd_noalloc",
    "leap_logprob_fwd",
    "leap_lmhead_workspace_size",
    "leap_lmhead_weight_t_size",
    "leap_lmhead_transpose_weight",
    "leap_grpo_lmhead_fwd_bwd",
    "leap_vocab_shard_stats",
    "leap_vocab_merge_workspace_size",
    "leap_vocab_merge_objective",
    "leap_vocab_shard_bwd",
    "leap_rollout_stats",
    "leap_probe_hbm",
    "leap_probe_mfma",
)


class LeapError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = int(status)
        super().__init__(f"{where}: {_status_name(status)} ({status})")


class leap_grpo_params(ctypes.Structure):
    _fields_ = [
        ("clip_eps_low", ctypes.c_float),
        ("clip_eps_high", ctypes.c_float),
        ("kl_coef", ctypes.c_float),
        ("kl_type", ctypes.c_int32),
        ("inv_temperature", ctypes.c_float),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libleap.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libleap.so not built at {LIB_PATH}; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f32, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                             ctypes.c_double)
    L.leap_status_string.restype = ctypes.c_char_p
    L.leap_status_string.argtypes = [ctypes.c_int]
    L.leap_version.restype = ctypes.c_char_p
    L.leap_version.argtypes = []
    L.leap_rank_advantages.restype = ctypes.c_int
    L.leap_rank_advantages.argtypes = [P, P, P, i64, i32, i32, i32, i32, f32, P, P, P, P, P, P, P]
    L.leap_dcp_gate.restype = ctypes.c_int
    L.leap_dcp_gate.argtypes = [P, i64, i32, i32, i32, P, P, P]
    L.leap_dcp_tau_from_pass_rate.restype = ctypes.c_int
    L.leap_dcp_tau_from_pass_rate.argtypes = [i32, i32, i32, i32, i32, i32, i32,
                                              ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.leap_token_advantages.restype = ctypes.c_int
    L.leap_token_advantages.argtypes = [P, P, P, P, P, i32, i64, f32, i32, f64, P, P, P, P]
    L.leap_grpo_workspace_size.restype = ctypes.c_size_t
    L.leap_grpo_workspace_size.argtypes = [i64, i32]
    L.leap_grpo_logprob_loss_fwd_bwd.restype = ctypes.c_int
    L.leap_grpo_logprob_loss_fwd_bwd.argtypes = [P, i64, i64, i32, P, P, P, P, P,
                                                 ctypes.POINTER(leap_grpo_params), P, P, P, P,
                                                 P, P, ctypes.c_size_t, P, P]
    L.leap_grpo_logprob_loss_fwd_bwd_noalloc.restype = ctypes.c_int
    L.leap_grpo_logprob_loss_fwd_bwd_noalloc.argtypes = [P, i64, i64, i32, P, P, P, P, P,
                                                         ctypes.POINTER(leap_grpo_params), P, P,
                                                         P, P, P, P, P]
    L.leap_logprob_fwd.restype = ctypes.c_int
    L.leap_logprob_fwd.argtypes = [P, i64, i64, i32, P, P, f32, P, P, P, P]
    L.leap_lmhead_workspace_size.restype = ctypes.c_size_t
    L.leap_lmhead_workspace_size.argtypes = [i64, i32, i32]
    L.leap_lmhead_weight_t_size.restype = ctypes.c_size_t
    L.leap_lmhead_weight_t_size.argtypes = [i32, i32]
    L.leap_lmhead_transpose_weight.restype = ctypes.c_int
    L.leap_lmhead_transpose_weight.argtypes = [P, i32, i32, P, ctypes.c_size_t, P]
    L.leap_grpo_lmhead_fwd_bwd.restype = ctypes.c_int
    L.leap_grpo_lmhead_fwd_bwd.argtypes = [P, P, P, i64, i32, i32, P, P, P, P, P,
                                           ctypes.POINTER(leap_grpo_params), P, P, P, P, P, i32,
                                           P, ctypes.c_size_t, P, P]
    L.leap_vocab_shard_stats.restype = ctypes.c_int
    L.leap_vocab_shard_stats.argtypes = [P, i64, i64, i32, i32, P, P, f32, P, P, P]
    L.leap_vocab_merge_workspace_size.restype = ctypes.c_size_t
    L.leap_vocab_merge_workspace_size.argtypes = [i64]
    L.leap_vocab_merge_objective.restype = ctypes.c_int
    L.leap_vocab_merge_objective.argtypes = [P, P, i32, i64, i32, P, P, P, P, P,
                                             ctypes.POINTER(leap_grpo_params), P, P, P, P, P, P,
                                             ctypes.c_size_t, P, P]
    L.leap_vocab_shard_bwd.restype = ctypes.c_int
    L.leap_vocab_shard_bwd.argtypes = [P, i64, i64, i32, i32, P, P, f32, P, P]
    L.leap_rollout_stats.restype = ctypes.c_int
    L.leap_rollout_stats.argtypes = [P, P, P, P, i64, i32, i32, i32, P, P, P]
    L.leap_probe_mfma.restype = ctypes.c_int
    L.leap_probe_mfma.argtypes = [i64, i32, i32, P, P]
    L.leap_probe_hbm.restype = ctypes.c_int
    L.leap_probe_hbm.argtypes = [P, P, ctypes.c_size_t, i32, P]
    _lib = L
    return L


def _status_name(s: int) -> str:
    try:
        return lib().leap_status_string(int(s)).decode()
    except Exception:  # noqa: BLE001 - only used to format an error message
        return "LEAP_ERR"


def _check(status: int, where: str) -> None:
    if status != LEAP_OK:
        raise LeapError(status, where)


_DTYPES = {}


def _ptr(x, dtype_name: str | None = None, name: str = "arg"):
    """Device address of a tensor (dtype/device/contiguity checked), an int, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    import torch
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, an int address or None")
    if dtype_name is not None:
        want = getattr(torch, dtype_name)
        if x.dtype != want:
            raise TypeError(f"{name}: expected dtype {want}, got {x.dtype}")
    if x.device.type != "cuda":
        raise ValueError(f"{name}: expected a device tensor, got {x.device}")
    if not x.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def leap_version() -> str:
    return lib().leap_version().decode()


def leap_status_string(status: int) -> str:
    return lib().leap_status_string(int(status)).decode()


def leap_rank_advantages(pass_turn, speedup_q, n_tokens, n_groups, G, M, key, norm, eps,
                         n_worse, n_better, rank_r, reward, advantage, dev_err=None,
                         stream=None) -> None:
    st = lib().leap_rank_advantages(
        _ptr(pass_turn, "int32", "pass_turn"), _ptr(speedup_q, "int32", "speedup_q"),
        _ptr(n_tokens, "int32", "n_tokens"), int(n_groups), int(G), int(M), int(key), int(norm),
        float(eps), _ptr(n_worse, "int32", "n_worse"), _ptr(n_better, "int32", "n_better"),
        _ptr(rank_r, "int32", "rank_r"), _ptr(reward, "float32", "reward"),
        _ptr(advantage, "float32", "advantage"), _ptr(dev_err, "int32", "dev_err"),
        _stream(stream))
    _check(st, "leap_rank_advantages")


def leap_dcp_gate(first_turn_pass, n_groups, G, tau_min, tau_max, n_fail, gate,
                  stream=None) -> None:
    st = lib().leap_dcp_gate(_ptr(first_turn_pass, "uint8", "first_turn_pass"), int(n_groups),
                             int(G), int(tau_min), int(tau_max), _ptr(n_fail, "int32", "n_fail"),
                             _ptr(gate, "uint8", "gate"), _stream(stream))
    _check(st, "leap_dcp_gate")


def leap_dcp_tau_from_pass_rate(G, lo_num, lo_den, lo_strict, hi_num, hi_den, hi_strict):
    """Returns (tau_min, tau_max)."""
    a, b = ctypes.c_int32(0), ctypes.c_int32(0)
    st = lib().leap_dcp_tau_from_pass_rate(int(G), int(lo_num), int(lo_den), int(lo_strict),
                                           int(hi_num), int(hi_den), int(hi_strict),
                                           ctypes.byref(a), ctypes.byref(b))
    _check(st, "leap_dcp_tau_from_pass_rate")
    return int(a.value), int(b.value)


def leap_token_advantages(advantage, tok_rollout, tok_turn, n_turns, n_gen_tokens, n_rollouts, N,
                          gamma, agg, denominator, adv_tok, w_tok, dev_err=None,
                          stream=None) -> None:
    st = lib().leap_token_advantages(
        _ptr(advantage, "float32", "advantage"), _ptr(tok_rollout, "int32", "tok_rollout"),
        _ptr(tok_turn, "int32", "tok_turn"), _ptr(n_turns, "int32", "n_turns"),
        _ptr(n_gen_tokens, "int32", "n_gen_tokens"), int(n_rollouts), int(N), float(gamma),
        int(agg), float(denominator), _ptr(adv_tok, "float32", "adv_tok"),
        _ptr(w_tok, "float32", "w_tok"), _ptr(dev_err, "int32", "dev_err"), _stream(stream))
    _check(st, "leap_token_advantages")


def leap_grpo_workspace_size(N, V) -> int:
    return int(lib().leap_grpo_workspace_size(int(N), int(V)))


def leap_grpo_logprob_loss_fwd_bwd(logits, ld, N, V, token_ids, old_logp, ref_logp, adv_tok, w_tok,
                                   params: leap_grpo_params, logp_out, tok_loss_out, entropy_out,
                                   loss_out, dlogits, workspace, ws_bytes, dev_err=None,
                                   stream=None) -> None:
    st = lib().leap_grpo_logprob_loss_fwd_bwd(
        _ptr(logits, "bfloat16", "logits"), int(ld), int(N), int(V),
        _ptr(token_ids, "int32", "token_ids"), _ptr(old_logp, "float32", "old_logp"),
        _ptr(ref_logp, "float32", "ref_logp"), _ptr(adv_tok, "float32", "adv_tok"),
        _ptr(w_tok, "float32", "w_tok"), ctypes.byref(params) if params is not None else None,
        _ptr(logp_out, "float32", "logp_out"), _ptr(tok_loss_out, "float32", "tok_loss_out"),
        _ptr(entropy_out, "float32", "entropy_out"), _ptr(loss_out, "float32", "loss_out"), _ptr(dlogits, "bfloat16", "dlogits"),
        _ptr(workspace, None, "workspace"), int(ws_bytes), _ptr(dev_err, "int32", "dev_err"),
        _stream(stream))
    _check(st, "leap_grpo_logprob_loss_fwd_bwd")


LEAP_NOALLOC_MAX_ROWS = 1048576
LEAP_MAX_V = 268435456


def leap_grpo_logprob_loss_fwd_bwd_noalloc(logits, ld, N, V, token_ids, old_logp, ref_logp,
                                           adv_tok, w_tok, params: leap_grpo_params, logp_out,
                                           tok_loss_out, entropy_out, loss_out, dlogits,
                                           dev_err=None, stream=None) -> None:
    st = lib().leap_grpo_logprob_loss_fwd_bwd_noalloc(
        _ptr(logits, "bfloat16", "logits"), int(ld), int(N), int(V),
        _ptr(token_ids, "int32", "token_ids"), _ptr(old_logp, "float32", "old_logp"),
        _ptr(ref_logp, "float32", "ref_logp"), _ptr(adv_tok, "float32", "adv_tok"),
        _ptr(w_tok, "float32", "w_tok"), ctypes.byref(params) if params is not None else None,
        _ptr(logp_out, "float32", "logp_out"), _ptr(tok_loss_out, "float32", "tok_loss_out"),
        _ptr(entropy_out, "float32", "entropy_out"), _ptr(loss_out, "float32", "loss_out"),
        _ptr(dlogits, "bfloat16", "dlogits"), _ptr(dev_err, "int32", "dev_err"),
        _stream(stream))
    _check(st, "leap_grpo_logprob_loss_fwd_bwd_noalloc")


def leap_logprob_fwd(logits, ld, N, V, token_ids, w_tok, inv_temperature, logp_out,
                     entropy_out=None, dev_err=None, stream=None) -> None:
    st = lib().leap_logprob_fwd(
        _ptr(logits, "bfloat16", "logits"), int(ld), int(N), int(V),
        _ptr(token_ids, "int32", "token_ids"), _ptr(w_tok, "float32", "w_tok"),
        float(inv_temperature), _ptr(logp_out, "float32", "logp_out"),
        _ptr(entropy_out, "float32", "entropy_out"), _ptr(dev_err, "int32", "dev_err"),
        _stream(stream))
    _check(st, "leap_logprob_fwd")


def leap_lmhead_workspace_size(N, V, H) -> int:
    return int(lib().leap_lmhead_workspace_size(int(N), int(V), int(H)))


def leap_lmhead_weight_t_size(V, H) -> int:
    return int(lib().leap_lmhead_weight_t_size(int(V), int(H)))


def leap_lmhead_transpose_weight(weight, V, H, weight_t, nbytes, stream=None) -> None:
    st = lib().leap_lmhead_transpose_weight(_ptr(weight, "bfloat16", "weight"), int(V), int(H),
                                            _ptr(weight_t, None, "weight_t"), int(nbytes),
                                            _stream(stream))
    _check(st, "leap_lmhead_transpose_weight")


def leap_grpo_lmhead_fwd_bwd(hidden, weight, N, V, H, token_ids, old_logp, ref_logp, adv_tok, w_tok,
                             params: leap_grpo_params, logp_out, tok_loss_out, loss_out, dhidden,
                             dweight, accumulate_dweight, workspace, ws_bytes, dev_err=None,
                             stream=None, weight_t=None) -> None:
    st = lib().leap_grpo_lmhead_fwd_bwd(
        _ptr(hidden, "bfloat16", "hidden"), _ptr(weight, "bfloat16", "weight"),
        _ptr(weight_t, None, "weight_t"), int(N), int(V), int(H), _ptr(token_ids, "int32", "token_ids"), _ptr(old_logp, "float32", "old_logp"),
        _ptr(ref_logp, "float32", "ref_logp"), _ptr(adv_tok, "float32", "adv_tok"),
        _ptr(w_tok, "float32", "w_tok"), ctypes.byref(params) if params is not None else None,
        _ptr(logp_out, "float32", "logp_out"), _ptr(tok_loss_out, "float32", "tok_loss_out"),
        _ptr(loss_out, "float32", "loss_out"), _ptr(dhidden, "float32", "dhidden"),
        _ptr(dweight, "float32", "dweight"), int(accumulate_dweight),
        _ptr(workspace, None, "workspace"), int(ws_bytes), _ptr(dev_err, "int32", "dev_err"),
        _stream(stream))
    _check(st, "leap_grpo_lmhead_fwd_bwd")


def leap_vocab_shard_stats(logits, ld, N, V_shard, vocab_start, token_ids, w_tok, inv_temperature,
                           partial, stream=None, partial_t=None) -> None:
    st = lib().leap_vocab_shard_stats(
        _ptr(logits, "bfloat16", "logits"), int(ld), int(N), int(V_shard), int(vocab_start),
        _ptr(token_ids, "int32", "token_ids"), _ptr(w_tok, "float32", "w_tok"),
        float(inv_temperature), _ptr(partial, "float32", "partial"),
        _ptr(partial_t, "float32", "partial_t"), _stream(stream))
    _check(st, "leap_vocab_shard_stats")


def leap_vocab_merge_workspace_size(N) -> int:
    return int(lib().leap_vocab_merge_workspace_size(int(N)))


def leap_vocab_merge_objective(partials, n_shards, N, V_total, token_ids, old_logp, ref_logp,
                               adv_tok, w_tok, params: leap_grpo_params, logp_out, tok_loss_out,
                               loss_out, row_state, workspace, ws_bytes, dev_err=None,
                               stream=None, partials_t=None, entropy_out=None) -> None:
    st = lib().leap_vocab_merge_objective(
        _ptr(partials, "float32", "partials"), _ptr(partials_t, "float32", "partials_t"),
        int(n_shards), int(N), int(V_total),
        _ptr(token_ids, "int32", "token_ids"), _ptr(old_logp, "float32", "old_logp"),
        _ptr(ref_logp, "float32", "ref_logp"), _ptr(adv_tok, "float32", "adv_tok"),
        _ptr(w_tok, "float32", "w_tok"), ctypes.byref(params) if params is not None else None,
        _ptr(logp_out, "float32", "logp_out"), _ptr(tok_loss_out, "float32", "tok_loss_out"),
        _ptr(entropy_out, "float32", "entropy_out"), _ptr(loss_out, "float32", "loss_out"),
        _ptr(row_state, "float32", "row_state"),
        _ptr(workspace, None, "workspace"), int(ws_bytes), _ptr(dev_err, "int32", "dev_err"),
        _stream(stream))
    _check(st, "leap_vocab_merge_objective")


def leap_vocab_shard_bwd(logits, ld, N, V_shard, vocab_start, token_ids, row_state,
                         inv_temperature, dlogits, stream=None) -> None:
    st = lib().leap_vocab_shard_bwd(
        _ptr(logits, "bfloat16", "logits"), int(ld), int(N), int(V_shard), int(vocab_start),
        _ptr(token_ids, "int32", "token_ids"), _ptr(row_state, "float32", "row_state"),
        float(inv_temperature), _ptr(dlogits, "bfloat16", "dlogits"), _stream(stream))
    _check(st, "leap_vocab_shard_bwd")


def leap_rollout_stats(pass_turn, n_turns, gate, advantage, n_groups, G, M, n_buckets, counters,
                       dev_err=None, stream=None) -> None:
    st = lib().leap_rollout_stats(
        _ptr(pass_turn, "int32", "pass_turn"), _ptr(n_turns, "int32", "n_turns"),
        _ptr(gate, "uint8", "gate"), _ptr(advantage, "float32", "advantage"), int(n_groups),
        int(G), int(M), int(n_buckets), _ptr(counters, "int64", "counters"),
        _ptr(dev_err, "int32", "dev_err"), _stream(stream))
    _check(st, "leap_rollout_stats")


def leap_probe_hbm(src, dst, nbytes, mode, stream=None) -> None:
    st = lib().leap_probe_hbm(_ptr(src, None, "src"), _ptr(dst, None, "dst"), int(nbytes),
                              int(mode), _stream(stream))
    _check(st, "leap_probe_hbm")


def leap_probe_mfma(iters, n_workgroups, sink, random_operands=0, stream=None) -> None:
    st = lib().leap_probe_mfma(int(iters), int(n_workgroups), int(random_operands),
                               _ptr(sink, "float32", "sink"), _stream(stream))
    _check(st, "leap_probe_mfma")
