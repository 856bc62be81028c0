"""The C-ABI library loads, exports every entry point include/leap.h declares,
and rejects bad arguments on the host (no kernel is launched: every call here
returns before any device work, so no GPU is needed)."""
import ctypes
import os
import re
import subprocess
from fractions import Fraction

import pytest

import oracle
from paper_2608_01804_amd import leap as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "leap.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(leap_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert _declared() == sorted(L.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = L.lib()
    for name in _declared():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", L.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (leap_[a-z0-9_]+)", out))
    assert set(_declared()) <= exported
    # nothing else leaks from the library
    assert exported == set(_declared())


C_CALLER = r"""
#include <stdio.h>
#include "leap.h"
int main(void) {
    int32_t lo = -1, hi = -1;
    leap_status st = leap_dcp_tau_from_pass_rate(16, 0, 1, 1, 3, 4, 1, &lo, &hi);
    printf("%s %s %d %d\n", leap_version(), leap_status_string(st), (int)lo, (int)hi);
    printf("%zu %zu\n", leap_grpo_workspace_size(16384, 151936),
           leap_vocab_merge_workspace_size(16384));
    return st == LEAP_OK ? 0 : 1;
}
"""


def test_header_compiles_as_c99_and_links(tmp_path):
    """A C99 caller (strict warnings on everything but the ROCm headers)
    includes leap.h, links libleap.so and calls its host-only entry points.
    Only against the product build: a sanitizer-instrumented copy needs its
    runtime at link time."""
    from paper_2608_01804_amd import _build
    if os.path.realpath(L.LIB_PATH) != os.path.realpath(_build.LIB_PATH):
        pytest.skip("the binding points at another build of the library")
    src = tmp_path / "caller.c"
    src.write_text(C_CALLER)
    exe = tmp_path / "caller"
    pkg = os.path.dirname(L.LIB_PATH)
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
                    "-isystem", os.path.join(rocm, "include"), str(src), "-L" + pkg, "-lleap",
                    "-Wl,-rpath," + pkg, "-o", str(exe)], check=True, capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()
    tmin, tmax = L.leap_dcp_tau_from_pass_rate(16, 0, 1, 1, 3, 4, 1)
    assert out[:4] == [L.leap_version(), "LEAP_OK", str(tmin), str(tmax)]
    assert int(out[4]) == L.leap_grpo_workspace_size(16384, 151936)
    assert int(out[5]) == L.leap_vocab_merge_workspace_size(16384)


def test_status_strings_and_version():
    assert L.leap_status_string(0) == "LEAP_OK"
    assert L.leap_status_string(3) == "LEAP_ERR_WORKSPACE"
    assert re.fullmatch(r"\d+\.\d+\.\d+", L.leap_version())


FAKE = 0x1000  # never dereferenced: every call below fails validation first


def _rank(**kw):
    a = dict(pass_turn=FAKE, speedup_q=None, n_tokens=None, n_groups=4, G=8, M=2,
             key=L.LEAP_KEY_TURN, norm=L.LEAP_ADV_STD, eps=1e-6, n_worse=None, n_better=None,
             rank_r=None, reward=FAKE, advantage=FAKE, dev_err=None, stream=0)
    a.update(kw)
    return L.leap_rank_advantages(**a)


@pytest.mark.parametrize("kw", [dict(G=1), dict(G=1025), dict(M=0), dict(n_groups=-1),
                                dict(eps=-1.0), dict(eps=float("nan")), dict(key=7),
                                dict(norm=9), dict(pass_turn=None), dict(reward=None),
                                dict(advantage=None), dict(key=L.LEAP_KEY_LEX)])
def test_rank_advantages_rejects(kw):
    with pytest.raises(L.LeapError) as e:
        _rank(**kw)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG


def test_empty_calls_are_ok_without_device_work():
    _rank(n_groups=0, pass_turn=None, reward=None, advantage=None)
    L.leap_dcp_gate(None, 0, 8, 0, 8, None, None, stream=0)
    L.leap_token_advantages(None, None, None, None, None, 0, 0, 0.9, L.LEAP_AGG_SUM, 1.0, None,
                            None, stream=0)


@pytest.mark.parametrize("args", [(0, 8), (4, 0), (4, 1025)])
def test_gate_rejects_sizes(args):
    n_groups, G = args
    with pytest.raises(L.LeapError):
        L.leap_dcp_gate(FAKE, n_groups, G, 0, 0, None, FAKE, stream=0) if n_groups else \
            L.leap_dcp_gate(FAKE, -1, G, 0, 0, None, FAKE, stream=0)


@pytest.mark.parametrize("tau", [(-1, 4), (5, 4), (0, 9)])
def test_gate_rejects_tau(tau):
    with pytest.raises(L.LeapError) as e:
        L.leap_dcp_gate(FAKE, 4, 8, tau[0], tau[1], None, FAKE, stream=0)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG


@pytest.mark.parametrize("G", [1, 2, 3, 5, 8, 16, 17, 64, 100, 1024])
@pytest.mark.parametrize("window", [
    (Fraction(0), True, Fraction(3, 4), True),
    (Fraction(0), False, Fraction(1, 2), False),
    (Fraction(1, 2), False, Fraction(1), False),
    (Fraction(1, 3), True, Fraction(2, 3), False),
    (Fraction(0), False, Fraction(1), False),
])
def test_tau_helper_matches_oracle_enumeration(G, window):
    lo, lo_s, hi, hi_s = window
    want = oracle.tau_from_pass_rate(G, lo, lo_s, hi, hi_s)
    if want is None:
        with pytest.raises(L.LeapError):
            L.leap_dcp_tau_from_pass_rate(G, lo.numerator, lo.denominator, int(lo_s),
                                          hi.numerator, hi.denominator, int(hi_s))
    else:
        got = L.leap_dcp_tau_from_pass_rate(G, lo.numerator, lo.denominator, int(lo_s),
                                            hi.numerator, hi.denominator, int(hi_s))
        assert got == want


def test_tau_helper_rejects_empty_window():
    with pytest.raises(L.LeapError):
        L.leap_dcp_tau_from_pass_rate(8, 1, 2, 1, 1, 2, 1)  # 1/2 < q < 1/2


@pytest.mark.parametrize("kw", [dict(N=-1), dict(gamma=0.0), dict(gamma=1.5), dict(agg=5),
                                dict(denominator=0.0), dict(tok_rollout=None), dict(adv_tok=None)])
def test_token_advantages_rejects(kw):
    a = dict(advantage=FAKE, tok_rollout=FAKE, tok_turn=FAKE, n_turns=FAKE, n_gen_tokens=FAKE,
             n_rollouts=4, N=16, gamma=0.9, agg=L.LEAP_AGG_SEQ_MEAN_TOKEN_MEAN, denominator=4.0,
             adv_tok=FAKE, w_tok=FAKE, dev_err=None, stream=0)
    a.update(kw)
    with pytest.raises(L.LeapError) as e:
        L.leap_token_advantages(**a)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG


def _grpo(**kw):
    p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
    a = dict(logits=FAKE, ld=1024, N=8, V=1000, token_ids=FAKE, old_logp=FAKE, ref_logp=FAKE,
             adv_tok=FAKE, w_tok=FAKE, params=p, logp_out=None, tok_loss_out=None, entropy_out=None,
             loss_out=FAKE,
             dlogits=FAKE + (1 << 30), workspace=FAKE, ws_bytes=1 << 20, dev_err=None, stream=0)
    a.update(kw)
    return L.leap_grpo_logprob_loss_fwd_bwd(**a)


@pytest.mark.parametrize("kw,status", [
    (dict(N=-1), L.LEAP_ERR_INVALID_ARG),
    (dict(V=0), L.LEAP_ERR_INVALID_ARG),
    (dict(ld=999), L.LEAP_ERR_INVALID_ARG),
    (dict(loss_out=None), L.LEAP_ERR_INVALID_ARG),
    (dict(params=None), L.LEAP_ERR_INVALID_ARG),
    (dict(token_ids=None), L.LEAP_ERR_INVALID_ARG),
    (dict(logits=FAKE + 2), L.LEAP_ERR_MISALIGNED),
    (dict(ld=1004), L.LEAP_ERR_MISALIGNED),
    (dict(workspace=None), L.LEAP_ERR_WORKSPACE),
    (dict(ws_bytes=16), L.LEAP_ERR_WORKSPACE),
    (dict(dlogits=FAKE + 2048), L.LEAP_ERR_INVALID_ARG),  # partial overlap with logits
    (dict(V=L.LEAP_MAX_V + 1, ld=L.LEAP_MAX_V + 8), L.LEAP_ERR_UNSUPPORTED),
    (dict(V=L.LEAP_MAX_V + 1, ld=L.LEAP_MAX_V + 8, N=0), L.LEAP_ERR_UNSUPPORTED),
])
def test_grpo_rejects(kw, status):
    with pytest.raises(L.LeapError) as e:
        _grpo(**kw)
    assert e.value.status == status


@pytest.mark.parametrize("kw,status", [
    (dict(N=L.LEAP_NOALLOC_MAX_ROWS + 1), L.LEAP_ERR_UNSUPPORTED),
    (dict(N=-1), L.LEAP_ERR_INVALID_ARG),
    (dict(loss_out=None), L.LEAP_ERR_INVALID_ARG),
    (dict(logits=FAKE + 2), L.LEAP_ERR_MISALIGNED),
    (dict(dlogits=FAKE + 2048), L.LEAP_ERR_INVALID_ARG),
    (dict(V=L.LEAP_MAX_V + 1, ld=L.LEAP_MAX_V + 8), L.LEAP_ERR_UNSUPPORTED),
])
def test_grpo_noalloc_rejects(kw, status):
    """The no-allocation form checks its arguments like the workspace form
    and refuses more rows than its device array holds, all on the host."""
    p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
    a = dict(logits=FAKE, ld=1024, N=8, V=1000, token_ids=FAKE, old_logp=FAKE, ref_logp=FAKE,
             adv_tok=FAKE, w_tok=FAKE, params=p, logp_out=None, tok_loss_out=None,
             entropy_out=None, loss_out=FAKE, dlogits=FAKE + (1 << 40), dev_err=None, stream=0)
    a.update(kw)
    with pytest.raises(L.LeapError) as e:
        L.leap_grpo_logprob_loss_fwd_bwd_noalloc(**a)
    assert e.value.status == status


@pytest.mark.parametrize("field,value,status", [
    ("clip_eps_low", -0.1, L.LEAP_ERR_INVALID_ARG),
    ("kl_coef", float("inf"), L.LEAP_ERR_INVALID_ARG),
    ("inv_temperature", 0.0, L.LEAP_ERR_INVALID_ARG),
    ("kl_type", 7, L.LEAP_ERR_UNSUPPORTED),
])
def test_grpo_rejects_params(field, value, status):
    p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
    setattr(p, field, value)
    with pytest.raises(L.LeapError) as e:
        _grpo(params=p)
    assert e.value.status == status


def test_workspace_size():
    assert L.leap_grpo_workspace_size(16384, 151936) >= 16384 * 4
    assert L.leap_grpo_workspace_size(0, 10) > 0
    assert L.leap_grpo_workspace_size(1000, 10) % 256 == 0


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        L._ptr(torch.zeros(4, dtype=torch.int32), "int32", "x")
    with pytest.raises(TypeError):
        L._ptr(torch.zeros(4, dtype=torch.float32), "int32", "x")


@pytest.mark.parametrize("kw,status", [
    (dict(N=-1), L.LEAP_ERR_INVALID_ARG),
    (dict(V=0), L.LEAP_ERR_INVALID_ARG),
    (dict(ld=999), L.LEAP_ERR_INVALID_ARG),
    (dict(inv_temperature=0.0), L.LEAP_ERR_INVALID_ARG),
    (dict(inv_temperature=float("nan")), L.LEAP_ERR_INVALID_ARG),
    (dict(token_ids=None), L.LEAP_ERR_INVALID_ARG),
    (dict(logp_out=None), L.LEAP_ERR_INVALID_ARG),
    (dict(logits=FAKE + 8), L.LEAP_ERR_MISALIGNED),
    (dict(ld=1012), L.LEAP_ERR_MISALIGNED),
    (dict(V=L.LEAP_MAX_V + 1, ld=L.LEAP_MAX_V + 8), L.LEAP_ERR_UNSUPPORTED),
])
def test_logprob_fwd_rejects(kw, status):
    a = dict(logits=FAKE, ld=1024, N=8, V=1000, token_ids=FAKE, w_tok=None, inv_temperature=1.0,
             logp_out=FAKE, dev_err=None, stream=0)
    a.update(kw)
    with pytest.raises(L.LeapError) as e:
        L.leap_logprob_fwd(**a)
    assert e.value.status == status


def test_probe_rejects():
    with pytest.raises(L.LeapError):
        L.leap_probe_hbm(FAKE, FAKE, 15, 0, stream=0)
    with pytest.raises(L.LeapError):
        L.leap_probe_hbm(FAKE, FAKE, 16, 3, stream=0)
    with pytest.raises(L.LeapError) as e:
        L.leap_probe_hbm(FAKE + 4, FAKE, 16, 0, stream=0)
    assert e.value.status == L.LEAP_ERR_MISALIGNED
    for iters, wgs, sink, rnd in ((0, 4, FAKE, 0), (10, 0, FAKE, 0), (10, 4, None, 0),
                                  (10, 4, FAKE, 2), (10, 4, FAKE, -1)):
        with pytest.raises(L.LeapError) as e:
            L.leap_probe_mfma(iters, wgs, sink, random_operands=rnd, stream=0)
        assert e.value.status == L.LEAP_ERR_INVALID_ARG


def _lmhead(**kw):
    p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
    a = dict(hidden=FAKE, weight=FAKE, N=8, V=1000, H=64, token_ids=FAKE, old_logp=FAKE,
             ref_logp=FAKE, adv_tok=FAKE, w_tok=FAKE, params=p, logp_out=None, tok_loss_out=None,
             loss_out=FAKE, dhidden=FAKE, dweight=FAKE, accumulate_dweight=0, workspace=FAKE,
             ws_bytes=1 << 20, dev_err=None, stream=0)
    a.update(kw)
    return L.leap_grpo_lmhead_fwd_bwd(**a)


@pytest.mark.parametrize("kw,status", [
    (dict(N=-1), L.LEAP_ERR_INVALID_ARG),
    (dict(V=0), L.LEAP_ERR_INVALID_ARG),
    (dict(H=0), L.LEAP_ERR_INVALID_ARG),
    (dict(accumulate_dweight=2), L.LEAP_ERR_INVALID_ARG),
    (dict(loss_out=None), L.LEAP_ERR_INVALID_ARG),
    (dict(params=None), L.LEAP_ERR_INVALID_ARG),
    (dict(hidden=None), L.LEAP_ERR_INVALID_ARG),
    (dict(w_tok=None), L.LEAP_ERR_INVALID_ARG),
    (dict(H=48), L.LEAP_ERR_UNSUPPORTED),
    (dict(H=96), L.LEAP_ERR_UNSUPPORTED),  # k-tiles of 64
    (dict(V=1 << 20, H=4096), L.LEAP_ERR_UNSUPPORTED),  # W beyond 32-bit offsets
    (dict(N=131072, V=151936, H=4096), L.LEAP_ERR_UNSUPPORTED),  # one 16384-column dZ chunk past 4 GiB
    (dict(N=130816, V=151936, H=4096), L.LEAP_ERR_WORKSPACE),  # largest N that fits; only the workspace is short
    (dict(hidden=FAKE + 8), L.LEAP_ERR_MISALIGNED),
    (dict(weight=FAKE + 2), L.LEAP_ERR_MISALIGNED),
    (dict(dweight=FAKE + 2), L.LEAP_ERR_MISALIGNED),
    (dict(dhidden=FAKE + 8), L.LEAP_ERR_MISALIGNED),
    (dict(workspace=None), L.LEAP_ERR_WORKSPACE),
    (dict(ws_bytes=1024), L.LEAP_ERR_WORKSPACE),
    (dict(weight_t=FAKE + 8), L.LEAP_ERR_MISALIGNED),
])
def test_lmhead_rejects(kw, status):
    if "ws_bytes" not in kw and "workspace" not in kw:
        kw["ws_bytes"] = L.leap_lmhead_workspace_size(8, 1000, 64)
    with pytest.raises(L.LeapError) as e:
        _lmhead(**kw)
    assert e.value.status == status


def test_lmhead_workspace_with_prepared_weight():
    # With a caller's transposed weight the call needs the workspace without
    # its last region (the transposed weight); without one, all of it.
    full = L.leap_lmhead_workspace_size(8, 1000, 64)
    wt = L.leap_lmhead_weight_t_size(1000, 64)
    for weight_t, short in ((None, full - 1), (FAKE + (1 << 30), full - wt - 1)):
        with pytest.raises(L.LeapError) as e:
            _lmhead(weight_t=weight_t, ws_bytes=short)
        assert e.value.status == L.LEAP_ERR_WORKSPACE


def test_lmhead_weight_t_size_and_transpose_rejects():
    assert L.leap_lmhead_weight_t_size(151936, 4096) == 2 * 4096 * 152064
    assert L.leap_lmhead_weight_t_size(1000, 64) == 2 * 64 * 1024
    assert L.leap_lmhead_weight_t_size(0, 64) == 0 and L.leap_lmhead_weight_t_size(10, 0) == 0
    n = L.leap_lmhead_weight_t_size(1000, 64)
    for kw, status in [(dict(V=0), L.LEAP_ERR_INVALID_ARG), (dict(H=0), L.LEAP_ERR_INVALID_ARG),
                       (dict(weight=None), L.LEAP_ERR_INVALID_ARG),
                       (dict(weight_t=None), L.LEAP_ERR_INVALID_ARG),
                       (dict(H=96), L.LEAP_ERR_UNSUPPORTED),
                       (dict(V=1 << 20, H=4096), L.LEAP_ERR_UNSUPPORTED),
                       (dict(weight=FAKE + 2), L.LEAP_ERR_MISALIGNED),
                       (dict(weight_t=FAKE + 8), L.LEAP_ERR_MISALIGNED),
                       (dict(nbytes=n - 1), L.LEAP_ERR_WORKSPACE)]:
        a = dict(weight=FAKE, V=1000, H=64, weight_t=FAKE, nbytes=n, stream=0)
        a.update(kw)
        with pytest.raises(L.LeapError) as e:
            L.leap_lmhead_transpose_weight(**a)
        assert e.value.status == status, kw


def test_lmhead_rejects_params():
    p = L.leap_grpo_params(0.2, 0.2, 0.01, 9, 1.0)
    with pytest.raises(L.LeapError) as e:
        _lmhead(params=p, ws_bytes=L.leap_lmhead_workspace_size(8, 1000, 64))
    assert e.value.status == L.LEAP_ERR_UNSUPPORTED


def test_lmhead_workspace_size():
    assert L.leap_lmhead_workspace_size(-1, 10, 64) == 0
    assert L.leap_lmhead_workspace_size(8, 0, 64) == 0
    small = L.leap_lmhead_workspace_size(8, 1000, 64)
    assert small > 0 and small % 256 == 0
    # the gathered live rows of H, row-major and transposed (2 H N_pad bf16
    # each), the transposed weight (H V_pad bf16), per-tile row statistics,
    # four per-row vectors and the row list (4 N_pad each), one bf16 chunk of
    # dZ, and the compaction's per-segment counts (4096-row segments); chunks
    # are 32768 columns unless a 32768-wide dZ chunk would reach 4 GiB
    def want(n, v, h):
        n_pad = (n + 255) // 256 * 256
        v_pad = (v + 255) // 256 * 256
        vc = 32768 if n_pad * 32768 * 2 < (1 << 32) - 64 else 16384
        vc = min(vc, v_pad)
        return (2 * 2 * h * n_pad + 2 * h * v_pad + 8 * n_pad * (v_pad // 256) + 5 * 4 * n_pad
                + 2 * n_pad * vc + 4 * -(-n_pad // 4096) + 4)

    for n, v, h in [(16384, 151936, 4096), (65280, 151936, 4096), (65281, 151936, 4096),
                    (1000, 20000, 512)]:
        assert abs(L.leap_lmhead_workspace_size(n, v, h) - want(n, v, h)) <= 12 * 256, (n, v, h)
    # the narrow chunk takes over from N_pad = 65536 (a 4 GiB dZ chunk otherwise)
    assert (L.leap_lmhead_workspace_size(65281, 151936, 4096)
            < L.leap_lmhead_workspace_size(65280, 151936, 4096))


def test_vocab_shard_entry_points_reject():
    p = L.leap_grpo_params(0.2, 0.2, 0.01, L.LEAP_KL_K3, 1.0)
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_shard_stats(FAKE, 1000, 8, 0, 0, FAKE, None, 1.0, FAKE, stream=0)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_shard_stats(FAKE, 1004, 8, 1000, 0, FAKE, None, 1.0, FAKE, stream=0)
    assert e.value.status == L.LEAP_ERR_MISALIGNED
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_shard_stats(FAKE, 1000, 8, 1000, -1, FAKE, None, 1.0, FAKE, stream=0)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG
    ws = L.leap_vocab_merge_workspace_size(8)
    assert ws % 256 == 0 and ws >= 32
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_merge_objective(FAKE, 0, 8, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, p, None, None,
                                     FAKE, FAKE, FAKE, ws, stream=0)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_merge_objective(FAKE, 2, 8, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, p, None, None,
                                     FAKE, FAKE, FAKE, 16, stream=0)
    assert e.value.status == L.LEAP_ERR_WORKSPACE
    with pytest.raises(L.LeapError) as e:  # the entropy needs the shards' entropy partials
        L.leap_vocab_merge_objective(FAKE, 2, 8, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, p, None, None,
                                     FAKE, FAKE, FAKE, 1 << 20, stream=0, entropy_out=FAKE)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_shard_bwd(FAKE, 1000, 8, 1000, 0, FAKE, FAKE, 1.0, FAKE + 2048, stream=0)
    assert e.value.status == L.LEAP_ERR_INVALID_ARG  # partial overlap with the logits
    # rows wider than LEAP_MAX_V columns are refused before anything is read
    wide, ld = L.LEAP_MAX_V + 1, L.LEAP_MAX_V + 8
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_shard_stats(FAKE, ld, 8, wide, 0, FAKE, None, 1.0, FAKE, stream=0)
    assert e.value.status == L.LEAP_ERR_UNSUPPORTED
    with pytest.raises(L.LeapError) as e:
        L.leap_vocab_shard_bwd(FAKE, ld, 8, wide, 0, FAKE, FAKE, 1.0, FAKE + (1 << 40), stream=0)
    assert e.value.status == L.LEAP_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw,status", [
    (dict(n_groups=-1), L.LEAP_ERR_INVALID_ARG),
    (dict(G=0), L.LEAP_ERR_INVALID_ARG),
    (dict(G=1025), L.LEAP_ERR_INVALID_ARG),
    (dict(M=0), L.LEAP_ERR_INVALID_ARG),
    (dict(n_buckets=0), L.LEAP_ERR_INVALID_ARG),
    (dict(n_buckets=257), L.LEAP_ERR_INVALID_ARG),
    (dict(counters=None), L.LEAP_ERR_INVALID_ARG),
    (dict(gate=None), L.LEAP_ERR_INVALID_ARG),
    (dict(counters=FAKE + 4), L.LEAP_ERR_MISALIGNED),
])
def test_rollout_stats_rejects(kw, status):
    a = dict(pass_turn=FAKE, n_turns=FAKE, gate=FAKE, advantage=None, n_groups=4, G=8, M=2,
             n_buckets=10, counters=FAKE, dev_err=None, stream=0)
    a.update(kw)
    with pytest.raises(L.LeapError) as e:
        L.leap_rollout_stats(**a)
    assert e.value.status == status
