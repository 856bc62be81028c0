"""Parity of the fused LM-head entry point (leap_grpo_lmhead_fwd_bwd) with
the fp64 oracle on seeded inputs shaped like the LM-head workload (hidden
~ N(0, 1), weight ~ N(0, 0.02^2), Gumbel-max tokens).

Bars: log-probs within 2e-3 absolute, per-token loss within 2e-3 relative,
total loss within 1e-3 relative; dH and dW entrywise within (2^-8 + 1e-4)
of the oracle's |dZ| |W| and |dZ|^T |H| (dZ is rounded to bf16 before the
gradient products, which moves every term by at most 2^-8 of itself, and the
fp32 softmax adds about 1e-5); excluded rows give exactly zero gradient
rows.  At the full 16384 x 151936 x 4096 shape, and at N = 65281 (where the
call takes 16384-column vocabulary chunks), the oracle scores 64 sampled rows
(log-prob, loss, dH); dW there is cross-checked against the logits-resident
kernel on bf16 logits plus a torch GEMM (a looser bar, since those logits are
rounded to bf16)."""
import numpy as np
import pytest

import oracle
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu


def _kw(kl_type=0, inv_temp=1.0, kl_coef=0.01):
    return dict(eps_lo=0.2, eps_hi=0.2, kl_coef=kl_coef, kl_type=kl_type, inv_temp=inv_temp)


_compare = U.compare_lmhead


def test_lmhead_reduced_shape_full_parity():
    N, V, H = 1024, 32768, 512
    U.log(f"lmhead reduced N={N} V={V} H={H} seed=1005")
    inp = U.lmhead_inputs(1005, N, V, H, bad_rows=(17,))
    gpu = U.run_lmhead(inp, **_kw())
    _compare(inp, gpu, _kw(), bad_expected=1, what="reduced")


@pytest.mark.parametrize("N,V,H,inv_temp,kl_type", [
    (300, 1000, 128, 0.8, 1),     # ragged rows and vocabulary, one chunk
    (257, 8492, 64, 1.0, 2),      # one chunk, 8704 wide with 8492 live columns
    (1, 300, 64, 1.0, 0),         # a single row, one k-tile
    (513, 16640, 128, 1.25, 0),   # one chunk, 65 tiles wide
    (129, 33000, 64, 1.0, 1),     # two 32768-column chunks, the last 256 wide with 232 live columns
    (65, 70000, 64, 1.0, 2),      # three chunks (dH accumulated twice), the last 4608 wide
    (70, 700, 192, 1.0, 0),       # three k-tiles along H (odd count > 1), ragged everywhere
])
def test_lmhead_ragged_shapes(N, V, H, inv_temp, kl_type):
    U.log(f"lmhead ragged N={N} V={V} H={H} T^-1={inv_temp} kl={kl_type}")
    inp = U.lmhead_inputs(2000 + N, N, V, H, inv_temp=inv_temp)
    kw = _kw(kl_type=kl_type, inv_temp=inv_temp, kl_coef=0.05)
    gpu = U.run_lmhead(inp, **kw)
    _compare(inp, gpu, kw, what=f"N={N} V={V}")


def test_lmhead_edge_tokens():
    # Rollout tokens on the column edges of the dZ pass: the first column, the
    # 8- and 128-column edges of a lane's and a wave's store, tile (256) and
    # chunk (32768) boundaries, and the first and last live column of the
    # partial last tile (V - 1).  Each of these rows has its token column
    # written by a different lane position of the transposed store.
    N, V, H = 64, 70000, 64
    U.log(f"lmhead edge tokens N={N} V={V} H={H}")
    inp = U.lmhead_inputs(4001, N, V, H)
    edges = [0, 7, 8, 127, 128, 255, 256, 32767, 32768, 65535, 65536, 69887, 69888, 69999]
    y = inp["y"].copy()
    y[:len(edges)] = edges
    w = inp["w"].copy()
    w[:len(edges)] = 1.0 / N
    z = np.zeros(N)
    c = oracle.lmhead(inp["h_u16"], inp["w_u16"], y, z, z, z, np.ones(N), want_grads=False)["logp"]
    n_old, n_ref = np.random.default_rng(4001).normal(0.0, 0.05, (2, N))
    inp.update(y=y, w=w, old=(c + n_old).astype(np.float32), ref=(c + 2 * n_ref).astype(np.float32))
    kw = _kw()
    gpu = U.run_lmhead(inp, **kw)
    _compare(inp, gpu, kw, what="edge tokens")


@pytest.mark.parametrize("V", [2, 50, 1000])
def test_lmhead_confident_rows(V):
    # Logits of std ~19 (hidden states scaled by 120): the sampled token is
    # nearly always the row's largest logit and p_y is within a small
    # fraction of 1, so the token's dZ entry g (1 - p_y) is far below |g|.
    # It is formed in fp32 from the log-prob, whose fp32 error bounds it to
    # 2^-12 |g| (as in the logits-resident kernel), a term the shared
    # comparison adds at each row's token column; rounding -g p_y to bf16
    # and adding g would leave up to 2^-9 |g| there.
    N, H = 200, 64
    U.log(f"lmhead confident rows N={N} V={V} H={H}")
    inp = U.lmhead_inputs(4501 + V, N, V, H, h_scale=120.0)
    kw = _kw()
    gpu = U.run_lmhead(inp, **kw)
    o = _compare(inp, gpu, kw, what=f"confident V={V}")
    assert np.median(np.exp(o["logp"][inp["w"] != 0])) > 0.9


def test_lmhead_accumulate_and_optional_gradients():
    N, V, H = 300, 1000, 192
    U.log(f"lmhead options N={N} V={V} H={H}")
    inp = U.lmhead_inputs(3001, N, V, H)
    kw = _kw()
    full = U.run_lmhead(inp, **kw)
    o = _compare(inp, full, kw, what="options")
    init = np.random.default_rng(5).normal(0, 1, (V, H)).astype(np.float32)
    acc = U.run_lmhead(inp, accumulate=1, dW_init=init, **kw)
    np.testing.assert_array_equal(acc["dW"], init + full["dW"])  # one fp32 add per entry
    only_h = U.run_lmhead(inp, want_dW=False, **kw)
    np.testing.assert_array_equal(only_h["dH"], full["dH"])
    only_w = U.run_lmhead(inp, want_dH=False, **kw)
    np.testing.assert_array_equal(only_w["dW"], full["dW"])
    fwd = U.run_lmhead(inp, want_dH=False, want_dW=False, **kw)
    np.testing.assert_array_equal(fwd["logp"], full["logp"])
    assert fwd["loss"] == full["loss"]
    assert abs(full["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-7


@pytest.mark.parametrize("N,V,H", [(300, 1000, 192), (129, 33000, 64)])
def test_lmhead_prepared_weight(N, V, H):
    # A transposed weight prepared once (leap_lmhead_transpose_weight) and
    # the call's own transpose give bitwise the same results; the prepared
    # call runs in the smaller workspace.
    U.log(f"lmhead prepared weight N={N} V={V} H={H}")
    inp = U.lmhead_inputs(3401 + N, N, V, H)
    kw = _kw()
    own = U.run_lmhead(inp, **kw)
    prep = U.run_lmhead(inp, prepared=True, **kw)
    for k in ("logp", "tok_loss", "dH", "dW"):
        np.testing.assert_array_equal(prep[k], own[k], err_msg=k)
    assert prep["loss"] == own["loss"]
    _compare(inp, prep, kw, what="prepared")


def test_lmhead_empty_batch():
    import torch
    from paper_2608_01804_amd import leap as L
    V, H = 1000, 64
    U.log("lmhead N=0")
    hid = torch.zeros((1, H), dtype=torch.bfloat16, device=U.dev())
    wt = torch.zeros((V, H), dtype=torch.bfloat16, device=U.dev())
    loss = torch.full((1,), float("nan"), dtype=torch.float32, device=U.dev())
    ws_bytes = L.leap_lmhead_workspace_size(0, V, H)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=U.dev())
    p = L.leap_grpo_params(0.2, 0.2, 0.01, 0, 1.0)
    one_f = torch.zeros(1, dtype=torch.float32, device=U.dev())
    one_i = torch.zeros(1, dtype=torch.int32, device=U.dev())
    for accumulate in (0, 1):
        dW = torch.full((V, H), 3.0, dtype=torch.float32, device=U.dev())
        L.leap_grpo_lmhead_fwd_bwd(hid, wt, 0, V, H, one_i, one_f, one_f, one_f, one_f, p, None,
                                   None, loss, None, dW, accumulate, ws, ws_bytes)
        torch.cuda.synchronize()
        assert loss.item() == 0.0
        assert torch.all(dW == (3.0 if accumulate else 0.0)).item()


def test_lmhead_all_rows_excluded():
    # Every weight 0: no live row is left after the compaction, so no GEMM
    # tile runs on data; every output is still written (zeros), and an
    # accumulated dW is left as it was.
    N, V, H = 300, 1000, 64
    U.log(f"lmhead all rows excluded N={N} V={V} H={H}")
    inp = U.lmhead_inputs(3101, N, V, H)
    inp["w"] = np.zeros(N, np.float32)
    kw = _kw()
    init = np.random.default_rng(6).normal(0, 1, (V, H)).astype(np.float32)
    for accumulate in (0, 1):
        gpu = U.run_lmhead(inp, accumulate=accumulate, dW_init=init if accumulate else None, **kw)
        assert gpu["bad"] == 0 and gpu["loss"] == 0.0
        assert np.all(gpu["logp"] == 0.0) and np.all(gpu["tok_loss"] == 0.0)
        assert np.all(gpu["dH"] == 0.0)
        np.testing.assert_array_equal(gpu["dW"], init if accumulate else np.zeros((V, H), np.float32))


def test_lmhead_excluded_rows_are_not_read():
    # Excluded rows (w = 0) take no part in the call: NaN and inf hidden
    # states there reach no output.  The excluded rows include the first and
    # the last row, a tile edge and a run longer than a 256-row tile; the
    # oracle scores the same inputs with finite values in those rows.
    import torch
    N, V, H = 700, 3000, 128
    U.log(f"lmhead excluded rows not read N={N} V={V} H={H}")
    inp = U.lmhead_inputs(3201, N, V, H, mask_frac=0.0)
    w = inp["w"].copy()
    excl = np.r_[0, 1, 2, 255, 256, 300:561, 699]
    w[excl] = 0.0
    ref_inp = dict(inp, w=w)
    hid = inp["hid"].clone()
    hid[torch.from_numpy(excl[0::2]).to(U.dev())] = float("nan")
    hid[torch.from_numpy(excl[1::2]).to(U.dev())] = float("inf")
    kw = _kw(kl_coef=0.05)
    gpu = U.run_lmhead(dict(ref_inp, hid=hid), **kw)
    _compare(ref_inp, gpu, kw, what="poisoned excluded rows")
    assert np.all(np.isfinite(gpu["dW"])) and np.all(np.isfinite(gpu["dH"]))


def test_lmhead_compaction_over_segments():
    # 9000 rows: three 4096-row segments of the live-row compaction, 40% of
    # the rows excluded at random, plus an excluded run that starts a
    # segment and one that crosses a segment boundary.
    N, V, H = 9000, 2000, 64
    U.log(f"lmhead compaction N={N} V={V} H={H}")
    inp = U.lmhead_inputs(3301, N, V, H, mask_frac=0.4, bad_rows=(4095, 8191))
    w = inp["w"].copy()
    w[4096:4700] = 0.0
    w[8150:8191] = 0.0
    w[8192:8400] = 0.0
    inp["w"] = w
    kw = _kw()
    gpu = U.run_lmhead(inp, **kw)
    _compare(inp, gpu, kw, bad_expected=2, what="compaction")


def _sampled_rows_and_dw_check(inp, gpu, kw, seed, what):
    """Oracle on 64 sampled rows (log-prob, loss, dH), then dW over every row
    against the logits-resident kernel on torch-formed bf16 logits and a
    torch fp32 GEMM (those logits are rounded to bf16, hence the looser bar)."""
    import torch
    N, H = inp["hid"].shape
    V = inp["wt"].shape[0]
    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, 5, N - 1], rng.choice(N, 61, replace=False)]))
    U.log(f"  oracle on {rows.size} rows")
    o = oracle.lmhead(inp["h_u16"], inp["w_u16"], inp["y"], inp["old"], inp["ref"], inp["adv"],
                      inp["w"], rows=rows, **kw)
    y, w = inp["y"][rows], inp["w"][rows]
    valid = (w != 0) & (y < V)
    err = np.max(np.abs(gpu["logp"][rows][valid] - o["logp"][valid]))
    U.log(f"  sampled logp max err {err:.3e}")
    assert err < 2e-3
    np.testing.assert_allclose(gpu["tok_loss"][rows][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    dH = gpu["dH"][torch.from_numpy(rows).to(U.dev())].cpu().numpy()
    Wf = U.bf16_f64(inp["w_u16"])
    U.check_grad(dH, o["dH"], np.abs(o["dZ"]) @ np.abs(Wf), f"{what} sampled dH")
    del Wf
    assert np.isfinite(gpu["loss"])

    U.log("  cross-check of dW via bf16 logits")
    hid, wt = inp["hid"], inp["wt"]
    lg = torch.empty((N, V), dtype=torch.bfloat16, device=U.dev())
    wf = wt.float()
    for r0 in range(0, N, 1024):
        lg[r0:r0 + 1024] = (hid[r0:r0 + 1024].float() @ wf.T).to(torch.bfloat16)
    del wf
    ref = U.run_grpo(lg, V, inp["y"], inp["old"], inp["ref"], inp["adv"], inp["w"], inplace=True, **kw)
    lp_err = np.max(np.abs(ref["logp"] - gpu["logp"]))
    U.log(f"  logp vs bf16-logits path: max diff {lp_err:.3e}")
    assert lp_err < 5e-2
    hf = hid.float()
    worst = 0.0
    for v0 in range(0, V, 8192):
        d = lg[:, v0:v0 + 8192].float()
        dw_x = d.T @ hf
        bound = d.abs().T @ hf.abs()
        diff = (gpu["dW"][v0:v0 + 8192] - dw_x).abs()
        worst = max(worst, float((diff / bound.clamp(min=1e-30)).max().item()))
        assert torch.all(diff <= 0.03 * bound + 1e-9).item(), v0
    U.log(f"  dW vs bf16-logits path: max diff/bound {worst:.3e}")


def test_lmhead_narrow_chunks():
    # N_pad = 65536: a 32768-column dZ chunk would pass the GEMM core's 4 GiB
    # operand offsets, so the call takes 16384-column chunks (two at V =
    # 20000, the second 3840 wide) and the k-major dW pass runs K = 65536.
    N, V, H = 65281, 20000, 64
    U.log(f"lmhead narrow chunks N={N} V={V} H={H}: inputs")
    inp = U.lmhead_inputs(5001, N, V, H, cur="torch", bad_rows=(5,))
    kw = _kw()
    U.log("  fused call")
    gpu = U.run_lmhead(inp, to_host=False, **kw)
    assert gpu["bad"] == 1
    _sampled_rows_and_dw_check(inp, gpu, kw, 5001, "narrow")


def _oracle_by_row_blocks(inp, kw, block=2048):
    """The oracle's fused LM head over every row, evaluated a block of rows
    at a time (``oracle.lmhead`` with ``rows``) so that Z and dZ never exist
    whole; dW = dZ^T H summed over the blocks in order.  Returns logp,
    tok_loss, loss, dH, dW and the bounds |dZ| |W| and |dZ|^T |H| of the
    gradient check."""
    N, H = inp["hid"].shape
    V = inp["wt"].shape[0]
    Hf, Wf = U.bf16_f64(inp["h_u16"]), U.bf16_f64(inp["w_u16"])
    aW, aH = np.abs(Wf), np.abs(Hf)
    out = {"logp": np.empty(N), "tok_loss": np.empty(N), "loss": 0.0, "bad": 0,
           "dH": np.empty((N, H)), "bH": np.empty((N, H)), "dW": np.zeros((V, H)),
           "bW": np.zeros((V, H))}
    for r0 in range(0, N, block):
        rows = np.arange(r0, min(N, r0 + block))
        o = oracle.lmhead(inp["h_u16"], inp["w_u16"], inp["y"], inp["old"], inp["ref"],
                          inp["adv"], inp["w"], rows=rows, **kw)
        out["logp"][rows], out["tok_loss"][rows] = o["logp"], o["tok_loss"]
        out["loss"] += o["loss"]
        out["bad"] += o["bad"]
        out["dH"][rows] = o["dH"]
        aZ = np.abs(o["dZ"])
        out["bH"][rows] = aZ @ aW
        out["dW"] += o["dZ"].T @ Hf[rows]
        out["bW"] += aZ.T @ aH[rows]
    return out


@pytest.mark.parametrize("N,V,H", [
    (16384, 4096, 128),   # dW pass: K = 16384, one 4096-column chunk
    (65281, 20000, 64),   # K = 65536, two 16384-column chunks (the second 3840 wide)
])
def test_lmhead_long_k_dw_oracle(N, V, H):
    """dW = dZ^T H on the k-major dW pass at the reduction lengths of the
    full-size calls (K = N_pad = 16384 and 65536), and the narrow-chunk
    split, element by element against the fp64 oracle over every row."""
    U.log(f"lmhead long-K N={N} V={V} H={H}: inputs")
    inp = U.lmhead_inputs(6000 + H, N, V, H, cur="torch", bad_rows=(3,))
    kw = _kw()
    U.log("  fused call")
    gpu = U.run_lmhead(inp, **kw)
    U.log("  oracle by row blocks")
    o = _oracle_by_row_blocks(inp, kw)
    valid = (inp["w"] != 0) & (inp["y"] < V)
    assert gpu["bad"] == o["bad"] == 1
    err = np.max(np.abs(gpu["logp"][valid] - o["logp"][valid]))
    U.log(f"  logp max err {err:.3e}")
    assert err < 2e-3
    np.testing.assert_allclose(gpu["tok_loss"][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    assert abs(gpu["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-7, (gpu["loss"], o["loss"])
    U.check_grad(gpu["dH"], o["dH"], o["bH"], f"long-K N={N} dH")
    U.check_grad(gpu["dW"], o["dW"], o["bW"], f"long-K N={N} dW")
    assert np.all(gpu["dH"][~valid] == 0.0)


def test_lmhead_full_shape_sampled_rows():
    N, V, H = 16384, 151936, 4096
    U.log(f"lmhead full N={N} V={V} H={H}: inputs")
    inp = U.lmhead_inputs(1005, N, V, H, cur="torch", bad_rows=(5,))
    kw = _kw()
    U.log("  fused call")
    gpu = U.run_lmhead(inp, to_host=False, **kw)
    assert gpu["bad"] == 1
    _sampled_rows_and_dw_check(inp, gpu, kw, 1005, "full")
