"""GPU parity: every libleap entry point against the fp64 oracle on the same
seeded inputs (integers bit-exact; R bit-exact as float32; A within 1e-6
relative; token advantages within float32 rounding; log-probs within 2e-3
absolute, loss within 1e-3 relative, dlogits within 2e-2 absolute).

Small shapes get full element-by-element parity; the full microbatch shapes
(8192 and 16384 rows of a 151936 vocabulary), in the same launch
configuration the benchmark times, get every log-prob, the loss, and sampled
dlogits rows."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads as wl
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu

KW = dict(eps_lo=0.2, eps_hi=0.2, kl_coef=0.01)


def _default_tau(G):
    return oracle.tau_from_pass_rate(G, Fraction(0), True, Fraction(3, 4), True)


def _step(name):
    lat = wl.draw_latent(name)
    tmin, tmax = _default_tau(lat.G)
    _, gate = oracle.dcp_gate(lat.first_turn_pass, lat.G, tmin, tmax)
    ro = wl.realize(lat, gate)
    return lat, ro


# ----------------------------------------------------------------------------
# DCP gate
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny", "mid", "full", "stress"])
def test_gate_parity(name):
    lat = wl.draw_latent(name)
    G = lat.G
    windows = [_default_tau(G), (0, G), (G // 2, G), (0, G // 2), (G, G), (0, 0)]
    for tmin, tmax in windows:
        U.log(f"gate {name} G={G} tau=[{tmin},{tmax}]")
        nf_o, g_o = oracle.dcp_gate(lat.first_turn_pass, G, tmin, tmax)
        nf_g, g_g = U.run_gate(lat.first_turn_pass, G, tmin, tmax)
        assert np.array_equal(nf_g, nf_o) and np.array_equal(g_g, g_o)


@pytest.mark.parametrize("G", [1, 3, 64, 65, 200, 1024])
def test_gate_sizes(G):
    rng = np.random.default_rng(G)
    n_groups = 37
    ftp = (rng.random((n_groups, G)) < 0.4).astype(np.uint8) * rng.integers(1, 256, (n_groups, G))
    tmin, tmax = G // 4, G - G // 5
    U.log(f"gate G={G}")
    nf_o, g_o = oracle.dcp_gate(ftp.astype(np.uint8), G, tmin, tmax)
    nf_g, g_g = U.run_gate(ftp.astype(np.uint8), G, tmin, tmax)
    assert np.array_equal(nf_g, nf_o) and np.array_equal(g_g, g_o)


# ----------------------------------------------------------------------------
# Rank advantages
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("name,key", [("tiny", 0), ("mid", 0), ("full", 0), ("stress", 0),
                                      ("stress", 1), ("full", 1)])
def test_rank_parity(name, key):
    lat, ro = _step(name)
    nt = wl.stress_token_counts(lat) if name == "stress" else ro.n_tokens
    U.log(f"rank {name} key={key} rollouts={ro.n_rollouts}")
    ora = oracle.rank_tournament(ro.pass_turn, ro.G, ro.M, key_mode=key, eps=U.EPS_ADV,
                                 speedup_q=ro.speedup_q, n_tokens=nt)
    gpu = U.run_rank(ro.pass_turn, ro.G, ro.M, key=key, speedup_q=ro.speedup_q if key else None,
                     n_tokens=nt if key else None)
    U.check_rank(gpu, ora)


@pytest.mark.parametrize("G", [2, 3, 63, 64, 65, 128, 200, 256, 1000, 1024])
@pytest.mark.parametrize("key", [0, 1])
def test_rank_group_sizes(G, key):
    rng = np.random.default_rng(1000 + G)
    n_groups, M = 29, 3
    pt = rng.integers(0, M + 1, size=n_groups * G).astype(np.int32)
    sq = np.where(pt > 0, rng.integers(0, 5, pt.size), 0).astype(np.int32)
    nt = rng.integers(1, 6, pt.size).astype(np.int32)
    U.log(f"rank G={G} key={key}")
    ora = oracle.rank_tournament(pt, G, M, key_mode=key, eps=U.EPS_ADV, speedup_q=sq, n_tokens=nt)
    gpu = U.run_rank(pt, G, M, key=key, speedup_q=sq if key else None, n_tokens=nt if key else None)
    U.check_rank(gpu, ora)


def test_rank_invalid_and_adv_none():
    pt = np.array([1, 4, -1, 0, 2, 2, 0, 1], np.int32)
    ora = oracle.rank_tournament(pt, 4, 2, adv_norm=oracle.ADV_NONE)
    gpu = U.run_rank(pt, 4, 2, norm=1)
    U.check_rank(gpu, ora)
    assert gpu["bad"] == 2
    assert np.array_equal(gpu["A"], gpu["R"])


def test_rank_all_equal_gives_zero():
    pt = np.ones(64 * 8, np.int32)
    gpu = U.run_rank(pt, 64, 2)
    assert np.all(gpu["R"] == 0) and np.all(gpu["A"] == 0)


# ----------------------------------------------------------------------------
# Token advantages
# ----------------------------------------------------------------------------
def _step_tokens(name, layout="packed"):
    lat, ro = _step(name)
    pack = wl.pack if layout == "packed" else wl.pack_right_padded
    mbs = pack(ro, lat.cfg["rows_per_mb"])
    tok_r = np.concatenate([m.tok_rollout for m in mbs])
    tok_t = np.concatenate([m.tok_turn for m in mbs])
    ora = oracle.rank_tournament(ro.pass_turn, ro.G, ro.M, eps=U.EPS_ADV)
    return lat, ro, mbs, tok_r, tok_t, ora["A"].astype(np.float32)


def _denom(agg, ro):
    if agg == oracle.AGG_SEQ_MEAN_TOKEN_MEAN:
        return float(ro.n_rollouts)
    if agg == oracle.AGG_TOKEN_MEAN:
        return float(ro.n_tokens.sum())
    return 1.0


@pytest.mark.parametrize("name", ["tiny", "mid", "full"])
@pytest.mark.parametrize("agg", [0, 1, 2])
def test_token_adv_parity(name, agg):
    lat, ro, mbs, tok_r, tok_t, A32 = _step_tokens(name)
    gamma = float(np.float32(lat.cfg["gamma"]))
    U.log(f"token_adv {name} agg={agg} N={tok_r.size}")
    adv_o, w_o, bad_o = oracle.token_advantages(A32.astype(np.float64), tok_r, tok_t, ro.n_turns,
                                                ro.n_tokens, gamma, agg, _denom(agg, ro))
    adv_g, w_g, bad_g = U.run_token_adv(A32, tok_r, tok_t, ro.n_turns, ro.n_tokens, gamma, agg,
                                        _denom(agg, ro))
    assert bad_o == 0 and bad_g == 0
    U.check_f32_rounding(adv_g, adv_o, "token advantage")
    U.check_f32_rounding(w_g, w_o, "weight")
    assert np.all((tok_r < 0) <= (w_g == 0))


def test_token_adv_invalid_rows_count():
    A = np.array([0.5, -1.0], np.float32)
    tok_r = np.array([0, 1, 2, -2, 1, -1], np.int32)
    tok_t = np.array([0, 1, 0, 0, 5, 0], np.int32)
    n_turns = np.array([1, 2], np.int32)
    n_gen = np.array([1, 2], np.int32)
    adv_o, w_o, bad_o = oracle.token_advantages(A.astype(np.float64), tok_r, tok_t, n_turns, n_gen,
                                                0.5, oracle.AGG_SUM, 1.0)
    adv_g, w_g, bad_g = U.run_token_adv(A, tok_r, tok_t, n_turns, n_gen, 0.5, oracle.AGG_SUM, 1.0)
    assert bad_o == bad_g == 3
    assert np.array_equal(adv_g, adv_o.astype(np.float32)) and np.array_equal(w_g, w_o)


# ----------------------------------------------------------------------------
# Fused log-softmax + surrogate + KL + dlogits
# ----------------------------------------------------------------------------
def _check_rows(gpu, o, valid, what=""):
    assert np.max(np.abs(gpu["logp"][valid] - o["logp"][valid]), initial=0) < 2e-3, what
    assert np.all(gpu["logp"][~valid] == 0) and np.all(gpu["tok_loss"][~valid] == 0)
    np.testing.assert_allclose(gpu["tok_loss"][valid], o["tok_loss"][valid], rtol=2e-3, atol=2e-4)
    assert abs(gpu["loss"] - o["loss"]) <= 1e-3 * abs(o["loss"]) + 1e-7, (gpu["loss"], o["loss"])


def _tiny_weights(agg):
    lat, ro, mbs, tok_r, tok_t, A32 = _step_tokens("tiny")
    adv, w, _ = oracle.token_advantages(A32.astype(np.float64), tok_r, tok_t, ro.n_turns,
                                        ro.n_tokens, 1.0, agg, _denom(agg, ro))
    return adv.astype(np.float32), w.astype(np.float32)


@pytest.mark.parametrize("mode", ["sum", "seq_mean", "clip", "clip_higher"])
def test_grpo_tiny_full_parity(mode):
    """Every row of the tiny workload.  The clip modes draw the old-policy
    log-probs with sigma 0.3, so a third of the rows are clipped;
    clip_higher runs the asymmetric bounds eps_lo = 0.2, eps_hi = 0.28."""
    N, V = 2048, 32768
    old_sigma = wl.CLIP_CASE_OLD_SIGMA if mode.startswith("clip") else wl.OLD_SIGMA
    kw = dict(KW, eps_hi=0.28) if mode == "clip_higher" else KW
    lg, tok, old, ref = U.make_inputs_host(1001, N, V, old_sigma=old_sigma)
    adv, w = _tiny_weights(oracle.AGG_SEQ_MEAN_TOKEN_MEAN if mode == "seq_mean" else oracle.AGG_SUM)
    U.log(f"grpo tiny {mode}")
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, **kw)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **kw)
    valid = w != 0
    _check_rows(gpu, o, valid, mode)
    assert gpu["bad"] == 0
    if mode == "clip_higher":
        # rows whose ratio sits in the windows where the two bounds' roles
        # matter: 1.2 < rho < 1.28 with A > 0, 0.72 < rho < 0.8 with A < 0
        rho = np.exp(o["logp"] - old.astype(np.float64))
        win = ((rho > 1.2) & (rho < 1.28) & (adv > 0)) | ((rho > 0.72) & (rho < 0.8) & (adv < 0))
        U.log(f"  {int(win.sum())} rows in the asymmetric windows")
        assert win.sum() >= 20
    for r0 in range(0, N, 256):
        rows = np.arange(r0, r0 + 256)
        U.check_dlogits(U.dl_rows(gpu["dl_dev"], rows, V), lg, rows, tok, old, ref, adv, w, V,
                        atol=1e-2 if mode == "seq_mean" else 2e-2, kw=kw,
                        rel_to_max=(mode == "seq_mean"))


# every row-kernel family: one-wave and 256-lane resident rows, the
# persistent row queue, rows partly in LDS, the streaming kernel
@pytest.mark.parametrize("V", [2, 7, 300, 5000, 32768, 151936, 200003, 300000])
def test_grpo_wide_range_and_peaked_rows(V):
    """Entry-wise relative check of dlogits on rows whose probabilities span
    many orders of magnitude: logits of std 6 and 12, and rows with one
    logit 30 above the rest (the token on the spike, or away from it).  The
    kernel keeps each lane's 2^(x c - m_lane c) in [0, 1] as fp16 between
    its two register passes: relative precision 2^-11 down to 2^-14, an
    absolute step of 2^-24 below (subnormals), 0 below 2^-25.  With the
    per-lane scale 2^(m_lane c - lse2) <= 1 and the bf16 store (2^-9), every
    entry of the gradient is within 2^-8 |d| + 2^-24 |g| of the oracle, g
    the row's d loss / d logp; the token's own column, g (1 - p_y), carries
    the fp32 log-prob's error instead: 2^-8 |d| + 2^-12 |g|."""
    N = 64
    rng = np.random.default_rng(V + 6)

    def edit(lg, tok):
        x = wl.bf16_bits_to_f32(lg[:, :V]).astype(np.float32)
        x[:16] *= 3.0                       # std 6
        x[48:] *= 6.0                       # std 12
        spike = rng.integers(0, V, N)
        for k in range(16, 48):
            x[k, spike[k]] += 30.0
            tok[k] = spike[k] if k < 32 else (spike[k] + 1 + rng.integers(0, V - 1)) % V
        lg[:, :V] = wl.f32_to_bf16_bits(x)
        for k in list(range(16)) + list(range(48, N)):  # tokens of the rescaled rows
            tok[k] = rng.integers(0, V)

    lg, tok, old, ref = U.make_inputs_host(V + 6, N, V, ld=(V + 7) // 8 * 8, edit=edit)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = np.ones(N, np.float32)
    kw = dict(KW, kl_coef=0.05)
    U.log(f"grpo wide-range / peaked rows V={V}")
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, **kw)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, **kw)
    assert gpu["bad"] == o["bad"] == 0
    _check_rows(gpu, o, w != 0)
    got = U.dl_rows(gpu["dl_dev"], np.arange(N), V)
    want = o["dlogits"]
    # |g| <= w (|A| rho + beta |d KL / d logp|), k3: d KL / d logp = 1 - e^(ref - logp)
    rho = np.exp(o["logp"] - old.astype(np.float64))
    g_max = w * (np.abs(adv) * rho + kw["kl_coef"] * np.abs(1.0 - np.exp(ref - o["logp"])))
    tol = 2.0 ** -8 * np.abs(want) + 2.0 ** -24 * g_max[:, None]
    tol[np.arange(N), tok] = 2.0 ** -8 * np.abs(want[np.arange(N), tok]) + 2.0 ** -12 * g_max
    ratio = np.abs(got - want) / tol
    k, v = np.unravel_index(np.argmax(ratio), ratio.shape)
    U.log(f"  max |err| / bound {ratio.max():.3f} at row {k}, column {v}")
    assert ratio.max() <= 1.0
    # the check is not vacuous: entries below fp16's normal range are present
    if V >= 32768:
        p = np.abs(want) / np.maximum(g_max[:, None], 1e-300)
        assert np.sum((p > 2.0 ** -24) & (p < 2.0 ** -14)) > 1000


SHAPES = [(16, 16, 64), (100, 104, 64), (1000, 1008, 64), (4093, 4096, 32), (8192, 8192, 32),
          (32000, 32000, 32), (32768, 32768, 32), (50257, 50264, 16), (65536, 65536, 16),
          (100000, 100000, 16), (128256, 128256, 16), (151936, 151936, 16),
          # the persistent kernel with a partial last chunk and padding columns
          (150001, 150016, 300),
          (152064, 152064, 16), (160000, 160000, 8), (196608, 196608, 8),
          # rows held partly in LDS (196608 < V <= 270336): one LDS slot with a
          # partial chunk, a ragged middle, exactly 32768 chunks, the largest
          (196609, 196616, 4), (200003, 200008, 8), (262144, 262144, 4), (270336, 270336, 4),
          # the streaming kernel just past it
          (270337, 270344, 4)]


@pytest.mark.parametrize("V,ld,N", SHAPES, ids=[f"V{s[0]}" for s in SHAPES])
def test_grpo_shapes(V, ld, N):
    rng = np.random.default_rng(V)

    def last_token(lg, tok):
        tok[0] = V - 1

    lg, tok, old, ref = U.make_inputs_host(V, N, V, ld=ld, edit=last_token)
    adv = rng.normal(0, 1.5, N).astype(np.float32)
    w = rng.choice([0.0, 1.0, 0.5], N).astype(np.float32)
    w[0] = 1.0
    U.log(f"grpo V={V} ld={ld} N={N}")
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, **KW)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **KW)
    _check_rows(gpu, o, w != 0, f"V={V}")
    rows = np.arange(N)
    U.check_dlogits(U.dl_rows(gpu["dl_dev"], rows, V), lg, rows, tok, old, ref, adv, w, V,
                    atol=2e-2, kw=KW)
    if ld > V:  # padding columns are left untouched
        pad = gpu["dl_dev"][:, V:].float().cpu().numpy()
        assert np.all(np.isnan(pad))


@pytest.mark.parametrize("kl_type,inv_temp", [(0, 0.7), (1, 1.0), (2, 1.3)])
def test_grpo_kl_types_and_temperature(kl_type, inv_temp):
    N, V = 64, 5000
    rng = np.random.default_rng(kl_type)
    lg = wl.logits_host(77, N, V)
    tok = wl.sample_tokens_host(lg, V, 77)
    cur, _ = oracle.logprob_rows(lg, tok, inv_temp=inv_temp)
    old = (cur + rng.normal(0, 0.05, N)).astype(np.float32)
    ref = (cur + rng.normal(0, 0.1, N)).astype(np.float32)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = np.ones(N, np.float32)
    kw = dict(KW, kl_coef=0.1, kl_type=kl_type, inv_temp=inv_temp)
    U.log(f"grpo kl={kl_type} T^-1={inv_temp}")
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, **kw)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, want_dlogits=False, **kw)
    _check_rows(gpu, o, w != 0)
    rows = np.arange(N)
    U.check_dlogits(U.dl_rows(gpu["dl_dev"], rows, V), lg, rows, tok, old, ref, adv, w, V,
                    atol=2e-2, kw=kw)


def test_grpo_special_values_and_errors():
    N, V = 8, 3000

    def edit(lg, tok):
        lg[1, ::5] = 0xFF80  # -inf columns
        tok[1] = 1  # a finite column
        lg[2, :] = 0xFF80  # all -inf: counted, excluded
        tok[3] = V  # out of range: counted, excluded
        tok[4] = -3  # out of range
        tok[5] = V - 1

    lg, tok, old, ref = U.make_inputs_host(5, N, V, edit=edit)
    adv = np.linspace(-2, 2, N).astype(np.float32)
    w = np.ones(N, np.float32)
    w[6] = 0.0  # masked
    U.log("grpo special values")
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, **KW)
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, want_dlogits=False, **KW)
    assert gpu["bad"] == o["bad"] == 3
    valid = np.array([True, True, False, False, False, True, False, True])
    _check_rows(gpu, o, valid)
    rows = np.arange(N)
    got = U.dl_rows(gpu["dl_dev"], rows, V)
    for k in (2, 3, 4, 6):
        assert np.all(got[k] == 0)
    U.check_dlogits(got, lg, rows, tok, old, ref, adv, w, V, atol=2e-2, kw=KW)


@pytest.mark.parametrize("V,N", [(151936, 300), (100003, 2600), (230000, 64)])
def test_grpo_inplace_and_deterministic(V, N):
    # 151936: the persistent kernel with more rows than one per workgroup for
    # some workgroups only; 100003 x 2600: every workgroup taking rows from
    # the queue, in place (each row's loads are issued only after the
    # previous row's stores, never for a row already written), with a
    # partial last chunk; 230000: rows held partly in LDS
    lg, tok, old, ref = U.make_inputs_host(9, N, V, ld=(V + 7) // 8 * 8)
    rng = np.random.default_rng(9)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = rng.choice([0.0, 1.0], N, p=[0.2, 0.8]).astype(np.float32)
    U.log(f"grpo in-place / determinism V={V} N={N}")
    a = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, want_entropy=True, **KW)
    b = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, **KW)
    c = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, adv, w, inplace=True, want_entropy=True,
                   **KW)
    import torch
    # columns V .. ld - 1 are not the call's (NaN-filled out of place, the
    # logits' padding in place)
    da, db, dc = (x["dl_dev"].view(torch.int16)[:, :V] for x in (a, b, c))
    assert torch.equal(da, db)
    assert torch.equal(da, dc)
    assert a["loss"] == b["loss"] == c["loss"]
    assert np.array_equal(a["logp"], c["logp"])
    assert np.array_equal(a["entropy"], c["entropy"])  # in place: the row is read before written
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **KW)
    _check_rows(a, o, w != 0, f"V={V}")
    rows = np.arange(N) if N <= 512 else np.sort(rng.choice(N, 48, replace=False))
    U.check_dlogits(U.dl_rows(a["dl_dev"], rows, V), lg, rows, tok, old, ref, adv, w, V, atol=2e-2,
                    kw=KW)


# The persistent kernel's row queue (55296 < V <= 155648): each workgroup's
# four fixed rows, then rows taken from the queue three ahead; runs of
# excluded rows long enough that workgroups take three or more in a row and
# refill the queue synchronously; tickets past N.  131080 columns is the
# 19-chunk shape's narrowest width (its last two register chunks are empty
# in the first wave), 55297 the persistent range's first.
def _queue_weights(pattern, N, rng):
    w = rng.choice([0.5, 1.0], N).astype(np.float32)
    if pattern == "alt":
        w[1::2] = 0.0
    elif pattern == "runs":  # masked runs of 900 and 500 rows, and a tail run
        w[1024:1924] = 0.0
        w[2000:2500] = 0.0
        w[N - 40:] = 0.0
    elif pattern == "sparse":  # 5% live
        w[rng.random(N) >= 0.05] = 0.0
    return w


QUEUE_CASES = [(151936, 1, "live"), (151936, 255, "live"), (151936, 1024, "alt"),
               (151936, 1100, "live"), (151936, 2600, "runs"), (131080, 2600, "sparse"),
               (131080, 1500, "alt"),
               # the 16-, 12- and 8-chunk shapes' persistent ranges, and the
               # width just below them (one workgroup per row)
               (100003, 2600, "runs"), (128256, 1300, "live"), (73728, 2600, "sparse"),
               (98304, 1100, "alt"), (55297, 2600, "runs"), (65536, 1300, "live"),
               (55296, 1100, "alt")]


@pytest.mark.parametrize("V,N,pattern", QUEUE_CASES,
                         ids=[f"V{v}-N{n}-{p}" for v, n, p in QUEUE_CASES])
def test_grpo_row_queue(V, N, pattern):
    import torch
    rng = np.random.default_rng(N + V)
    ld = (V + 7) // 8 * 8
    U.log(f"grpo row queue V={V} N={N} {pattern}: generating logits")
    lg_dev = torch.empty((N, ld), dtype=torch.bfloat16, device=U.dev())
    wl.logits_device(4242 + N, N, V, ld=ld, device=U.dev(), out=lg_dev)
    tok = wl.sample_tokens_device(lg_dev[:, :V], V, 4242 + N).cpu().numpy()
    lg = lg_dev.view(torch.int16).cpu().numpy().view(np.uint16)
    cur, _ = oracle.logprob_rows(lg, tok, V=V)
    old = (cur + rng.normal(0, 0.05, N)).astype(np.float32)
    ref = (cur + rng.normal(0, 0.1, N)).astype(np.float32)
    adv = rng.normal(0, 1.5, N).astype(np.float32)
    w = _queue_weights(pattern, N, rng)
    a = U.run_grpo(lg_dev, V, tok, old, ref, adv, w, want_entropy=True, **KW)
    b = U.run_grpo(lg_dev, V, tok, old, ref, adv, w, want_entropy=True, **KW)
    assert torch.equal(a["dl_dev"].view(torch.int16), b["dl_dev"].view(torch.int16))
    assert a["loss"] == b["loss"] and np.array_equal(a["logp"], b["logp"])
    assert np.array_equal(a["entropy"], b["entropy"])
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, V=V, want_dlogits=False, **KW)
    valid = w != 0
    _check_rows(a, o, valid, f"V={V} N={N} {pattern}")
    dead = torch.as_tensor(np.flatnonzero(~valid), device=U.dev())
    if dead.numel():
        assert int(a["dl_dev"].index_select(0, dead)[:, :V].view(torch.int16).abs().max()) == 0
    live = np.flatnonzero(valid)
    rows = live if live.size <= 48 else live[np.linspace(0, live.size - 1, 48).astype(int)]
    U.check_dlogits(U.dl_rows(a["dl_dev"], rows, V), lg, rows, tok, old, ref, adv, w, V,
                    atol=2e-2, kw=KW)


def test_grpo_overlapping_calls_on_two_streams():
    """Two fused calls with their own workspaces and outputs, launched on two
    streams without ordering between them, give bitwise the results of the
    same calls run one after the other.  Each call's row queue lives in its
    own workspace, and no workgroup waits for another, so the two persistent
    grids need not be resident together."""
    import torch
    from paper_2608_01804_amd import leap as L
    V, N = 151936, 2000
    cases = []
    for seed in (11, 12):
        rng = np.random.default_rng(seed)
        lg = torch.empty((N, V), dtype=torch.bfloat16, device=U.dev())
        wl.logits_device(seed, N, V, device=U.dev(), out=lg)
        tok = wl.sample_tokens_device(lg, V, seed)
        old = torch.from_numpy(rng.normal(-11.0, 0.5, N).astype(np.float32)).to(U.dev())
        adv = torch.from_numpy(rng.normal(0, 1, N).astype(np.float32)).to(U.dev())
        w = torch.from_numpy(rng.choice([0.0, 1.0], N, p=[0.3, 0.7]).astype(np.float32)).to(U.dev())
        cases.append((lg, tok, old, adv, w))
    p = L.leap_grpo_params(0.2, 0.2, 0.01, 0, 1.0)
    wsb = L.leap_grpo_workspace_size(N, V)

    def outputs():
        return [dict(dl=torch.empty((N, V), dtype=torch.bfloat16, device=U.dev()),
                     lp=torch.empty(N, dtype=torch.float32, device=U.dev()),
                     loss=torch.empty(1, dtype=torch.float32, device=U.dev()),
                     ws=torch.empty(wsb, dtype=torch.uint8, device=U.dev())) for _ in cases]

    def launch(case, o, stream):
        lg, tok, old, adv, w = case
        L.leap_grpo_logprob_loss_fwd_bwd(lg, V, N, V, tok, old, old, adv, w, p, o["lp"], None,
                                         None, o["loss"], o["dl"], o["ws"], wsb, None,
                                         stream=stream)

    U.log("fused calls one after the other, then overlapping on two streams")
    seq = outputs()
    for c, o in zip(cases, seq):
        launch(c, o, torch.cuda.current_stream())
    torch.cuda.synchronize()
    par = outputs()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        for c, o, s in zip(cases, par, streams):
            launch(c, o, s)
    torch.cuda.synchronize()
    for a, b in zip(seq, par):
        assert torch.equal(a["dl"].view(torch.int16), b["dl"].view(torch.int16))
        assert torch.equal(a["lp"], b["lp"]) and torch.equal(a["loss"], b["loss"])


def test_grpo_all_masked_and_empty():
    N, V = 32, 1024
    lg, tok, old, ref = U.make_inputs_host(3, N, V)
    z = np.zeros(N, np.float32)
    gpu = U.run_grpo(U.bf16_device(lg), V, tok, old, ref, z, z, **KW)
    assert gpu["loss"] == 0.0 and np.all(gpu["logp"] == 0)
    assert np.all(U.dl_rows(gpu["dl_dev"], np.arange(N), V) == 0)
    import torch
    empty = torch.empty((0, V), dtype=torch.bfloat16, device=U.dev())
    e = U.run_grpo(empty, V, [], [], [], [], [], **KW)
    assert e["loss"] == 0.0


# ----------------------------------------------------------------------------
# Full-size microbatches (sampled rows), in the benchmark's configuration
# ----------------------------------------------------------------------------
def _full_size_case(name, mb_index, seed, layout="packed"):
    import torch
    lat, ro, mbs, tok_r, tok_t, A32 = _step_tokens(name, layout)
    mb = mbs[mb_index]
    V = lat.cfg["V"]
    N = mb.tok_rollout.size
    gamma = float(np.float32(lat.cfg["gamma"]))
    agg = oracle.AGG_SEQ_MEAN_TOKEN_MEAN
    adv, w, _ = oracle.token_advantages(A32.astype(np.float64), mb.tok_rollout, mb.tok_turn,
                                        ro.n_turns, ro.n_tokens, gamma, agg, float(ro.n_rollouts))
    U.log(f"{name} microbatch {mb_index}: generating {N}x{V} logits on the device")
    lg_dev = wl.logits_device(seed, N, V, device=U.dev())
    tok = wl.sample_tokens_device(lg_dev, V, seed).cpu().numpy()
    lg = lg_dev.view(torch.int16).cpu().numpy().view(np.uint16)
    U.log("oracle log-probs for the old / reference inputs")
    cur, bad = oracle.logprob_rows(lg, tok)
    assert bad == 0
    n_old, n_ref = wl.logp_noise(seed, N)
    old = (cur + n_old).astype(np.float32)
    ref = (cur + n_ref).astype(np.float32)
    return lg_dev, lg, tok, old, ref, adv.astype(np.float32), w.astype(np.float32), V, N


@pytest.mark.parametrize("name,mb_index,layout", [
    ("mid", 0, "packed"), ("mid", -1, "packed"), ("full", 0, "packed"),
    ("mid", 5, "right_padded"),  # three 2304-row slots and a 1280-row tail
    ("full", -1, "right_padded"),  # one 11840-row slot holding the step's last sequence
])
def test_grpo_full_size_microbatch(name, mb_index, layout):
    import torch
    seed = 4242 + (mb_index % 7) + (100 if layout != "packed" else 0)
    lg_dev, lg, tok, old, ref, adv, w, V, N = _full_size_case(name, mb_index, seed, layout)
    valid = w != 0
    rng = np.random.default_rng(seed)
    sample = np.unique(np.concatenate([rng.choice(np.flatnonzero(valid), 24, replace=False),
                                       rng.choice(N, 8, replace=False), [0, N - 1]]))
    # (1) the configuration the benchmark runs: sample-level weights
    U.log(f"{name}[{mb_index}] {layout}: {int(valid.sum())} of {N} rows live; GPU run, default weights")
    gpu = U.run_grpo(lg_dev, V, tok, old, ref, adv, w, **KW)
    U.log("oracle over every row (log-probs and loss)")
    o = oracle.grpo_rows(lg, tok, old, ref, adv, w, want_dlogits=False, **KW)
    _check_rows(gpu, o, valid, name)
    U.check_dlogits(U.dl_rows(gpu["dl_dev"], sample, V), lg, sample, tok, old, ref, adv, w, V,
                    atol=1e-2, kw=KW, rel_to_max=True)
    # every excluded row (feedback, slot and tail padding) is written as zeros
    masked = torch.as_tensor(np.flatnonzero(~valid), device=lg_dev.device)
    if masked.numel():
        assert int(gpu["dl_dev"].index_select(0, masked).view(torch.int16).abs().max().item()) == 0
    del gpu
    torch.cuda.empty_cache()
    # (2) unit weights, where a 2e-2 absolute bound on dlogits is meaningful
    w1 = valid.astype(np.float32)
    U.log(f"{name}[{mb_index}] GPU run, unit weights")
    gpu1 = U.run_grpo(lg_dev, V, tok, old, ref, adv, w1, want_tok_loss=False, **KW)
    U.check_dlogits(U.dl_rows(gpu1["dl_dev"], sample, V), lg, sample, tok, old, ref, adv, w1, V,
                    atol=2e-2, kw=KW)
    assert gpu1["bad"] == 0


# ----------------------------------------------------------------------------
# Optional per-token entropy output of the fused call
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("V,N,inv_temp", [(1000, 64, 1.0), (5000, 32, 0.7), (32768, 64, 1.0),
                                          (151936, 24, 1.0), (151936, 8, 1.3), (200003, 8, 1.0)])
def test_grpo_entropy_output(V, N, inv_temp):
    import torch
    rng = np.random.default_rng(V + N)

    def edit(lg, tok):
        lg[1, ::7] = 0xFF80  # -inf columns
        tok[1] = 3
        tok[2] = V  # out of range: counted, excluded

    ld = (V + 7) // 8 * 8
    lg, tok, old, ref = U.make_inputs_host(V + 3, N, V, ld=ld, edit=edit)
    adv = rng.normal(0, 1, N).astype(np.float32)
    w = rng.choice([0.0, 1.0], N, p=[0.25, 0.75]).astype(np.float32)
    w[:3] = 1.0
    kw = dict(KW, inv_temp=inv_temp)
    U.log(f"grpo entropy V={V} N={N} T^-1={inv_temp}")
    lg_dev = U.bf16_device(lg)
    a = U.run_grpo(lg_dev, V, tok, old, ref, adv, w, want_entropy=True, **kw)
    b = U.run_grpo(lg_dev, V, tok, old, ref, adv, w, **kw)
    # requesting the entropy changes no other output
    assert torch.equal(a["dl_dev"].view(torch.int16), b["dl_dev"].view(torch.int16))
    assert np.array_equal(a["logp"], b["logp"]) and a["loss"] == b["loss"]
    assert a["bad"] == b["bad"] == 1
    h, bad = oracle.entropy_rows(lg, V=V, inv_temp=inv_temp)
    assert bad == 0
    valid = (w != 0) & (tok >= 0) & (tok < V)
    assert np.all(a["entropy"][~valid] == 0)
    np.testing.assert_allclose(a["entropy"][valid], h[valid], rtol=1e-4, atol=2e-4)
