"""The step's calls under HIP graph capture: the library allocates nothing,
never synchronises and issues no memset, so one step (gate, tournament,
token advantages, fused objective per microbatch) can be captured once and
replayed.  Every replay, with eager work and synchronisations between
replays, must reproduce the eager step bit for bit."""
import pytest

pytestmark = pytest.mark.gpu


def test_step_graph_replays_match_eager():
    import torch

    import bench
    from paper_2608_01804_amd import leap as L
    from tests import _gpu_util as U

    L.lib()
    dev = torch.device("cuda:0")
    U.log("graph: building the 2048-row step (V = 32768)")
    s = bench.build_step(L, torch, dev, "tiny", 1001)
    names = ("n_fail", "gate", "reward", "adv_roll", "adv_tok", "w_tok", "loss", "dlogits")

    def snapshot():
        return [s[k].clone() for k in names]

    def scramble():
        for k in ("reward", "adv_roll", "adv_tok", "w_tok", "loss", "dlogits"):
            s[k].fill_(float("nan"))
        s["gate"].fill_(7)
        s["n_fail"].fill_(-1)

    bench.run_step(L, s)
    torch.cuda.synchronize()
    eager = snapshot()
    assert int(s["err"].item()) == 0

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        bench.run_step(L, s)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    U.log("graph: capturing one step")
    with torch.cuda.graph(g):
        bench.run_step(L, s)
    torch.cuda.synchronize()

    for rep in range(3):
        scramble()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, a, b in zip(names, eager, snapshot()):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (rep, k)
        U.log(f"graph: replay {rep} matches the eager step")
    assert int(s["err"].item()) == 0


@pytest.mark.parametrize("prepared", [False, True])
def test_lmhead_graph_replays_match_eager(prepared):
    """The fused LM-head call under capture: its GEMM extents come from a
    live-row count the call itself writes on the device, so replays with a
    scrambled workspace and outputs in between must still reproduce the
    eager call bit for bit (with the call's own weight transpose, and with
    a transposed weight prepared outside the graph)."""
    import torch

    from paper_2608_01804_amd import leap as L
    from tests import _gpu_util as U

    L.lib()
    N, V, H = 700, 3000, 128
    U.log(f"graph: lmhead N={N} V={V} H={H} prepared={prepared}")
    inp = U.lmhead_inputs(3501, N, V, H, mask_frac=0.3)
    dev = U.dev()
    T = U.T
    y, old, ref, adv, w = T(inp["y"]), T(inp["old"]), T(inp["ref"]), T(inp["adv"]), T(inp["w"])
    logp = torch.empty(N, dtype=torch.float32, device=dev)
    tl = torch.empty(N, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dH = torch.empty((N, H), dtype=torch.float32, device=dev)
    dW = torch.empty((V, H), dtype=torch.float32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ws_bytes = L.leap_lmhead_workspace_size(N, V, H)
    w_t = None
    if prepared:
        nb = L.leap_lmhead_weight_t_size(V, H)
        w_t = torch.empty(nb, dtype=torch.uint8, device=dev)
        L.leap_lmhead_transpose_weight(inp["wt"], V, H, w_t, nb)
        ws_bytes -= nb
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    p = L.leap_grpo_params(0.2, 0.28, 0.01, L.LEAP_KL_K3, 1.0)
    outs = (logp, tl, loss, dH, dW)

    def call():
        L.leap_grpo_lmhead_fwd_bwd(inp["hid"], inp["wt"], N, V, H, y, old, ref, adv, w, p, logp, tl,
                                   loss, dH, dW, 0, ws, ws_bytes, err, weight_t=w_t)

    def scramble():
        for t in outs:
            t.fill_(float("nan"))
        ws.fill_(0xA5)

    scramble()
    call()
    torch.cuda.synchronize()
    eager = [t.clone() for t in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for rep in range(3):
        scramble()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(eager, outs)):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (rep, i)
        U.log(f"graph: lmhead replay {rep} matches the eager call")
    assert int(err.item()) == 0
