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
