"""The measurement helpers on the GPU: the HBM probe copies, reads and
writes what it is asked to; the MFMA probe runs every round of every chain
(with ones its sink holds iters * 32, the sum of 32 products of ones per
MFMA) and, with random operands, multiplies the hashed values it states.

The random-operand check recomputes, on the host, element (0, 0) of each
chain's product in wave 0 of each workgroup: row 0 of A and column 0 of B
lie in lanes 0, 16, 32 and 48 (lane % 16 is the row of A and the column of
B), and both operands use one k order inside a lane, so the element is the
sum over those lanes of the lane-wise dot products whatever that order is.
Products of two bf16 of magnitude [1, 2) are multiples of 2^-14 below 4,
so each chain's element stays exact in fp32 for a few rounds (under 2^24
units of 2^-14); the sum over the chains is rounded in fp32 in the same
order on both sides, so the host reproduces the sink bit for bit."""
import numpy as np
import pytest

from tests import _gpu_util as U

pytestmark = pytest.mark.gpu


def test_hbm_probe_modes():
    import torch
    from paper_2608_01804_amd import leap as L
    n = 3 << 20
    a = torch.arange(n // 4, dtype=torch.int32, device=U.dev())
    b = torch.full_like(a, -1)
    L.leap_probe_hbm(a, b, n, 0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    L.leap_probe_hbm(None, b, n, 2)
    torch.cuda.synchronize()
    assert int(b.abs().max().item()) == 0
    L.leap_probe_hbm(a, b, n, 1)  # read only: b untouched past its first 16 bytes
    torch.cuda.synchronize()
    assert int(b[4:].abs().max().item()) == 0


@pytest.mark.parametrize("iters,wgs", [(1, 1), (1000, 37), (100000, 1024)])
def test_mfma_probe_runs_every_round(iters, wgs):
    import torch
    from paper_2608_01804_amd import leap as L
    sink = torch.full((wgs,), float("nan"), dtype=torch.float32, device=U.dev())
    L.leap_probe_mfma(iters, wgs, sink)
    torch.cuda.synchronize()
    assert np.all(sink.cpu().numpy() == np.float32(iters * 32))


def _fmix32(h):
    # MurmurHash3's 32-bit finaliser, on uint64 arrays masked to 32 bits
    m = np.uint64(0xFFFFFFFF)
    h = h & m
    h ^= h >> np.uint64(16)
    h = (h * np.uint64(0x85EBCA6B)) & m
    h ^= h >> np.uint64(13)
    h = (h * np.uint64(0xC2B2AE35)) & m
    h ^= h >> np.uint64(16)
    return h


def _random_operand(seed):
    """The eight bf16 values (as float64) of the probe's operand `seed`:
    four hashed words, each two bf16 of magnitude [1, 2) with hashed sign and
    mantissa, low half first."""
    seed = np.asarray(seed, np.uint64)
    vals = []
    for i in range(4):
        h = _fmix32(seed * np.uint64(4) + np.uint64(i))
        for half in (h & np.uint64(0xFFFF), h >> np.uint64(16)):
            bits = (np.uint64(0x3F80) | (half & np.uint64(0x807F))) << np.uint64(16)
            vals.append(bits.astype(np.uint32).view(np.float32).astype(np.float64))
    return np.stack(vals, axis=-1)


@pytest.mark.parametrize("iters,wgs", [(1, 5), (3, 300)])
def test_mfma_probe_random_operands(iters, wgs):
    import torch
    from paper_2608_01804_amd import leap as L
    sink = torch.full((wgs,), float("nan"), dtype=torch.float32, device=U.dev())
    L.leap_probe_mfma(iters, wgs, sink, random_operands=1)
    torch.cuda.synchronize()
    got = sink.cpu().numpy()
    chains, block = 8, 256
    want = np.zeros(wgs, np.float32)
    for g in range(wgs):
        v = None
        for c in range(chains):
            lanes = np.array([0, 16, 32, 48], np.uint64)
            base = ((np.uint64(g * block) + lanes) * np.uint64(chains) + np.uint64(c)) * 2
            a = _random_operand(base)
            b = _random_operand(base + np.uint64(1))
            d = np.float32(iters * float((a * b).sum()))  # exact: see the module docstring
            v = d if v is None else np.float32(v + d)
        want[g] = v
    assert np.all(np.isfinite(got))
    np.testing.assert_array_equal(got, want)
