"""The peak probes compute what include/bitlogic.h specifies: the VALU probe's
per-lane words against a numpy model of its multiplexer chains, and the copy
probe byte for byte."""
import numpy as np
import pytest
import torch

from paper_2602_07400_amd import bitlogic as bl

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
M32 = np.uint64(0xFFFFFFFF)


def valu_model(blocks, iters, seed):
    lane = np.arange(blocks * bl.PROBE_THREADS, dtype=np.uint64)
    a = [(((lane + 1) * np.uint64(0x9E3779B1)) ^ ((np.uint64((seed + c) & 0xFFFFFFFF)
                                                   * np.uint64(0x85EBCA77)))) & M32
         for c in range(bl.PROBE_CHAINS)]
    for _ in range(iters):
        for c in range(bl.PROBE_CHAINS):
            s = a[(c + 1) % bl.PROBE_CHAINS]
            a[c] = ((s & a[c]) | (~s & M32 & a[(c + 2) % bl.PROBE_CHAINS])) & M32
    r = np.zeros_like(lane)
    for v in a:
        r ^= v
    return r.astype(np.uint32)


@pytest.mark.parametrize("blocks,iters,seed", [(1, 0, 0), (2, 1, 5), (3, 37, 123456789),
                                               (1, 64, 0xFFFFFFFF)])
def test_valu_probe_matches_model(blocks, iters, seed):
    out = torch.empty(blocks * bl.PROBE_THREADS, dtype=torch.int32, device=DEV)
    ops = bl.bitlogic_probe_valu(out, blocks, iters, seed)
    torch.cuda.synchronize()
    assert ops == blocks * 256 * iters * 8
    got = out.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, valu_model(blocks, iters, seed))


@pytest.mark.parametrize("nbytes", [0, 16, 4096 + 48, (1 << 22) + 16 * 1001])
def test_copy_probe_copies(nbytes):
    rng = np.random.default_rng(nbytes)
    src = torch.from_numpy(rng.integers(0, 256, size=nbytes, dtype=np.uint8)).to(DEV)
    dst = torch.zeros(nbytes, dtype=torch.uint8, device=DEV)
    moved = bl.bitlogic_probe_copy(src, dst)
    torch.cuda.synchronize()
    assert moved == 2 * nbytes
    assert torch.equal(src, dst)
