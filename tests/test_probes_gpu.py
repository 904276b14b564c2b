"""The peak probes compute what include/bitlogic.h specifies: the VALU probe's
per-lane words against a numpy model of its multiplexer chains, and the HBM
streaming probes (copy, read with an XOR of the pieces, write of a pattern)
byte for byte."""
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


SIZES = [0, 16, 4096 + 48, (1 << 22) + 16 * 1001]


@pytest.mark.parametrize("unroll", [1, 2, 4, 8])
@pytest.mark.parametrize("nbytes", SIZES)
def test_hbm_copy_probe_copies(nbytes, unroll):
    rng = np.random.default_rng(nbytes + unroll)
    src = torch.from_numpy(rng.integers(0, 256, size=nbytes, dtype=np.uint8)).to(DEV)
    dst = torch.zeros(nbytes, dtype=torch.uint8, device=DEV)
    moved = bl.bitlogic_probe_hbm(bl.PROBE_HBM_COPY, src, dst, unroll=unroll)
    torch.cuda.synchronize()
    assert moved == 2 * nbytes
    assert torch.equal(src, dst)


@pytest.mark.parametrize("unroll,blocks", [(1, 0), (2, 3), (4, 0), (8, 1), (8, 5000)])
@pytest.mark.parametrize("nbytes", SIZES)
def test_hbm_read_probe_xors(nbytes, unroll, blocks):
    rng = np.random.default_rng(nbytes * 3 + unroll)
    host = rng.integers(0, 256, size=nbytes, dtype=np.uint8)
    src = torch.from_numpy(host).to(DEV)
    out = torch.full((16,), 0x5A, dtype=torch.uint8, device=DEV)     # cleared by the probe
    moved = bl.bitlogic_probe_hbm(bl.PROBE_HBM_READ, src if nbytes else out, out, nbytes,
                                  unroll=unroll, blocks=blocks)
    torch.cuda.synchronize()
    assert moved == nbytes
    ref = np.zeros(16, np.uint8)
    if nbytes:
        ref = np.bitwise_xor.reduce(host.reshape(-1, 16), axis=0)
    assert np.array_equal(out.cpu().numpy(), ref)


@pytest.mark.parametrize("unroll", [1, 8])
@pytest.mark.parametrize("nbytes", SIZES)
def test_hbm_write_probe_pattern(nbytes, unroll):
    dst = torch.zeros(nbytes + 16, dtype=torch.uint8, device=DEV)
    moved = bl.bitlogic_probe_hbm(bl.PROBE_HBM_WRITE, None, dst, nbytes, unroll=unroll)
    torch.cuda.synchronize()
    assert moved == nbytes
    got = dst.cpu().numpy()
    i = np.arange(nbytes // 16, dtype=np.uint64)
    lo, hi = (i & np.uint64(0xFFFFFFFF)).astype(np.uint32), (i >> np.uint64(32)).astype(np.uint32)
    ref = np.stack([lo, hi, ~lo, ~hi], axis=1).view(np.uint8).reshape(-1)
    assert np.array_equal(got[:nbytes], ref)
    assert not got[nbytes:].any()                  # nothing past the end
