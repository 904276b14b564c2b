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


# ------------------------------------------------------ instruction-rate probe

def valu_op_model(op, blocks, seed):
    lane = np.arange(blocks * bl.PROBE_THREADS, dtype=np.uint64)
    c0 = (((lane + 1) * np.uint64(0x9E3779B1)) & M32) ^ np.uint64(seed & 0xFFFFFFFF)
    s = (c0 * np.uint64(0x85EBCA77)) & M32
    z = ~c0 & M32
    if op == bl.PROBE_OP_BFE:
        c = np.where((s >> np.uint64(5)) & np.uint64(1), M32, np.uint64(0))
    else:
        c = (s & c0) | (~s & M32 & z)
    return ((np.uint64(8) * c) & M32).astype(np.uint32)


@pytest.mark.parametrize("op", [bl.PROBE_OP_MUX, bl.PROBE_OP_MUX_BANK, bl.PROBE_OP_BFE])
@pytest.mark.parametrize("blocks,iters,seed", [(1, 1, 0), (3, 5, 0xDEADBEEF)])
def test_valu_op_probe_matches_model(op, blocks, iters, seed):
    out = torch.empty(blocks * bl.PROBE_THREADS, dtype=torch.int32, device=DEV)
    n = bl.bitlogic_probe_valu_op(op, out, blocks, iters, seed)
    torch.cuda.synchronize()
    assert n == blocks * 4 * iters * 64
    assert np.array_equal(out.cpu().numpy().view(np.uint32), valu_op_model(op, blocks, seed))


# ------------------------------------------------------------- gather probe

def probe_row(seed, x):
    y = ((np.uint64(x) ^ np.uint64(seed)) * np.uint64(0x9E3779B1)) & M32
    return int(y ^ (y >> np.uint64(16)))


def gather_model(rows, lpr, blocks, passes, seed):
    """rows uint32 [n_rows][32] -> (out [blocks*256], sink pieces dict)."""
    n_rows = rows.shape[0]
    pieces = rows.reshape(n_rows, 8, 4)
    out = np.zeros(blocks * 256, np.uint32)
    sink = np.zeros((blocks * passes * 4 * 128, 4), np.uint32)
    for b in range(blocks):
        for t in range(256):
            w, l = t // 64, t % 64
            acc = np.zeros(4, np.uint32)
            for p in range(passes):
                j0 = (b * passes + p) * 64 + w * 16
                got = []
                if lpr == 4:
                    j, q = j0 + l // 4, l % 4
                    for i in range(6):
                        r = probe_row(seed, 6 * j + i) % n_rows
                        got += [pieces[r, 2 * q], pieces[r, 2 * q + 1]]
                else:
                    for h in range(2):
                        for i in range(6):
                            j = j0 + h * 8 + l // 8
                            r = probe_row(seed, 6 * j + i) % n_rows
                            got.append(pieces[r, l % 8])
                for g in got:
                    acc ^= g
                base = ((b * passes + p) * 4 + w) * 128 + 2 * l
                sink[base], sink[base + 1] = got[0], got[1]
            out[t + 256 * b] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3]
    return out, sink


@pytest.mark.parametrize("lpr", [4, 8])
@pytest.mark.parametrize("valu", [0, 512])
@pytest.mark.parametrize("n_rows,blocks,passes,occ", [(37, 2, 3, 0), (1000, 1, 2, 4)])
def test_gather_probe_matches_model(lpr, valu, n_rows, blocks, passes, occ):
    rng = np.random.default_rng(n_rows + lpr + valu)
    host = rng.integers(0, 2**32, size=(n_rows, 32), dtype=np.uint32)
    rows = torch.from_numpy(host.view(np.int32)).to(DEV)
    out = torch.empty(blocks * 256, dtype=torch.int32, device=DEV)
    sink = torch.zeros(blocks * passes * 8192 // 4, dtype=torch.int32, device=DEV)
    n = bl.bitlogic_probe_gather(rows, lpr, valu, blocks, passes, out, sink, waves_per_simd=occ,
                                 seed=12345)
    torch.cuda.synchronize()
    assert n == blocks * passes * 64 * 6
    ref_out, ref_sink = gather_model(host, lpr, blocks, passes, 12345)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref_out)
    assert np.array_equal(sink.cpu().numpy().view(np.uint32).reshape(-1, 4), ref_sink)
