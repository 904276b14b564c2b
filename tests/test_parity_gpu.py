"""Bit-exact parity of the HIP path (through the C ABI) with the CPU oracle.

Per-kernel cases cover every fan-in, ragged word counts (the tail window),
odd word counts and 8-byte-only alignment (the 8-byte access path), node
counts that are not whole node blocks, repeated connection indices, junk
table bits above 2^k, threshold edge values, unaligned pixel rows, and head
groups from 1 node to thousands (split counters).  Whole-network cases run
every configuration at a reduced batch (several windows plus a ragged tail)
and at its full batch, every sample against the oracle.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import CONFIG_ORDER, CONFIGS, make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def unpack(bits: torch.Tensor, n: int) -> np.ndarray:
    """int64 [rows][W] packed bits -> uint8 [n][rows] (bit s%64 of word s/64)."""
    b = bits.cpu().numpy().view(np.uint8)                  # [rows][W*8], little-endian
    v = np.unpackbits(b, axis=1, bitorder="little")        # [rows][W*64]
    return np.ascontiguousarray(v[:, :n].T)


def pack(v: np.ndarray) -> torch.Tensor:
    """uint8 [n][rows] (0/1) -> int64 [rows][ceil(n/64)] on the GPU."""
    n, rows = v.shape
    W = (n + 63) // 64
    buf = np.zeros((rows, W * 8), dtype=np.uint8)
    p = np.packbits(v.T, axis=1, bitorder="little")
    buf[:, :p.shape[1]] = p
    return torch.from_numpy(buf.view(np.int64).copy()).to(DEV)


def to_dev(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _report(name, got, ref):
    bad = np.argwhere(got != ref)
    return f"{name}: {len(bad)} mismatches, first {bad[:5].tolist()}"


# ------------------------------------------------------------------ encoder

ENC_CASES = [
    # n, d, b, threshold kind
    (64, 4, 1, "random"),
    (64 * 3 + 5, 37, 3, "random"),          # ragged samples, d % 4 != 0 (byte path)
    (4096 + 17, 784, 1, "128"),
    (1000, 100, 7, "edges"),                 # 0 / 255 / duplicates / unsorted
    (2048, 3072, 3, "random"),
    (777, 33, 64, "random"),                 # b at its maximum
    (64 * 16 * 2, 64, 8, "zero"),            # the quantile collapse: all thresholds 0
    (64 * 16 + 3, 96, 7, "random"),          # 32-feature tiles read as 16-byte pieces
    (64 * 5, 200, 3, "random"),              # 64-feature tiles, ragged last tile
]


@pytest.mark.parametrize("n,d,b,kind", ENC_CASES)
def test_encode_parity(n, d, b, kind):
    rng = np.random.default_rng(n * 131 + d * 7 + b)
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    x[: min(n, 5)] = 0
    x[min(n, 5): min(n, 9)] = 255
    if kind == "128":
        th = np.full((d, b), 128, np.uint8)
    elif kind == "edges":
        th = rng.choice(np.array([0, 255, 128, 128, 1, 254], np.uint8), size=(d, b))
    elif kind == "zero":
        th = np.zeros((d, b), np.uint8)
    else:
        th = rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    bits = bl.bitlogic_encode(to_dev(x), to_dev(th))
    torch.cuda.synchronize()
    got = unpack(bits, bits.shape[1] * 64)
    ref = oracle.encode(x, th)
    assert np.array_equal(got[:n], ref), _report("encode", got[:n], ref)
    assert not got[n:].any(), "padding bits must be 0"


@pytest.mark.parametrize("b", [3, 7, 8])
def test_encode_dword_aligned_rows(b):
    """Rows 4-byte but not 16-byte aligned take the dword loads, not the
    16-byte ones."""
    rng = np.random.default_rng(50 + b)
    n, d = 64 * 16 + 9, 128
    big = rng.integers(0, 256, size=n * d + 16, dtype=np.uint8)
    xt = to_dev(big)[4:4 + n * d].view(n, d)
    assert xt.data_ptr() % 4 == 0 and xt.data_ptr() % 16 != 0
    th = rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    bits = bl.bitlogic_encode(xt, to_dev(th))
    ref = oracle.encode(big[4:4 + n * d].reshape(n, d), th)
    assert np.array_equal(unpack(bits, n), ref)


def test_encode_unaligned_rows():
    """Pixels whose base address is not 4-byte aligned take the byte path."""
    rng = np.random.default_rng(5)
    n, d, b = 300, 40, 3
    big = rng.integers(0, 256, size=(n + 1) * d + 1, dtype=np.uint8)
    xt = to_dev(big)[1:1 + n * d].view(n, d)
    assert xt.data_ptr() % 4 != 0
    th = rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    bits = bl.bitlogic_encode(xt, to_dev(th))
    ref = oracle.encode(big[1:1 + n * d].reshape(n, d), th)
    assert np.array_equal(unpack(bits, n), ref)


# ---------------------------------------------------------------- LUT layer

LAYER_CASES = [
    # n_words, w_in, w_out, k, repeats
    (1, 6, 1, 6, False),
    (4, 7, 5, 3, True),              # tail window only
    (16, 100, 256, 6, False),        # exactly one window, one node block
    (16 * 3 + 5, 1000, 300, 6, False),   # full windows + tail; partial node block
    (33, 64, 70, 4, True),           # odd word count: 8-byte path
    (64, 300, 513, 5, False),
    (40, 50, 64, 1, True),
    (40, 50, 64, 2, False),
    (128, 21504, 1000, 6, False),    # C4-shaped input width
]


@pytest.mark.parametrize("n_words,w_in,w_out,k,repeats", LAYER_CASES)
def test_lut_layer_parity(n_words, w_in, w_out, k, repeats):
    rng = np.random.default_rng(n_words * 1009 + w_in + k)
    n = n_words * 64
    v = rng.integers(0, 2, size=(n, w_in), dtype=np.uint8)
    if repeats:
        conn = rng.integers(0, w_in, size=(w_out, k)).astype(np.int32)
        conn[: w_out // 2, :min(k, 2)] = conn[: w_out // 2, :1]
    else:
        conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w_out)]
                        ).astype(np.int32)
    tables = rng.integers(0, np.iinfo(np.uint64).max, size=w_out, dtype=np.uint64,
                          endpoint=True)   # junk above 2^k for k < 6 must be ignored
    out = bl.bitlogic_lut_layer(pack(v), to_dev(conn), to_dev(tables))
    ref = oracle.lut_layer(v, conn, tables)
    got = unpack(out, n)
    assert np.array_equal(got, ref), _report("lut_layer", got, ref)


def test_lut_layer_8byte_alignment_path():
    """Buffers that are 8- but not 16-byte aligned use 8-byte accesses."""
    rng = np.random.default_rng(17)
    n_words, w_in, w_out, k = 48, 90, 130, 6
    n = n_words * 64
    v = rng.integers(0, 2, size=(n, w_in), dtype=np.uint8)
    packed = pack(v)
    big_in = torch.zeros(w_in * n_words + 1, dtype=torch.int64, device=DEV)
    big_in[1:] = packed.reshape(-1)
    bits_in = big_in[1:].view(w_in, n_words)
    big_out = torch.zeros(w_out * n_words + 1, dtype=torch.int64, device=DEV)
    bits_out = big_out[1:].view(w_out, n_words)
    assert bits_in.data_ptr() % 16 == 8
    conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w_out)]).astype(np.int32)
    tables = rng.integers(0, 1 << 63, size=w_out).astype(np.uint64)
    bl.bitlogic_lut_layer(bits_in, to_dev(conn), to_dev(tables), bits_out=bits_out)
    assert np.array_equal(unpack(bits_out, n), oracle.lut_layer(v, conn, tables))
    assert big_out[0].item() == 0


def test_lut_layer_projection_tables():
    """Closed-form projection tables reproduce their input wires on the GPU."""
    rng = np.random.default_rng(3)
    n_words, w_in = 20, 64
    v = rng.integers(0, 2, size=(n_words * 64, w_in), dtype=np.uint8)
    bits_in = pack(v)
    proj = [0xAAAAAAAAAAAAAAAA, 0xCCCCCCCCCCCCCCCC, 0xF0F0F0F0F0F0F0F0,
            0xFF00FF00FF00FF00, 0xFFFF0000FFFF0000, 0xFFFFFFFF00000000]
    conn = np.stack([rng.choice(w_in, size=6, replace=False) for _ in range(6)]).astype(np.int32)
    tables = np.array(proj, dtype=np.uint64)
    out = bl.bitlogic_lut_layer(bits_in, to_dev(conn), to_dev(tables))
    got = out.cpu().numpy()
    ref_in = bits_in.cpu().numpy()
    for i in range(6):
        assert np.array_equal(got[i], ref_in[conn[i, i]])


# --------------------------------------------------------------------- head

HEAD_CASES = [
    # n, c, g, density
    (64, 1, 1, 0.5),
    (100, 3, 5, 0.5),          # g < 8: ripple-only counter
    (4096 + 33, 10, 100, 0.5),
    (2048, 100, 64, 0.5),
    (700, 10, 6400, 0.5),      # long groups, split counters
    (1000, 7, 1000, 0.0),      # all zero: every class ties at 0 -> argmax 0
    (1000, 7, 1000, 1.0),      # all one: ties at g -> argmax 0
    (1500, 10, 3200, 0.5),
    (128, 4, 65535, 0.02),      # the largest group size
    (200, 129, 40, 0.5),       # a second chunk of one class in the finish
    (100, 300, 7, 0.5),        # three chunks
    (70, 1000, 2, 0.5),        # many classes of two nodes
]


@pytest.mark.parametrize("n,c,g,density", HEAD_CASES)
def test_head_parity(n, c, g, density):
    rng = np.random.default_rng(n + c * 31 + g)
    w = c * g
    v = (rng.random((n, w), dtype=np.float32) < density).astype(np.uint8)
    bits = pack(v)
    scores, argmax = bl.bitlogic_groupsum_head(bits, n, c)
    ref_s, ref_p = oracle.groupsum(v, c)
    got_s, got_p = scores.cpu().numpy(), argmax.cpu().numpy()
    assert np.array_equal(got_s, ref_s), _report("scores", got_s, ref_s)
    assert np.array_equal(got_p, ref_p), _report("argmax", got_p, ref_p)


def test_head_argmax_only_and_padding_ignored():
    rng = np.random.default_rng(8)
    n, c, g = 130, 5, 40
    v = rng.integers(0, 2, size=(n, c * g), dtype=np.uint8)
    bits = pack(v)
    # set every padding bit: the head must ignore samples >= n
    W = bits.shape[1]
    pad = np.zeros((W * 64, c * g), np.uint8)
    pad[:n] = v
    pad[n:] = 1
    bits = pack(pad)
    _, argmax = bl.bitlogic_groupsum_head(bits, n, c, want_scores=False)
    assert np.array_equal(argmax.cpu().numpy(), oracle.groupsum(v, c)[1])


# ------------------------------------------------------------ whole network

def _check_forward(wl, idx=None):
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    x = torch.from_numpy(wl.x).to(DEV)
    scores, argmax = model.forward(x)
    torch.cuda.synchronize()
    got_s, got_p = scores.cpu().numpy(), argmax.cpu().numpy()
    if idx is None:
        ref_s, ref_p = oracle.forward(wl.x, wl.thresholds, wl.layers, wl.n_classes)
        sel = slice(None)
    else:
        ref_s, ref_p = oracle.forward(wl.x[idx], wl.thresholds, wl.layers, wl.n_classes)
        sel = idx
    assert np.array_equal(got_s[sel], ref_s), _report("scores", got_s[sel], ref_s)
    assert np.array_equal(got_p[sel], ref_p), _report("argmax", got_p[sel], ref_p)
    return got_s, got_p


@pytest.mark.parametrize("name", CONFIG_ORDER)
def test_forward_reduced_batch(name):
    # several 16-word windows plus a ragged last word
    wl = make_workload(name, seed=0, n=64 * 16 * 2 + 64 * 3 + 17)
    _check_forward(wl)


@pytest.mark.parametrize("name", CONFIG_ORDER)
def test_forward_full_batch(name):
    # every sample of the configuration's full batch against the oracle
    # (App. C.1 "Correctness anchor": the packed path equals the per-sample one)
    cfg = CONFIGS[name]
    wl = make_workload(name, seed=0)
    assert wl.n == cfg.n
    print(f"[full] {name}: n={cfg.n}, every sample", flush=True)
    _check_forward(wl)


def test_forward_hidden_layers_with_partial_node_blocks():
    # hidden layers of up to 4 inputs in the 512-node-block mode (>= 2048
    # blocks) whose widths are not whole blocks, so that every layer runs
    # both loops: the whole blocks gather all passes before storing any (the
    # depth ahead differs per fan-in: all passes at k <= 2, 10 at k = 3, 4 at
    # k = 4), the last block runs the two-register-set loop.  8096 nodes at
    # k = 4 leave a last block of 13 passes (an odd count: that loop ends on
    # its first set); 8100 nodes at k = 2 leave 14 passes whose last holds 4
    # nodes and 28 padding lanes; 4700 at k = 3 and 4300 at k = 1 leave 92
    # and 204 nodes.
    rng = np.random.default_rng(31)
    n, d, b = 1 << 18, 784, 2
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b), dtype=np.uint8), axis=1)
    layers, w_in = [], d * b
    for w, k in ((8096, 4), (8100, 2), (4700, 3), (4300, 1), (8000, 6)):
        conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)]).astype(np.int32)
        tab = rng.integers(0, 2**64, size=w, dtype=np.uint64)
        layers.append((conn, tab))
        w_in = w
    model = bl.BitlogicModel.from_numpy(th, layers, 10, device=DEV)
    xd = torch.from_numpy(x).to(DEV)
    scores, argmax = model.forward(xd)
    torch.cuda.synchronize()
    ref_s, ref_p = oracle.forward(x, th, layers, 10)
    got_s, got_p = scores.cpu().numpy(), argmax.cpu().numpy()
    assert np.array_equal(got_s, ref_s), _report("scores", got_s, ref_s)
    assert np.array_equal(got_p, ref_p), _report("argmax", got_p, ref_p)


def test_forward_matches_staged_calls_and_is_deterministic():
    wl = make_workload("c3_cifar10", seed=3, n=5000)
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    x = torch.from_numpy(wl.x).to(DEV)
    s1, p1 = model.forward(x)
    s2, p2 = model.forward(x)
    bits = bl.bitlogic_encode(x, model.thresholds)
    for conn, tab in model.layers:
        bits = bl.bitlogic_lut_layer(bits, conn, tab)
    s3, p3 = bl.bitlogic_groupsum_head(bits, wl.n, wl.n_classes)
    assert torch.equal(s1, s2) and torch.equal(p1, p2)
    assert torch.equal(s1, s3) and torch.equal(p1, p3)


def test_forward_single_layer_and_deep_stack():
    rng = np.random.default_rng(12)
    n, d, b = 1500, 50, 2
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    widths, ks = [120, 90, 60, 40, 30], [6, 5, 4, 3, 2]
    layers, w_in = [], d * b
    for w, k in zip(widths, ks):
        conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)]).astype(np.int32)
        layers.append((conn, rng.integers(0, 1 << 63, size=w).astype(np.uint64)))
        w_in = w
    for L, c in ((1, 6), (5, 3)):
        m = bl.BitlogicModel.from_numpy(th, layers[:L], c, device=DEV)
        s, p = m.forward(torch.from_numpy(x).to(DEV))
        rs, rp = oracle.forward(x, th, layers[:L], c)
        assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(p.cpu().numpy(), rp)


def test_forward_on_side_stream():
    wl = make_workload("c1_mnist_tiny", seed=4, n=1000)
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    x = torch.from_numpy(wl.x).to(DEV)
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        s, p = model.forward(x)
    st.synchronize()
    rs, rp = oracle.forward(wl.x, wl.thresholds, wl.layers, wl.n_classes)
    assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(p.cpu().numpy(), rp)


@pytest.mark.parametrize("n,d,b", [(64 * 4 * 3 + 77, 30, 10), (1000, 13, 64), (300, 7, 8)])
def test_forward_encoder_variants(n, d, b):
    """b > 8 takes the ballot encoder; d % 4 != 0 takes the byte-staging path."""
    rng = np.random.default_rng(n + d + b)
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    layers, w_in = [], d * b
    for w, k in ((200, 6), (120, 4)):
        conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)]).astype(np.int32)
        layers.append((conn, rng.integers(0, 1 << 63, size=w).astype(np.uint64)))
        w_in = w
    m = bl.BitlogicModel.from_numpy(th, layers, 6, device=DEV)
    s, p = m.forward(torch.from_numpy(x).to(DEV))
    rs, rp = oracle.forward(x, th, layers, 6)
    assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(p.cpu().numpy(), rp)


def test_forward_timed_records_stage_events():
    wl = make_workload("c3_cifar10", seed=5, n=3000)
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    x = torch.from_numpy(wl.x).to(DEV)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(wl.layers) + 3)]
    for e in ev:
        e.record()
    s1, p1 = bl.bitlogic_forward_timed(x, model.thresholds, model.layers, model.n_classes, ev)
    torch.cuda.synchronize()
    times = [ev[i].elapsed_time(ev[i + 1]) for i in range(len(ev) - 1)]
    assert all(t >= 0 for t in times) and sum(times) > 0
    s2, p2 = model.forward(x)
    assert torch.equal(s1, s2) and torch.equal(p1, p2)


@pytest.mark.parametrize("g,c,k,n", [(32, 3, 6, 1000), (96, 5, 4, 64 * 16 + 7), (736, 2, 6, 2500),
                                     (800, 4, 5, 64 * 16 * 3), (640, 7, 6, 3000), (64, 40, 2, 777)])
def test_forward_fused_head_matches_oracle_and_unfused(g, c, k, n, monkeypatch):
    """The last layer fused with the head gives the oracle's result, and the
    same result as the separate layer + head kernels."""
    rng = np.random.default_rng(g * 7 + c + k + n)
    d, b = 60, 3
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b)), axis=1).astype(np.uint8)
    w1, w2 = 500, g * c
    layers = []
    for w, w_in in ((w1, d * b), (w2, w1)):
        conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)]).astype(np.int32)
        layers.append((conn, rng.integers(0, 1 << 63, size=w).astype(np.uint64)))
    m = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV)
    xt = torch.from_numpy(x).to(DEV)
    s_f, p_f = m.forward(xt)
    monkeypatch.setenv("BITLOGIC_UNFUSED_HEAD", "1")
    s_u, p_u = m.forward(xt)
    monkeypatch.delenv("BITLOGIC_UNFUSED_HEAD")
    rs, rp = oracle.forward(x, th, layers, c)
    assert np.array_equal(s_f.cpu().numpy(), rs) and np.array_equal(p_f.cpu().numpy(), rp)
    assert torch.equal(s_f, s_u) and torch.equal(p_f, p_u)


@pytest.mark.parametrize("c,g", [(600, 2), (1000, 1)])
def test_forward_index_space_beyond_int32(c, g):
    """A 4M-sample batch with 600 or 1000 classes: scores hold n * c > 2^31
    entries (> 2^32 at 1000 classes), so every score index needs 64-bit
    arithmetic; the batch has a ragged tail.  The oracle checks sampled rows,
    the first and last ones included."""
    n, d, b = (1 << 22) + 37, 16, 2
    rng = np.random.default_rng(c + g)
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b), dtype=np.uint8), axis=1)
    layers, w_in = [], d * b
    for w, k in ((1500, 6), (c * g, 4)):
        conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)]).astype(np.int32)
        layers.append((conn, rng.integers(0, 1 << 63, size=w, dtype=np.int64).astype(np.uint64)))
        w_in = w
    model = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV)
    scores, argmax = model.forward(torch.from_numpy(x).to(DEV))
    torch.cuda.synchronize()
    assert scores.numel() > (1 << 31)
    idx = np.unique(np.concatenate([np.arange(64), np.arange(n - 101, n),
                                    rng.choice(n, size=800, replace=False)]))
    sel = torch.from_numpy(idx).to(DEV)
    got_s, got_p = scores[sel].cpu().numpy(), argmax[sel].cpu().numpy()
    ref_s, ref_p = oracle.forward(x[idx], th, layers, c)
    assert np.array_equal(got_s, ref_s), _report("scores", got_s, ref_s)
    assert np.array_equal(got_p, ref_p), _report("argmax", got_p, ref_p)
    del scores, argmax
    torch.cuda.empty_cache()
