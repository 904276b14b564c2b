"""C-ABI checks that need no GPU: the library loads, exports every function
include/bitlogic.h declares, and rejects bad arguments on the host before any
HIP call (so fake, never-dereferenced pointers are safe here)."""
import ctypes
import os
import re

import pytest

from paper_2602_07400_amd import bitlogic as bl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bitlogic.h")

# a non-NULL address that is never dereferenced (every call below fails its
# host-side checks first)
FAKE = 0x10000
OK, ENULL, ESHAPE, EALIGN, EUNSUP, EHIP, EWS = range(7)


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bitlogic_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    # the fake pointers below must never reach a device: if a check were
    # missing, a launch would dereference them
    import torch
    if torch.cuda.is_available():
        pytest.skip("fake-pointer argument checks run only where no GPU is visible")
    return bl.load_library()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"bitlogic_encode", "bitlogic_lut_layer", "bitlogic_groupsum_head",
            "bitlogic_forward"} <= set(names)
    raw = ctypes.CDLL(bl.library_path())
    for name in names:
        assert hasattr(raw, name), name


def test_status_strings(lib):
    for s in range(7):
        assert bl.bitlogic_status_string(s) and bl.bitlogic_status_string(s) != "unknown status"
    assert bl.bitlogic_status_string(99) == "unknown status"
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "bitlogic.h")).read()
    assert bl.bitlogic_version() == int(re.search(r"#define BITLOGIC_VERSION (\d+)", hdr).group(1))


def _err(lib):
    return lib.bitlogic_last_error().decode()


def test_encode_validation(lib):
    assert lib.bitlogic_encode(None, 64, 4, FAKE, 1, FAKE, None) == ENULL
    assert lib.bitlogic_encode(FAKE, -1, 4, FAKE, 1, FAKE, None) == ESHAPE
    assert lib.bitlogic_encode(FAKE, 64, 0, FAKE, 1, FAKE, None) == ESHAPE
    assert lib.bitlogic_encode(FAKE, 64, 4, FAKE, 0, FAKE, None) == ESHAPE
    assert lib.bitlogic_encode(FAKE, 64, 4, FAKE, 65, FAKE, None) == ESHAPE
    assert "b <= 64" in _err(lib)
    assert lib.bitlogic_encode(FAKE, 64, 4, FAKE, 1, FAKE + 4, None) == EALIGN
    # n = 0 is valid and enqueues nothing
    assert lib.bitlogic_encode(FAKE, 0, 4, FAKE, 1, FAKE, None) == OK
    assert _err(lib) == ""


@pytest.mark.parametrize("k", [0, 7, -1])
def test_layer_rejects_fan_in(lib, k):
    assert lib.bitlogic_lut_layer(FAKE, 10, 4, FAKE, FAKE, 10, k, FAKE, None) == EUNSUP


def test_layer_validation(lib):
    assert lib.bitlogic_lut_layer(None, 10, 4, FAKE, FAKE, 10, 6, FAKE, None) == ENULL
    assert lib.bitlogic_lut_layer(FAKE, 10, 4, None, FAKE, 10, 6, FAKE, None) == ENULL
    assert lib.bitlogic_lut_layer(FAKE, 0, 4, FAKE, FAKE, 10, 6, FAKE, None) == ESHAPE
    assert lib.bitlogic_lut_layer(FAKE, 10, -4, FAKE, FAKE, 10, 6, FAKE, None) == ESHAPE
    assert lib.bitlogic_lut_layer(FAKE, 10, 4, FAKE, FAKE, 0, 6, FAKE, None) == ESHAPE
    assert lib.bitlogic_lut_layer(FAKE + 2, 10, 4, FAKE, FAKE, 10, 6, FAKE, None) == EALIGN
    assert lib.bitlogic_lut_layer(FAKE, 10, 4, FAKE + 1, FAKE, 10, 6, FAKE, None) == EALIGN
    assert lib.bitlogic_lut_layer(FAKE, 10, 0, FAKE, FAKE, 10, 6, FAKE, None) == OK


def test_head_validation(lib):
    ws = lib.bitlogic_groupsum_head_workspace_bytes(100, 4096, 10)
    assert ws > 0 and ws % 8 == 0
    assert lib.bitlogic_groupsum_head_workspace_bytes(101, 4096, 10) == 0
    assert lib.bitlogic_groupsum_head(None, 100, 4096, 10, FAKE, FAKE, FAKE, ws, None) == ENULL
    assert lib.bitlogic_groupsum_head(FAKE, 100, 4096, 10, None, None, FAKE, ws, None) == ENULL
    assert lib.bitlogic_groupsum_head(FAKE, 101, 4096, 10, FAKE, FAKE, FAKE, ws, None) == ESHAPE
    assert lib.bitlogic_groupsum_head(FAKE, 100, 4096, 0, FAKE, FAKE, FAKE, ws, None) == ESHAPE
    assert lib.bitlogic_groupsum_head(FAKE, 70000 * 2, 64, 2, FAKE, FAKE, FAKE, 1 << 30,
                                      None) == ESHAPE
    assert lib.bitlogic_groupsum_head(FAKE, 100, 4096, 10, FAKE, FAKE, FAKE, ws - 1,
                                      None) == EWS
    assert lib.bitlogic_groupsum_head(FAKE, 100, 4096, 10, FAKE, FAKE, None, ws, None) == ENULL
    assert lib.bitlogic_groupsum_head(FAKE, 100, 4096, 10, FAKE, FAKE, FAKE + 8, ws,
                                      None) == EALIGN
    assert lib.bitlogic_groupsum_head(FAKE, 100, 0, 10, FAKE, FAKE, FAKE, ws, None) == OK


def _layers(specs):
    arr = (bl._Layer * len(specs))()
    for i, (w, k) in enumerate(specs):
        arr[i].conn, arr[i].tables, arr[i].w_out, arr[i].k = FAKE, FAKE, w, k
    return ctypes.cast(arr, ctypes.c_void_p), arr


def test_forward_workspace_formula(lib, monkeypatch):
    p, keep = _layers([(1000, 6), (1000, 6)])
    n, d, b, c = 4096, 784, 1, 10
    W = 64
    rnd = lambda v: (v + 255) // 256 * 256
    # fused last layer + head: layer 2 is not stored; counter planes of two
    # one-pass blocks per class (a batch this small takes the most blocks:
    # 100 nodes -> 64 + 36, 7 planes each)
    monkeypatch.delenv("BITLOGIC_UNFUSED_HEAD", raising=False)
    need = lib.bitlogic_forward_workspace_bytes(n, d, b, p, 2, c)
    assert need == rnd(d * b * W * 8) + rnd(1000 * W * 8) + rnd(c * 2 * 7 * W * 8)
    # separate head: both layers stored, plus the head's own workspace
    monkeypatch.setenv("BITLOGIC_UNFUSED_HEAD", "1")
    need = lib.bitlogic_forward_workspace_bytes(n, d, b, p, 2, c)
    head = lib.bitlogic_groupsum_head_workspace_bytes(1000, n, c)
    assert need == rnd(d * b * W * 8) + 2 * rnd(1000 * W * 8) + rnd(head)
    monkeypatch.delenv("BITLOGIC_UNFUSED_HEAD")
    # bad shapes give 0
    assert lib.bitlogic_forward_workspace_bytes(n, d, b, p, 2, 7) == 0
    assert lib.bitlogic_forward_workspace_bytes(n, d, b, p, 0, c) == 0
    p7, keep7 = _layers([(1000, 7)])
    assert lib.bitlogic_forward_workspace_bytes(n, d, b, p7, 1, c) == 0


def test_forward_validation(lib):
    p, keep = _layers([(1000, 6), (1000, 6)])
    need = lib.bitlogic_forward_workspace_bytes(4096, 784, 1, p, 2, 10)
    args = lambda **o: [o.get("x", FAKE), o.get("n", 4096), 784, FAKE, 1, o.get("layers", p),
                        o.get("L", 2), o.get("c", 10), FAKE, FAKE, o.get("ws", FAKE * 16),
                        o.get("wsb", need), None]
    assert lib.bitlogic_forward(*args(x=None)) == ENULL
    assert lib.bitlogic_forward(*args(layers=None)) == ENULL
    assert lib.bitlogic_forward(*args(L=0)) == ESHAPE
    assert lib.bitlogic_forward(*args(c=7)) == ESHAPE
    assert lib.bitlogic_forward(*args(ws=None)) == ENULL
    assert lib.bitlogic_forward(*args(wsb=need - 1)) == EWS
    assert lib.bitlogic_forward(*args(ws=FAKE * 16 + 64)) == EALIGN
    assert lib.bitlogic_forward(*args(n=0)) == OK
    pk, keepk = _layers([(1000, 6), (1000, 0)])
    assert lib.bitlogic_forward(*args(layers=pk)) == EUNSUP


def test_python_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros((64, 4), dtype=torch.uint8)
    th = torch.zeros((4, 1), dtype=torch.uint8)
    with pytest.raises(ValueError, match="GPU"):
        bl.bitlogic_encode(x, th, bits_out=torch.zeros((4, 1), dtype=torch.int64))


def test_model_checks_connection_range():
    import numpy as np
    th = np.zeros((4, 2), np.uint8)
    conn = np.array([[0, 8]], np.int32)          # 8 >= w_in = 8
    with pytest.raises(ValueError, match="outside"):
        bl.BitlogicModel.from_numpy(th, [(conn, np.zeros(1, np.uint64))], 1, device="cpu")


def test_forward_timed_validation(lib):
    p, keep = _layers([(1000, 6), (1000, 6)])
    need = lib.bitlogic_forward_workspace_bytes(4096, 784, 1, p, 2, 10)
    ev = (ctypes.c_void_p * 5)(*([FAKE] * 5))
    base = [FAKE, 4096, 784, FAKE, 1, p, 2, 10, FAKE, FAKE, FAKE * 16, need, None]
    assert lib.bitlogic_forward_timed(*base, None, 5) == ENULL
    assert lib.bitlogic_forward_timed(*base, ctypes.cast(ev, ctypes.c_void_p), 4) == ESHAPE
    ev[3] = None
    assert lib.bitlogic_forward_timed(*base, ctypes.cast(ev, ctypes.c_void_p), 5) == ENULL


def test_forward_plan(lib, monkeypatch):
    monkeypatch.delenv("BITLOGIC_UNFUSED_HEAD", raising=False)
    info = bl._ForwardInfo()
    ref = ctypes.byref(info)
    # group size 100: fused; at 4096 samples one-pass blocks (64 + 36 nodes);
    # at 2^20 samples one block of two passes (the second one short)
    p, keep = _layers([(1000, 6), (1000, 6)])
    assert lib.bitlogic_forward_plan(4096, 784, 1, p, 2, 10, ref) == OK
    assert info.workspace_bytes == lib.bitlogic_forward_workspace_bytes(4096, 784, 1, p, 2, 10)
    assert info.fused_head == 1 and info.slab_words >= 1
    assert info.head_splits == 2 and info.head_planes == 7          # counts up to 64
    assert lib.bitlogic_forward_plan(1 << 20, 784, 1, p, 2, 10, ref) == OK
    assert info.head_splits == 1 and info.head_planes == 8          # counts up to 128
    # group size 640: one block of 10 passes per class; planes hold counts up
    # to the block size
    p4, keep4 = _layers([(64000, 6), (64000, 6)])
    assert lib.bitlogic_forward_plan(1 << 18, 3072, 7, p4, 2, 100, ref) == OK
    assert info.fused_head == 1
    assert info.workspace_bytes == lib.bitlogic_forward_workspace_bytes(1 << 18, 3072, 7, p4, 2,
                                                                        100)
    assert info.head_splits == 1 and info.head_planes == 10
    # group size 6400 (C5): 100 passes as 10 equal blocks of 10
    p5, keep5 = _layers([(64000, 4), (64000, 4)])
    assert lib.bitlogic_forward_plan(1 << 18, 3072, 3, p5, 2, 10, ref) == OK
    assert info.head_splits == 10 and info.head_planes == 10
    # group size 800 (C2): 12.5 passes, one block with a short last pass
    p2, keep2 = _layers([(8000, 6), (8000, 6)])
    assert lib.bitlogic_forward_plan(1 << 20, 784, 7, p2, 2, 10, ref) == OK
    assert info.head_splits == 1 and info.head_planes == 10
    # group size 1 (one node per class) still fuses: one padded pass
    p1, keep1 = _layers([(1000, 6), (64, 6)])
    assert lib.bitlogic_forward_plan(4096, 784, 1, p1, 2, 64, ref) == OK
    assert info.fused_head == 1 and info.head_splits == 1
    monkeypatch.setenv("BITLOGIC_UNFUSED_HEAD", "1")
    assert lib.bitlogic_forward_plan(1 << 18, 3072, 7, p4, 2, 100, ref) == OK
    assert info.fused_head == 0
    # the checks of bitlogic_forward
    assert lib.bitlogic_forward_plan(4096, 784, 1, p, 2, 10, None) == ENULL
    assert lib.bitlogic_forward_plan(4096, 784, 1, p, 2, 7, ref) == ESHAPE
    assert lib.bitlogic_forward_plan(4096, 784, 1, None, 2, 10, ref) == ENULL


def test_grouped_dsp_validation(lib):
    f = lib.bitlogic_grouped_dsp_head
    assert f(None, 64, 10, FAKE, FAKE, FAKE, None) == ENULL
    assert f(FAKE, 64, 10, None, FAKE, FAKE, None) == ENULL
    assert f(FAKE, 64, 10, FAKE, None, None, None) == ENULL
    assert f(FAKE, -1, 10, FAKE, FAKE, FAKE, None) == ESHAPE
    assert f(FAKE, 64, 0, FAKE, FAKE, FAKE, None) == ESHAPE
    assert f(FAKE, 64, 129, FAKE, FAKE, FAKE, None) == EUNSUP
    assert "128" in _err(lib)
    assert f(FAKE + 2, 64, 10, FAKE, FAKE, FAKE, None) == EALIGN
    assert f(FAKE, 0, 10, FAKE, FAKE, FAKE, None) == OK        # nothing to do


def test_forward_grouped_dsp_validation(lib):
    p, keep = _layers([(1000, 6), (1000, 6)])
    need = lib.bitlogic_forward_workspace_bytes(4096, 784, 1, p, 2, 10)
    args = lambda **o: [FAKE, o.get("n", 4096), 784, FAKE, 1, p, 2, o.get("c", 10),
                        o.get("w", FAKE), FAKE, FAKE, FAKE * 16, need, None]
    f = lib.bitlogic_forward_grouped_dsp
    assert f(*args(w=None)) == ENULL
    assert f(*args(c=7)) == ESHAPE                      # 1000 nodes do not split into 7 groups
    p2, keep2 = _layers([(1000, 6), (250 * 4 * 129 // 129 * 129, 6)])
    assert f(FAKE, 4096, 784, FAKE, 1, p2, 2, 129, FAKE, FAKE, FAKE, FAKE * 16, 1 << 40,
             None) == EUNSUP
    assert f(*args(n=0)) == OK


def test_encode_binary_validation(lib):
    f = lib.bitlogic_encode_binary
    assert f(None, 64, 4, 2, FAKE, None) == ENULL
    assert f(FAKE, 64, 4, 0, FAKE, None) == ESHAPE
    assert f(FAKE, 64, 4, 9, FAKE, None) == ESHAPE
    assert f(FAKE, -1, 4, 2, FAKE, None) == ESHAPE
    assert f(FAKE, 64, 4, 2, FAKE + 4, None) == EALIGN
    assert f(FAKE, 0, 4, 2, FAKE, None) == OK


def test_fit_quantiles_validation(lib):
    ws = lib.bitlogic_fit_quantile_thresholds_workspace_bytes
    assert ws(1) == 256 * 8 and ws(3) == 3 * 256 * 8
    assert ws(0) == 0 and ws(33) == 0
    f = lib.bitlogic_fit_quantile_thresholds
    good = [FAKE, 100, 12, 3, 3, FAKE, FAKE * 16, ws(3), None]
    bad = lambda i, v: f(*(good[:i] + [v] + good[i + 1:]))
    assert bad(0, None) == ENULL and bad(5, None) == ENULL and bad(6, None) == ENULL
    assert bad(1, 0) == ESHAPE                   # no samples to fit on
    assert bad(3, 0) == ESHAPE and bad(3, 65) == ESHAPE
    assert bad(4, 5) == ESHAPE                   # 12 features do not split into 5 groups
    assert bad(4, 33) == ESHAPE
    assert bad(7, ws(3) - 1) == EWS
    assert bad(6, FAKE * 16 + 4) == EALIGN
    assert bad(1, 1 << 55) == ESHAPE             # n * d beyond 2^56


def _net(p, **o):
    net = bl._Network()
    net.n_features, net.encoder, net.n_bits = o.get("d", 784), o.get("enc", 0), o.get("b", 1)
    net.thresholds = o.get("th", FAKE)
    net.layers, net.n_layers, net.n_classes = p, o.get("L", 2), o.get("c", 10)
    net.head, net.head_weights = o.get("head", 0), o.get("w", None)
    return net


def test_network_validation(lib):
    p, keep = _layers([(1000, 6), (1000, 6)])
    ws = lambda net: lib.bitlogic_network_workspace_bytes(ctypes.byref(net), 4096)
    # same plan as the legacy call
    assert ws(_net(p)) == lib.bitlogic_forward_workspace_bytes(4096, 784, 1, p, 2, 10)
    pb, keepb = _layers([(1000, 6), (1000, 6)])
    assert ws(_net(pb, enc=1, b=4, th=None)) == lib.bitlogic_forward_workspace_bytes(
        4096, 784, 4, pb, 2, 10)
    fwd = lambda net, **o: lib.bitlogic_network_forward(
        ctypes.byref(net), o.get("x", FAKE), o.get("n", 4096), FAKE, FAKE, FAKE * 16,
        o.get("wsb", 1 << 40), None, None, 0)
    assert lib.bitlogic_network_forward(None, FAKE, 64, FAKE, FAKE, FAKE * 16, 1 << 40, None,
                                        None, 0) == ENULL
    assert fwd(_net(p, th=None)) == ENULL                    # thermometer without thresholds
    assert fwd(_net(p, enc=2)) == EUNSUP                     # unknown encoder
    assert fwd(_net(p, enc=1, b=9, th=None)) == EUNSUP       # binary code wider than 8 bits
    assert fwd(_net(p, head=2)) == EUNSUP                    # unknown head
    assert fwd(_net(p, head=1)) == ENULL                     # quantized head without weights
    p2, keep2 = _layers([(1000, 6), (129000, 6)])
    assert fwd(_net(p2, head=1, w=FAKE, c=129)) == EUNSUP
    assert fwd(_net(p), x=None) == ENULL
    assert fwd(_net(p), wsb=0) == EWS
    assert fwd(_net(p), n=0) == OK
    assert fwd(_net(p, enc=1, b=8, th=None), n=0) == OK
    info = bl._ForwardInfo()
    assert lib.bitlogic_network_plan(ctypes.byref(_net(p)), 4096, ctypes.byref(info)) == OK
    assert info.workspace_bytes == ws(_net(p))


def test_network_noalloc_validation(lib):
    p, keep = _layers([(1000, 6), (1000, 6)])
    fwd = lambda net, **o: lib.bitlogic_network_forward_noalloc(
        ctypes.byref(net) if net is not None else None, o.get("x", FAKE), o.get("n", 4096),
        o.get("out", FAKE), o.get("am", FAKE), None)
    assert fwd(None) == ENULL
    assert fwd(_net(p), x=None) == ENULL
    assert fwd(_net(p), out=None, am=None) == ENULL
    assert fwd(_net(p), out=FAKE + 2) == EALIGN
    assert fwd(_net(p, enc=2)) == EUNSUP
    # the static scratch bounds the batch: rejected before any HIP call
    cap = bl.NOALLOC_SCRATCH_BYTES
    ws = lambda n: lib.bitlogic_network_workspace_bytes(ctypes.byref(_net(p)), n)
    big = 64
    while ws(big) <= cap:
        big *= 2
    assert fwd(_net(p), n=big) == EWS
    assert "static buffer" in _err(lib)
    assert fwd(_net(p), n=0) == OK
    hdr = open(HEADER).read()
    assert re.search(r"#define BITLOGIC_NOALLOC_SCRATCH_BYTES \(64u << 20\)", hdr)


def test_pass_fanin_plan(lib):
    # a specialized network keeps the fused head and the workspace
    p, keep = _layers([(1280, 6), (1280, 6)])     # g = 128 per class: fused head
    info = bl._ForwardInfo()
    ref = ctypes.byref(info)
    assert lib.bitlogic_network_plan(ctypes.byref(_net(p)), 4096, ref) == OK
    plain_ws, plain_fused = info.workspace_bytes, info.fused_head
    assert plain_fused == 1
    arr = (ctypes.c_void_p * 2)(FAKE, FAKE)
    net = _net(p)
    net.pass_fanin = ctypes.cast(arr, ctypes.c_void_p)
    assert lib.bitlogic_network_plan(ctypes.byref(net), 4096, ref) == OK
    assert info.fused_head == 1 and info.workspace_bytes == plain_ws


def test_probe_validation(lib):
    assert lib.bitlogic_probe_valu(None, 1, 1, 0, None) == ENULL
    assert lib.bitlogic_probe_valu(FAKE, 0, 1, 0, None) == ESHAPE
    assert lib.bitlogic_probe_valu(FAKE, 1, -1, 0, None) == ESHAPE
    assert lib.bitlogic_probe_valu(FAKE + 2, 1, 1, 0, None) == EALIGN
    C, R, Wr = 0, 1, 2
    hbm = lambda mode, i, o, n, u=4, b=0: lib.bitlogic_probe_hbm(mode, i, o, n, u, b, None)
    assert hbm(3, FAKE, FAKE * 4, 16) == EUNSUP                # unknown mode
    assert hbm(C, FAKE, FAKE * 4, 16, u=3) == EUNSUP           # unroll not 1, 2, 4, 8
    assert hbm(C, None, FAKE, 16) == ENULL
    assert hbm(C, FAKE, None, 16) == ENULL
    assert hbm(R, FAKE, None, 16) == ENULL                      # the read probe writes 16 bytes
    assert hbm(Wr, None, None, 16) == ENULL
    assert hbm(C, FAKE, FAKE * 4, 24) == ESHAPE
    assert hbm(C, FAKE, FAKE * 4, -16) == ESHAPE
    assert hbm(C, FAKE, FAKE * 4, 16, b=-1) == ESHAPE
    assert hbm(C, FAKE + 8, FAKE * 4, 16) == EALIGN
    assert hbm(R, FAKE, FAKE * 4 + 4, 16) == EALIGN
    assert hbm(Wr, None, FAKE + 8, 16) == EALIGN
    assert hbm(C, FAKE, FAKE + 16, 64) == ESHAPE                # overlap
    assert "overlap" in _err(lib)
    assert hbm(C, FAKE, FAKE * 4, 0) == OK
    assert lib.bitlogic_probe_valu_op(3, FAKE, 1, 1, 0, None) == EUNSUP
    assert lib.bitlogic_probe_valu_op(0, None, 1, 1, 0, None) == ENULL
    assert lib.bitlogic_probe_valu_op(0, FAKE, 0, 1, 0, None) == ESHAPE
    assert lib.bitlogic_probe_valu_op(2, FAKE, 1, 0, 0, None) == ESHAPE
    assert lib.bitlogic_probe_valu_op(1, FAKE + 2, 1, 1, 0, None) == EALIGN
    g = lambda **o: lib.bitlogic_probe_gather(
        o.get("rows", FAKE), o.get("n", 100), o.get("lpr", 4), o.get("v", 0), o.get("b", 1),
        o.get("p", 1), o.get("occ", 0), 0, o.get("out", FAKE), o.get("sink", None), None)
    assert g(lpr=2) == EUNSUP
    assert g(v=100) == EUNSUP
    assert g(rows=None) == ENULL
    assert g(out=None) == ENULL
    assert g(n=0) == ESHAPE
    assert g(b=0) == ESHAPE
    assert g(p=0) == ESHAPE
    assert g(occ=9) == ESHAPE
    assert g(b=1 << 20, p=1 << 10) == ESHAPE
    assert g(rows=FAKE + 8) == EALIGN
    assert g(sink=FAKE + 8) == EALIGN
    assert hbm(Wr, None, FAKE * 4, 0) == OK
