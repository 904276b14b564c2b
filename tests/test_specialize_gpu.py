"""Table-specialized networks against the oracle.

The model is built with table specialization (bitlogic_specialize_network on
the host: nodes ordered by effective fan-in, each kernel pass evaluating its
fan-in); the oracle runs the original network.  Every comparison is
bit-exact: scores and argmax.  Cases: tied connections from small per-node
pools, tables that ignore some of their inputs, constant and pass-through
nodes, the fused and the unfused head, small-batch launches, both encoders,
both heads, ragged and single-sample batches, and the collapsed-routing
CIFAR-100 workload at its full batch on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _network(rng, w_in, widths, ks, pool):
    layers = []
    for w, k in zip(widths, ks):
        p = min(pool, w_in)
        base = np.stack([rng.choice(w_in, size=p, replace=False) for _ in range(w)])
        conn = np.take_along_axis(base, rng.integers(0, p, size=(w, k)), axis=1)
        tab = rng.integers(0, 2 ** 63, size=w).astype(np.uint64)
        tab |= rng.integers(0, 2, size=w).astype(np.uint64) << np.uint64(63)
        if k < 6:
            tab &= np.uint64((1 << (1 << k)) - 1)
        # a third of the nodes: constant, pass-through or 2-input functions
        for j in range(0, w, 3):
            kind = j // 3 % 3
            if kind == 0:
                tab[j] = np.uint64(0) if rng.integers(2) else np.uint64((1 << (1 << k)) - 1)
            elif kind == 1:
                s = int(rng.integers(k))
                tab[j] = np.uint64(sum(((a >> s) & 1) << a for a in range(1 << k)))
            elif k >= 2:
                tab[j] = np.uint64(sum((((a & 1) ^ ((a >> 1) & 1))) << a for a in range(1 << k)))
        layers.append((conn.astype(np.int32), tab))
        w_in = w
    return layers


def _check(x, th, layers, c, specialize, binary_bits=0, dsp=None, sample=None):
    kw = dict(encoder="binary", n_features=x.shape[1], n_bits=binary_bits) if binary_bits else {}
    m = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV, head_weights=dsp,
                                    specialize=specialize, **kw)
    if dsp is None and x.shape[0] > 0:
        plain = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV, **kw)
        assert m.plan(x.shape[0])["fused_head"] == plain.plan(x.shape[0])["fused_head"]
    s, p = m.forward(torch.from_numpy(x).to(DEV))
    torch.cuda.synchronize()
    s, p = s.cpu().numpy(), p.cpu().numpy()
    xs = x if sample is None else x[sample]
    if dsp is None:
        rs, rp = oracle.forward(xs, th, layers, c, binary_bits=binary_bits)
    else:
        rs, rp = _oracle_dsp(xs, th, layers, c, binary_bits, dsp)
    sel = slice(None) if sample is None else sample
    assert np.array_equal(s[sel], rs)
    assert np.array_equal(p[sel], rp)
    return m


def _oracle_dsp(x, th, layers, c, binary_bits, dsp):
    counts, _ = oracle.forward(x, th, layers, c, binary_bits=binary_bits)
    return oracle.grouped_dsp(counts, dsp)


@pytest.mark.parametrize("case", [
    # d, b, widths, fan-ins, classes, n, pool   (fused head when g % 32 == 0)
    (64, 4, [3000, 2560], [6, 6], 10, 64 * 16 * 40 + 64 * 3 + 17, 3),    # fused, 512-node blocks
    (64, 4, [3000, 2000], [6, 6], 10, 64 * 16 * 2 + 64 * 3 + 17, 3),     # unfused head
    (64, 4, [3000, 2560], [4, 4], 10, 5000, 3),
    (64, 4, [3000, 2000], [2, 2], 10, 5000, 2),
    (100, 3, [800, 600, 400], [6, 3, 5], 4, 777, 4),
    (30, 8, [640, 640], [5, 6], 20, 64 * 40, 6),
    (13, 7, [50], [6], 5, 1, 2),
    (40, 5, [600, 640], [1, 6], 10, 4096 + 1, 1),
    (48, 7, [6400, 6400], [6, 6], 100, 64 * 16 * 24, 3),                 # C4-like head, g = 64
])
def test_specialized_forward(case):
    d, b, widths, ks, c, n, pool = case
    spec = 0.0                                    # every layer specialized
    rng = np.random.default_rng(n + pool)
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b)), axis=1).astype(np.uint8)
    layers = _network(rng, d * b, widths, ks, pool)
    print(f"[spec] d={d} b={b} widths={widths} k={ks} c={c} n={n} pool={pool} spec={spec}",
          flush=True)
    m = _check(x, th, layers, c, spec)
    assert [int(h.sum()) for h in m.fanin_histogram] == widths
    assert all(f is not None for f in m.pass_fanin)


def test_gain_threshold_mixes_kept_and_specialized_layers():
    # layer 1 distinct routing with random tables (kept), layers 2 and 3
    # collapsed (specialized): the kept layer's connections are unchanged, the
    # next one reads through the specialized layer's new order
    rng = np.random.default_rng(11)
    d, b, c, n = 64, 4, 10, 64 * 16 * 3 + 5
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b)), axis=1).astype(np.uint8)
    conn0 = np.stack([rng.choice(d * b, size=6, replace=False) for _ in range(2000)])
    first = [(conn0.astype(np.int32), rng.integers(0, 2 ** 63, size=2000).astype(np.uint64))]
    rest = _network(rng, 2000, [1500, 1280], [6, 6], 2)
    layers = first + rest
    print("[spec-mixed]", flush=True)
    m = _check(x, th, layers, c, True)
    assert m.pass_fanin[0] is None and m.pass_fanin[1] is not None


@pytest.mark.parametrize("n", [1000, 64 * 33])
def test_specialized_binary_encoder_and_dsp_head(n):
    rng = np.random.default_rng(n)
    d, b, c = 48, 5, 12
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    layers = _network(rng, d * b, [1200, 1200], [6, 4], 3)
    dsp = rng.integers(-127, 128, size=(c, c)).astype(np.int8)
    print(f"[spec-binary-dsp] n={n}", flush=True)
    _check(x, None, layers, c, 0.0, binary_bits=b, dsp=dsp)
    th = np.sort(rng.integers(0, 256, size=(d, b)), axis=1).astype(np.uint8)
    _check(x, th, layers, c, 0.0, dsp=dsp)


def test_specialized_unique_routing_matches_unspecialized():
    # distinct random routing: specialization leaves almost every node at
    # fan-in k; forced on (0.0) the result must not change, and by default
    # the layers are kept
    wl = make_workload("c1_mnist_tiny")
    print("[spec-c1]", flush=True)
    _check(wl.x, wl.thresholds, wl.layers, wl.n_classes, 0.0)
    m = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV,
                                    specialize=True)
    assert m.pass_fanin is None


def test_collapsed_workload_full_batch():
    cfg = CONFIGS["c4_collapsed"]
    wl = make_workload("c4_collapsed")
    print(f"[spec-full] c4_collapsed n={cfg.n}, every sample", flush=True)
    m = _check(wl.x, wl.thresholds, wl.layers, wl.n_classes, True)
    for h in m.fanin_histogram:
        assert h[4:].sum() == 0                      # at most 3 distinct wires per node
    assert all(layer[0].shape[1] == 3 for layer in m.layers)


def test_specialized_large_batch_block_modes():
    # 2^18 samples: the stored layers run 512-node blocks (>= 2048 a launch),
    # specialized to fan-in 4, 2 and 1 (slots drawn from 4, 2 and 1 wires);
    # blocks whose passes share one fan-in run the plain loops of that
    # fan-in, blocks that mix fan-ins the per-pass loop, and widths that are
    # not multiples of 512 leave a short last block.  The last layer (fan-in
    # 3, 256 nodes a class) is fused with the head.
    rng = np.random.default_rng(2024)
    n, d, b = 1 << 18, 64, 4
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b)), axis=1).astype(np.uint8)
    layers, w_in = [], d * b
    for w, k, pool in ((5000, 6, 4), (4700, 4, 2), (4300, 3, 1), (2560, 6, 3)):
        layers += _network(rng, w_in, [w], [k], pool)
        w_in = w
    print(f"[spec-blocks] n={n}, widths 5000/4700/4300/2560, every sample", flush=True)
    m = _check(x, th, layers, 10, 0.0)
    assert [int(conn.shape[1]) for conn, _ in m.layers] == [4, 2, 1, 3]
    assert m.plan(n)["fused_head"]
