"""The whole network in one kernel (net_fused.hip) against the oracle.

For small networks and batches the forward runs encoder, every layer and the
GroupSum head in one block per 64 samples with the activations in LDS.  Each
case runs it (BITLOGIC_FUSED_NETWORK=1) and the layered kernels
(BITLOGIC_FUSED_NETWORK=0) and compares both with the oracle, bit-exactly:
C1 itself, the paper's deployed network shape (3136 wires, 2 x 4000 nodes,
n = 4), deep stacks with mixed fan-in, both encoders, one class and 100
classes, a single sample, ragged batches and repeated connections.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _network(rng, d, widths, ks, repeats=False):
    layers, w_in = [], d
    for w, k in zip(widths, ks):
        if repeats:
            conn = rng.integers(0, w_in, size=(w, k)).astype(np.int32)
        else:
            conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)])
        tab = rng.integers(0, 2 ** 63, size=w).astype(np.uint64)
        tab |= rng.integers(0, 2, size=w).astype(np.uint64) << np.uint64(63)
        layers.append((conn.astype(np.int32), tab))
        w_in = w
    return layers


def _run_both(monkeypatch, x, th, layers, c, binary_bits=0):
    kw = dict(encoder="binary", n_features=x.shape[1], n_bits=binary_bits) if binary_bits else {}
    m = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV, **kw)
    xt = torch.from_numpy(x).to(DEV)
    out = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("BITLOGIC_FUSED_NETWORK", mode)
        assert m.plan(x.shape[0])["fused_network"] == (mode == "1")
        s, p = m.forward(xt)
        torch.cuda.synchronize()
        out[mode] = (s.cpu().numpy(), p.cpu().numpy())
    monkeypatch.delenv("BITLOGIC_FUSED_NETWORK")
    rs, rp = oracle.forward(x, th, layers, c, binary_bits=binary_bits)
    for mode in ("1", "0"):
        assert np.array_equal(out[mode][0], rs), mode
        assert np.array_equal(out[mode][1], rp), mode


def test_c1_full_batch(monkeypatch):
    wl = make_workload("c1_mnist_tiny")
    _run_both(monkeypatch, wl.x, wl.thresholds, wl.layers, wl.n_classes)


@pytest.mark.parametrize("n", [1024, 64, 1000])
def test_paper_network_shape(n, monkeypatch):
    # 784 features, b = 4 sorted thresholds (3136 wires), 2 x 4000 nodes of
    # fan-in 4, 10 classes x 400
    rng = np.random.default_rng(n)
    x = rng.integers(0, 256, size=(n, 784), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(784, 4)), axis=1).astype(np.uint8)
    layers = _network(rng, 784 * 4, [4000, 4000], [4, 4])
    _run_both(monkeypatch, x, th, layers, 10)


@pytest.mark.parametrize("case", [
    # d, b, binary, widths, fan-ins, classes, n, repeats
    (100, 3, True, [500, 300, 200], [6, 3, 2], 4, 777, False),
    (30, 8, True, [64, 64, 64, 64, 64], [1, 2, 3, 4, 5], 1, 130, False),
    (13, 7, False, [50], [6], 5, 1, False),
    (64, 2, False, [2000, 1000], [6, 6], 100, 300, False),
    (40, 5, False, [600, 600, 600], [6, 6, 6], 6, 64 * 7 + 1, True),
    (7, 1, True, [12, 8], [6, 4], 2, 200, True),
])
def test_networks(case, monkeypatch):
    d, b, binary, widths, ks, c, n, repeats = case
    rng = np.random.default_rng(sum(widths) + n)
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    x[:2] = 0
    x[2:4] = 255
    th = None if binary else rng.integers(0, 256, size=(d, b)).astype(np.uint8)
    layers = _network(rng, d * b, widths, ks, repeats)
    _run_both(monkeypatch, x, th, layers, c, binary_bits=b if binary else 0)
