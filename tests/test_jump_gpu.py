"""The node-per-wave LUT layer (csrc/lut_jump.hip) through the whole forward.

BITLOGIC_JUMP_LAYER=1 runs every stored, unspecialized layer of fan-in 5 or 6
on the node-per-wave kernel wherever it can (batches of an even number of
1024-sample slabs), so small networks exercise it too; =0 keeps every layer on
the per-lane kernel.  Each case checks which layers the plan puts on the
kernel, compares scores and argmax with the oracle on every sample, and with
the per-lane path.  Cases: widths that are not whole 16-node waves or 64-node
blocks (a wave's last nodes, blocks past the end), fewer nodes than one wave,
depth 3 with two node-per-wave layers in a row, fan-in 5 (a sixth input the
extended table ignores), repeated connections, junk table bits above 2^k,
projection / constant / textbook tables, and batches that cannot use the
kernel (an odd slab count, one slab).  Without the switch, the plan of each
configuration at its full batch is checked: layer 1 of C3 and of C5 at k = 6
runs on the node-per-wave kernel; C4, whose 21504-row input slab pair does not
fit the L2, stays on the per-lane kernel.
"""
import os
from contextlib import contextmanager

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")

# projection tables of inputs 0..5, constants, AND / OR / parity / majority of
# inputs 0..2 (LSB-first address: bit i of the entry index is input i)
SPECIAL = [0xAAAAAAAAAAAAAAAA, 0xCCCCCCCCCCCCCCCC, 0xF0F0F0F0F0F0F0F0, 0xFF00FF00FF00FF00,
           0xFFFF0000FFFF0000, 0xFFFFFFFF00000000, 0, 0xFFFFFFFFFFFFFFFF, 0x8000000000000000,
           0xFFFFFFFFFFFFFFFE, 0x6996966996696996, 0xE8E8E8E8E8E8E8E8]


@contextmanager
def jump_switch(value):
    old = os.environ.get("BITLOGIC_JUMP_LAYER")
    if value is None:
        os.environ.pop("BITLOGIC_JUMP_LAYER", None)
    else:
        os.environ["BITLOGIC_JUMP_LAYER"] = value
    try:
        yield
    finally:
        if old is None:
            os.environ.pop("BITLOGIC_JUMP_LAYER", None)
        else:
            os.environ["BITLOGIC_JUMP_LAYER"] = old


def build(seed, n, d, b, widths, ks, repeats=False, special=False):
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b), dtype=np.uint8), axis=1)
    layers, w_in = [], d * b
    for w, k in zip(widths, ks):
        if repeats:
            conn = rng.integers(0, w_in, size=(w, k))
        else:
            conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)])
        tables = rng.integers(0, 1 << 63, size=w, dtype=np.int64).astype(np.uint64)
        tables |= rng.integers(0, 2, size=w).astype(np.uint64) << np.uint64(63)
        if special:
            for i in range(0, w, 3):
                tables[i] = np.uint64(SPECIAL[(i // 3) % len(SPECIAL)])
        layers.append((conn.astype(np.int32), tables))
        w_in = w
    return x, th, layers


# n, d, b, widths, ks, classes, repeats, special, layers expected on the kernel
CASES = [
    (2048, 64, 1, [100, 70], [6, 6], 7, False, False, [0]),
    (2048, 64, 1, [10, 70], [6, 6], 7, False, False, [0]),          # fewer nodes than a wave
    (6144, 200, 3, [1000, 640], [6, 6], 10, False, True, [0]),
    (4096, 784, 1, [1000, 1000], [6, 6], 10, False, False, [0]),    # C1 shape
    (8192, 100, 4, [3000, 2000, 1000], [6, 5, 6], 10, True, False, [0, 1]),
    (4096, 30, 2, [777, 80], [5, 6], 8, False, True, [0]),
    (4096, 40, 1, [500, 100], [4, 6], 10, False, False, []),        # fan-in 4: per-lane kernel
    (3 * 1024, 64, 1, [300, 70], [6, 6], 7, False, False, []),      # 3 slabs: odd
    (1024, 64, 1, [300, 70], [6, 6], 7, False, False, []),          # one slab
    (2048, 16, 1, [64], [6], 8, False, False, []),                  # depth 1: only the fused layer
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_forced_jump_layer_matches_oracle(case):
    n, d, b, widths, ks, c, repeats, special, expect = CASES[case]
    print(f"[jump case {case}] n={n} d={d} b={b} widths={widths} ks={ks} c={c} "
          f"repeats={repeats} special={special}", flush=True)
    x, th, layers = build(100 + case, n, d, b, widths, ks, repeats, special)
    model = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV)
    xd = torch.from_numpy(x).to(DEV)
    with jump_switch("1"):
        assert model.plan(n)["jump_layers"] == expect
        s1, p1 = model.forward(xd)
        torch.cuda.synchronize()
    with jump_switch("0"):
        assert model.plan(n)["jump_layers"] == []
        s0, p0 = model.forward(xd)
        torch.cuda.synchronize()
    rs, rp = oracle.forward(x, th, layers, c)
    s1, p1 = s1.cpu().numpy(), p1.cpu().numpy()
    bad = np.nonzero((s1 != rs).any(axis=1) | (p1 != rp))[0]
    assert bad.size == 0, f"{bad.size} of {n} samples differ from the oracle, first {bad[:8]}"
    assert np.array_equal(s1, s0.cpu().numpy()) and np.array_equal(p1, p0.cpu().numpy())


def test_forced_jump_layer_repeated_calls_and_workspace():
    # the record array is rebuilt on every call: two networks of different
    # tables through one workspace, alternately, each against the oracle
    n, c = 4096, 10
    nets = [build(300 + i, n, 96, 2, [800, 200], [6, 6]) for i in range(2)]
    models = [bl.BitlogicModel.from_numpy(th, layers, c, device=DEV) for _, th, layers in nets]
    with jump_switch("1"):
        ws_bytes = max(m.workspace_bytes(n) for m in models)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
        refs = [oracle.forward(x, th, layers, c) for x, th, layers in nets]
        for rep in range(3):
            for (x, _, _), m, (rs, rp) in zip(nets, models, refs):
                s, p = m.forward(torch.from_numpy(x).to(DEV), workspace=ws)
                torch.cuda.synchronize()
                assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(p.cpu().numpy(), rp)


@pytest.mark.parametrize("name,expect", [("c1_mnist_tiny", []), ("c2_fmnist", [0]),
                                         ("c3_cifar10", [0]), ("c4_cifar100_wide", []),
                                         ("c5_fanin_k2", []), ("c5_fanin_k4", []),
                                         ("c5_fanin_k6", [0])])
def test_default_plan_of_each_configuration(name, expect):
    wl = make_workload(name, seed=0, n=64)          # shapes only; the plan is for the full batch
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    with jump_switch(None):
        plan = model.plan(CONFIGS[name].n)
    assert plan["jump_layers"] == expect, plan


def draw_jump_case(seed):
    # seeded networks whose hidden layers the node-per-wave kernel takes when
    # forced: an even number of slabs, hidden fan-ins 5 or 6, and otherwise
    # mixed widths, depths, encoders, heads, class groups and repeats
    rng = np.random.default_rng(5000 + seed)
    n = 1024 * int(rng.choice([2, 4, 6, 8, 18, 64])) - int(rng.choice([0, 0, 1, 63, 500]))
    d = int(rng.integers(1, 300))
    binary = bool(rng.random() < 0.3)
    b = int(rng.integers(1, 9)) if binary else int(rng.choice([1, 2, 3, 7]))
    depth = int(rng.integers(2, 5))
    c = int(rng.choice([1, 3, 10, 17, 100]))
    g = int(rng.choice([1, 7, 64, 100, 333]))
    while c * g > 12000:
        g //= 2
    widths = [int(rng.integers(1, 4000)) for _ in range(depth - 1)] + [c * g]
    ks = [int(rng.choice([5, 6])) for _ in range(depth - 1)] + [int(rng.integers(1, 7))]
    return dict(seed=seed, n=n, d=d, binary=binary, b=b, widths=widths, ks=ks, c=c,
                dsp=bool(rng.random() < 0.25), repeats=bool(rng.random() < 0.3))


@pytest.mark.parametrize("seed", range(40))
def test_random_networks_forced_onto_the_node_per_wave_kernel(seed):
    case = draw_jump_case(seed)
    print("[case]", case, flush=True)
    rng = np.random.default_rng(6000 + seed)
    n, d, b, c = case["n"], case["d"], case["b"], case["c"]
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = None if case["binary"] else rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    layers, w_in = [], d * b
    for w, k in zip(case["widths"], case["ks"]):
        if case["repeats"] or k > w_in:
            conn = rng.integers(0, w_in, size=(w, k))
        else:
            conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)])
        tables = rng.integers(0, 1 << 63, size=w, dtype=np.int64).astype(np.uint64)
        tables |= rng.integers(0, 2, size=w).astype(np.uint64) << np.uint64(63)
        layers.append((conn.astype(np.int32), tables))
        w_in = w
    q = rng.integers(-128, 128, size=(c, c), dtype=np.int16).astype(np.int8) if case["dsp"] else None
    kw = (dict(encoder="binary", n_features=d, n_bits=b) if case["binary"] else {})
    model = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV, head_weights=q, **kw)
    with jump_switch("1"):
        plan = model.plan(n)
        s, p = model.forward(torch.from_numpy(x).to(DEV))
        torch.cuda.synchronize()
    hidden = list(range(len(layers) - 1)) if plan["fused_head"] else list(range(len(layers)))
    assert plan["jump_layers"] == [l for l in hidden if case["ks"][l] in (5, 6)], plan
    rs, rp = oracle.forward(x, th, layers, c, binary_bits=b if case["binary"] else 0)
    if q is not None:
        rs, rp = oracle.grouped_dsp(rs, q)
    s, p = s.cpu().numpy(), p.cpu().numpy()
    bad = np.nonzero((s != rs).any(axis=1) | (p != rp))[0]
    assert bad.size == 0, f"{bad.size} of {n} samples differ, first {bad[:8]}"
