"""Seeded random networks of mixed shapes through the whole forward.

Each case draws its batch (1 sample up to 70 k, ragged and whole words),
feature count, encoder (thermometer with 1..16 thresholds, or the binary
code with 1..8 bits), depth 1..3, per-layer widths and fan-ins 1..6
(connections with and without repeats, junk table bits above 2^k), class
count and group size (1 node up to 1000 per class, fused and separate head),
head (GroupSum or the quantized head) and table specialization, and compares
scores (or logits) and argmax with the oracle on every sample.  The case
parameters are printed before each run, so a failure names its shape.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl

DEV = torch.device("cuda:0")
N_CASES = 160


def draw_case(seed):
    rng = np.random.default_rng(7000 + seed)
    n = int(rng.choice([1, 2, 63, 64, 65, 127, 1000, 1024, 1025, 4096, 4133, 16389, 70000]))
    d = int(rng.integers(1, 200))
    binary = bool(rng.random() < 0.3)
    b = int(rng.integers(1, 9)) if binary else int(rng.choice([1, 2, 3, 4, 7, 8, 9, 16]))
    depth = int(rng.integers(1, 4))
    c = int(rng.choice([1, 2, 3, 10, 17, 100]))
    g = int(rng.choice([1, 5, 31, 32, 64, 65, 100, 640, 1000]))
    while c * g > 20000:
        g //= 2
    widths = [int(rng.integers(1, 3000)) for _ in range(depth - 1)] + [c * g]
    if n >= 16389:                       # keep the oracle's share of the case small
        widths = [min(w, 1500) for w in widths[:-1]] + [min(c * g, 3000) // c * c or c]
    ks = [int(rng.integers(1, 7)) for _ in range(depth)]
    dsp = bool(rng.random() < 0.25)
    specialize = bool(rng.random() < 0.25)
    repeats = bool(rng.random() < 0.2)
    return dict(seed=seed, n=n, d=d, binary=binary, b=b, widths=widths, ks=ks, c=c, dsp=dsp,
                specialize=specialize, repeats=repeats)


def build(case):
    rng = np.random.default_rng(9000 + case["seed"])
    n, d, b, c = case["n"], case["d"], case["b"], case["c"]
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = None if case["binary"] else rng.integers(0, 256, size=(d, b), dtype=np.uint8)
    layers, w_in = [], d * b
    for w, k in zip(case["widths"], case["ks"]):
        if case["specialize"]:           # small per-node pools: tied inputs to remove
            pool = min(int(rng.integers(1, 4)), w_in)
            base = np.stack([rng.choice(w_in, size=pool, replace=False) for _ in range(w)])
            conn = np.take_along_axis(base, rng.integers(0, pool, size=(w, k)), axis=1)
        elif case["repeats"] or k > w_in:
            conn = rng.integers(0, w_in, size=(w, k))
        else:
            conn = np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)])
        tables = rng.integers(0, 1 << 63, size=w, dtype=np.int64).astype(np.uint64)
        tables |= rng.integers(0, 2, size=w).astype(np.uint64) << np.uint64(63)
        layers.append((conn.astype(np.int32), tables))
        w_in = w
    q = rng.integers(-128, 128, size=(c, c), dtype=np.int16).astype(np.int8) if case["dsp"] else None
    return x, th, layers, q


def test_case_draws_are_valid():
    for s in range(N_CASES):
        case = draw_case(s)
        assert case["widths"][-1] % case["c"] == 0
        assert case["widths"][-1] // case["c"] <= 65535
        assert all(1 <= k <= 6 for k in case["ks"])


@pytest.mark.gpu
@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_network(seed):
    case = draw_case(seed)
    print("[case]", case, flush=True)
    x, th, layers, q = build(case)
    c = case["c"]
    kw = (dict(encoder="binary", n_features=case["d"], n_bits=case["b"]) if case["binary"]
          else {})
    model = bl.BitlogicModel.from_numpy(th, layers, c, device=DEV, head_weights=q,
                                        specialize=0.0 if case["specialize"] else False, **kw)
    s, p = model.forward(torch.from_numpy(x).to(DEV))
    torch.cuda.synchronize()
    bits = case["b"] if case["binary"] else 0
    rs, rp = oracle.forward(x, th, layers, c, binary_bits=bits)
    if q is not None:
        rs, rp = oracle.grouped_dsp(rs, q)
    s, p = s.cpu().numpy(), p.cpu().numpy()
    bad = np.nonzero((s != rs).any(axis=1) | (p != rp))[0]
    assert bad.size == 0, f"{bad.size} of {case['n']} samples differ, first {bad[:8]}"
