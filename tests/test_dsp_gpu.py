"""Quantized (DSP-backed) head on the GPU against the oracle, bit-exact.

The head multiplies the group sums by a c x c signed 8-bit matrix (Sec. 3
"Encoders and heads"; Sec. 5 "Head") on the matrix cores.  Cases: the
hand-worked golden examples, class counts that are not multiples of the
16-wide output tiles or the 32-deep K steps (1 .. 128), sample counts with a
ragged last 64-sample block, counts at both ends of 0..65535 with weights at
both ends of the int8 range, either output omitted, and the whole forward
with the quantized head on the fused and the separate head paths.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _check(counts, Q):
    lg, am = bl.bitlogic_grouped_dsp_head(_dev(counts), _dev(Q))
    torch.cuda.synchronize()
    rl, rp = oracle.grouped_dsp(counts, Q)
    assert np.array_equal(lg.cpu().numpy().astype(np.int64), rl)
    assert np.array_equal(am.cpu().numpy(), rp)


def test_golden_cases():
    for line in open(os.path.join(GOLDEN, "grouped_dsp.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        cnt, q, lg, pr = [f.strip() for f in line.split("|")]
        counts = np.array([[int(v) for v in cnt.split(",")]], np.int32)
        Q = np.array([[int(v) for v in r.split(",")] for r in q.split(";")], np.int8)
        got, am = bl.bitlogic_grouped_dsp_head(_dev(counts), _dev(Q))
        assert got.cpu().numpy()[0].tolist() == [int(v) for v in lg.split(",")]
        assert int(am.cpu()[0]) == int(pr)


@pytest.mark.parametrize("c", [1, 2, 10, 15, 16, 17, 31, 32, 33, 64, 100, 127, 128])
@pytest.mark.parametrize("n", [1, 64, 64 * 5 + 13])
def test_random_counts(c, n):
    rng = np.random.default_rng(c * 1000 + n)
    counts = rng.integers(0, 65536, size=(n, c)).astype(np.int32)
    counts[0, :] = 65535
    if n > 1:
        counts[1, :] = 0
    Q = rng.integers(-128, 128, size=(c, c)).astype(np.int8)
    Q[0, :] = 127
    if c > 1:
        Q[1, :] = -128
    _check(counts, Q)


def test_extremes_and_ties():
    c = 128
    counts = np.full((70, c), 65535, np.int32)
    for Q in (np.full((c, c), 127, np.int8), np.full((c, c), -128, np.int8),
              np.zeros((c, c), np.int8)):
        _check(counts, Q)          # all logits equal: argmax 0


@pytest.mark.parametrize("c", [17, 37, 100, 128])
def test_partial_ties_across_lanes_and_tiles(c):
    # Q = +-identity makes logit i = +-count i; each sample's maximum is
    # shared by 2-5 classes spread over different lanes (class % 16) and
    # N tiles (class // 16), so the argmax must merge the lanes' and tiles'
    # partial maxima and keep the lowest tied class
    rng = np.random.default_rng(c)
    n = 64 * 3 + 21
    for sign in (1, -1):
        counts = rng.integers(1, 1000, size=(n, c)).astype(np.int32)
        lowest = np.empty(n, np.int64)
        for s in range(n):
            tied = rng.choice(c, size=int(rng.integers(2, 6)), replace=False)
            counts[s, tied] = 2000 if sign > 0 else 0        # above / below every other count
            lowest[s] = tied.min()
        Q = (sign * np.eye(c)).astype(np.int8)
        assert np.array_equal(oracle.grouped_dsp(counts, Q)[1], lowest)
        _check(counts, Q)


def test_one_output_only():
    rng = np.random.default_rng(8)
    counts = rng.integers(0, 700, size=(300, 100)).astype(np.int32)
    Q = rng.integers(-127, 128, size=(100, 100)).astype(np.int8)
    rl, rp = oracle.grouped_dsp(counts, Q)
    _, am = bl.bitlogic_grouped_dsp_head(_dev(counts), _dev(Q), want_logits=False)
    assert np.array_equal(am.cpu().numpy(), rp)
    lg = torch.empty((300, 100), dtype=torch.int32, device=DEV)
    bl.bitlogic_grouped_dsp_head(_dev(counts), _dev(Q), logits=lg)
    assert np.array_equal(lg.cpu().numpy().astype(np.int64), rl)


def _forward_dsp(wl, x, idx=None):
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    lg, am = bl.bitlogic_forward_grouped_dsp(_dev(x), model.thresholds, model.layers,
                                             wl.n_classes, _dev(wl.dsp_weights))
    torch.cuda.synchronize()
    xs = x if idx is None else x[idx]
    counts, _ = oracle.forward(xs, wl.thresholds, wl.layers, wl.n_classes)
    rl, rp = oracle.grouped_dsp(counts, wl.dsp_weights)
    got_l, got_p = lg.cpu().numpy(), am.cpu().numpy()
    if idx is not None:
        got_l, got_p = got_l[idx], got_p[idx]
    assert np.array_equal(got_l.astype(np.int64), rl)
    assert np.array_equal(got_p, rp)


@pytest.mark.parametrize("name", ["c1_mnist_tiny", "c4_cifar100_wide", "c5_fanin_k4"])
def test_forward_grouped_dsp_reduced(name, monkeypatch):
    # C1 (group of 100) runs the separate head kernels, C4/C5 the fused one;
    # C4 is also run with the separate kernels
    wl = make_workload(name, seed=0, n=64 * 16 * 2 + 64 * 3 + 17)
    _forward_dsp(wl, wl.x)
    if name == "c4_cifar100_wide":
        monkeypatch.setenv("BITLOGIC_UNFUSED_HEAD", "1")
        _forward_dsp(wl, wl.x)


def test_forward_grouped_dsp_full_c4():
    # every sample of the full C4 batch through the quantized head
    wl = make_workload("c4_cifar100_wide", seed=0)
    assert wl.n == CONFIGS["c4_cifar100_wide"].n
    _forward_dsp(wl, wl.x)
