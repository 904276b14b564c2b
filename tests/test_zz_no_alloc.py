"""bitlogic_network_forward_noalloc against bitlogic_network_forward.

The allocation-free entry point runs the same kernels with the library's
static per-GPU scratch instead of a caller workspace.  Its scores and argmax
must equal the workspace entry point's bit for bit (and the oracle's), on two
calls in a row whose second batch is smaller, so that the second call runs
over scratch the first one left behind.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _model(wl, head_weights=None):
    return bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV,
                                       head_weights=head_weights)


def _both(model, x):
    n = x.shape[0]
    ref_s, ref_p = model.forward(x)                      # caller workspace
    out = torch.full((n, model.n_classes), -7, dtype=torch.int32, device=DEV)
    am = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    print(f"[noalloc] n={n} workspace={model.workspace_bytes(n)}", flush=True)
    bl.bitlogic_network_forward_noalloc(model, x, out, am)
    torch.cuda.synchronize()
    return ref_s.cpu().numpy(), ref_p.cpu().numpy(), out.cpu().numpy(), am.cpu().numpy()


@pytest.mark.parametrize("name,n1,n2", [
    ("c1_mnist_tiny", 64 * 16 * 5 + 64 * 3 + 17, 64 * 16 + 5),    # 6 slabs, then 2
    ("c3_cifar10", 64 * 16 * 2 + 9, 100),
])
def test_noalloc_matches_workspace_forward_twice(name, n1, n2):
    wl = make_workload(name, seed=5, n=n1)
    model = _model(wl)
    x = torch.from_numpy(wl.x).to(DEV)
    assert model.workspace_bytes(n1) <= bl.NOALLOC_SCRATCH_BYTES
    for n in (n1, n2):                    # the second call is smaller
        rs, rp, gs, gp = _both(model, x[:n])
        assert np.array_equal(gs, rs), f"{name} n={n}: scores differ"
        assert np.array_equal(gp, rp), f"{name} n={n}: argmax differs"
        os_, op = oracle.forward(wl.x[:n], wl.thresholds, wl.layers, wl.n_classes)
        assert np.array_equal(gs, os_) and np.array_equal(gp, op), f"{name} n={n}: oracle"


def test_noalloc_with_the_node_per_wave_layer(monkeypatch):
    # layer 1 forced onto the node-per-wave kernel: its per-node records live
    # in the static scratch too, and the second, smaller call (4 slabs, then
    # 2) rebuilds them over what the first call left
    monkeypatch.setenv("BITLOGIC_JUMP_LAYER", "1")
    n1, n2 = 64 * 16 * 4, 64 * 16 * 2
    wl = make_workload("c3_cifar10", seed=7, n=n1)
    model = _model(wl)
    x = torch.from_numpy(wl.x).to(DEV)
    assert model.plan(n1)["jump_layers"] == [0]
    assert model.workspace_bytes(n1) <= bl.NOALLOC_SCRATCH_BYTES
    for n in (n1, n2):
        rs, rp, gs, gp = _both(model, x[:n])
        assert np.array_equal(gs, rs) and np.array_equal(gp, rp), f"n={n}: noalloc differs"
        os_, op = oracle.forward(wl.x[:n], wl.thresholds, wl.layers, wl.n_classes)
        assert np.array_equal(gs, os_) and np.array_equal(gp, op), f"n={n}: oracle"


def test_noalloc_quantized_head_and_argmax_only():
    wl = make_workload("c1_mnist_tiny", seed=6, n=3000)
    rng = np.random.default_rng(6)
    q = rng.integers(-127, 128, size=(wl.n_classes, wl.n_classes), dtype=np.int8)
    model = _model(wl, head_weights=q)
    x = torch.from_numpy(wl.x).to(DEV)
    for n in (3000, 1000):
        rs, rp, gs, gp = _both(model, x[:n])
        assert np.array_equal(gs, rs) and np.array_equal(gp, rp)
        am = torch.full((n,), -7, dtype=torch.int32, device=DEV)
        bl.bitlogic_network_forward_noalloc(model, x[:n], None, am)
        torch.cuda.synchronize()
        assert np.array_equal(am.cpu().numpy(), rp)


def test_noalloc_rejects_batch_beyond_scratch():
    wl = make_workload("c4_cifar100_wide", seed=0, n=64)
    model = _model(wl)
    n = 64
    while model.workspace_bytes(n) <= bl.NOALLOC_SCRATCH_BYTES:
        n *= 2
    x = torch.zeros((n, wl.x.shape[1]), dtype=torch.uint8, device=DEV)
    out = torch.zeros((n, wl.n_classes), dtype=torch.int32, device=DEV)
    am = torch.zeros((n,), dtype=torch.int32, device=DEV)
    with pytest.raises(bl.BitlogicError, match="static buffer"):
        bl.bitlogic_network_forward_noalloc(model, x, out, am)
