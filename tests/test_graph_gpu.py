"""The forward inside a captured HIP graph (torch.cuda.CUDAGraph).

Serving loops capture the whole forward once and replay it on new inputs
copied into the captured buffers.  Every launch of the library goes to the
stream it is handed and the forward records no memset or host
synchronisation, so a capture holds the complete pass.  Each case replays
the graph several times on fresh pixels, with eager forwards of the same
model on other inputs and synchronisations between the replays, and checks
every replay bit-exactly against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_07400_amd import bitlogic as bl
from paper_2602_07400_amd.workloads import make_workload

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _replays(model, wl, ref_fn, n, seeds=(11, 12, 13)):
    x_static = torch.from_numpy(wl.x[:n]).to(DEV)
    out = torch.empty((n, model.n_classes), dtype=torch.int32, device=DEV)
    arg = torch.empty((n,), dtype=torch.int32, device=DEV)
    ws = torch.empty((max(model.workspace_bytes(n), 1),), dtype=torch.uint8, device=DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                       # warm the path up off the capture
        model.forward(x_static, out=out, argmax=arg, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        model.forward(x_static, out=out, argmax=arg, workspace=ws)
    torch.cuda.synchronize()
    for seed in seeds:
        rng = np.random.default_rng(seed)
        xs = rng.integers(0, 256, size=(n, wl.x.shape[1]), dtype=np.uint8)
        x_static.copy_(torch.from_numpy(xs))
        g.replay()
        torch.cuda.synchronize()
        got_s, got_p = out.cpu().numpy().copy(), arg.cpu().numpy().copy()
        # eager work on other data between the replays
        other = rng.integers(0, 256, size=(n // 2 + 1, wl.x.shape[1]), dtype=np.uint8)
        es, ep = model.forward(torch.from_numpy(other).to(DEV))
        torch.cuda.synchronize()
        rs, rp = ref_fn(xs)
        assert np.array_equal(got_s, rs), f"replay with seed {seed}: scores differ"
        assert np.array_equal(got_p, rp), f"replay with seed {seed}: argmax differs"
        ros, rop = ref_fn(other)
        assert np.array_equal(es.cpu().numpy(), ros) and np.array_equal(ep.cpu().numpy(), rop)
    del g


@pytest.mark.parametrize("name,n", [("c1_mnist_tiny", 4096 + 37), ("c3_cifar10", 2000)])
def test_graph_replay_groupsum(name, n):
    wl = make_workload(name, seed=21, n=n)
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    _replays(model, wl, lambda xs: oracle.forward(xs, wl.thresholds, wl.layers, wl.n_classes), n)


def test_graph_replay_binary_encoder_quantized_head():
    wl = make_workload("c1_mnist_tiny", seed=22, n=3000)
    d, b = wl.x.shape[1], 1
    rng = np.random.default_rng(5)
    q = rng.integers(-127, 128, size=(wl.n_classes, wl.n_classes), dtype=np.int8)
    model = bl.BitlogicModel.from_numpy(None, wl.layers, wl.n_classes, device=DEV,
                                        encoder="binary", n_features=d, n_bits=b, head_weights=q)

    def ref(xs):
        counts, _ = oracle.forward(xs, None, wl.layers, wl.n_classes, binary_bits=b)
        logits, pred = oracle.grouped_dsp(counts, q)
        return logits.astype(np.int32), pred

    _replays(model, wl, ref, 3000)


def test_graph_replay_specialized():
    wl = make_workload("c4_collapsed", seed=23, n=1500)
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV,
                                        specialize=True)
    assert model.pass_fanin is not None
    _replays(model, wl, lambda xs: oracle.forward(xs, wl.thresholds, wl.layers, wl.n_classes),
             1500)


def test_graph_replay_node_per_wave_layer(monkeypatch):
    # layer 1 on the node-per-wave kernel (forced at this batch): the capture
    # holds its record kernel, so every replay rebuilds the records it jumps
    # through, and the eager forwards between replays use the same workspace
    # layout in their own buffers
    monkeypatch.setenv("BITLOGIC_JUMP_LAYER", "1")
    wl = make_workload("c3_cifar10", seed=24, n=4096)
    model = bl.BitlogicModel.from_numpy(wl.thresholds, wl.layers, wl.n_classes, device=DEV)
    assert model.plan(4096)["jump_layers"] == [0]
    _replays(model, wl, lambda xs: oracle.forward(xs, wl.thresholds, wl.layers, wl.n_classes),
             4096)
