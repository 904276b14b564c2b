"""Seeded generators: determinism, shapes and the documented draws."""
import numpy as np
import pytest

from paper_2602_07400_amd.workloads import (CONFIG_ORDER, CONFIGS, draw_connectivity,
                                            draw_tables, make_workload, uniform_thresholds)


@pytest.mark.parametrize("name", CONFIG_ORDER)
def test_same_seed_same_bytes(name):
    a = make_workload(name, seed=0, n=256)
    b = make_workload(name, seed=0, n=256)
    assert a.x.tobytes() == b.x.tobytes()
    assert a.thresholds.tobytes() == b.thresholds.tobytes()
    for (c1, t1), (c2, t2) in zip(a.layers, b.layers):
        assert c1.tobytes() == c2.tobytes() and t1.tobytes() == t2.tobytes()
    c = make_workload(name, seed=1, n=256)
    assert c.x.tobytes() != a.x.tobytes()


@pytest.mark.parametrize("name", CONFIG_ORDER)
def test_shapes(name):
    cfg = CONFIGS[name]
    wl = make_workload(name, n=128)
    assert wl.x.shape == (128, cfg.d) and wl.x.dtype == np.uint8
    assert wl.thresholds.shape == (cfg.d, cfg.b)
    w_in = cfg.d * cfg.b
    for (conn, tab), w in zip(wl.layers, cfg.widths):
        assert conn.shape == (w, cfg.k) and conn.dtype == np.int32
        assert tab.shape == (w,) and tab.dtype == np.uint64
        assert conn.min() >= 0 and conn.max() < w_in
        s = np.sort(conn, axis=1)
        assert not (s[:, 1:] == s[:, :-1]).any(), "inputs of a node must be distinct"
        if cfg.k < 6:
            assert not (tab >> np.uint64(1 << cfg.k)).any()
        w_in = w
    assert cfg.widths[-1] % cfg.n_classes == 0


def test_model_draws_do_not_depend_on_n():
    a = make_workload("c3_cifar10", n=64)
    b = make_workload("c3_cifar10", n=512)
    assert a.thresholds.tobytes() == b.thresholds.tobytes()
    assert a.layers[1][0].tobytes() == b.layers[1][0].tobytes()


def test_fan_in_family_shares_pixels_and_thresholds():
    a = make_workload("c5_fanin_k2", n=64)
    b = make_workload("c5_fanin_k6", n=64)
    assert a.x.tobytes() == b.x.tobytes()
    assert a.thresholds.tobytes() == b.thresholds.tobytes()


def test_threshold_ladders():
    np.testing.assert_array_equal(uniform_thresholds(2, 7)[0], [31, 63, 95, 127, 159, 191, 223])
    np.testing.assert_array_equal(uniform_thresholds(1, 3)[0], [63, 127, 191])
    assert (make_workload("c1_mnist_tiny", n=64).thresholds == 128).all()
    q = make_workload("c3_cifar10", n=64).thresholds
    # quantiles of uniform pixels sit near 64/128/192 and are ladder-ordered
    assert (np.abs(q.astype(int) - [64, 128, 192]) <= 3).all()
    assert (np.diff(q.astype(int), axis=1) > 0).all()


def test_gaussian_mixture_pixels():
    wl = make_workload("c2_fmnist", n=4096)
    assert wl.labels is not None and wl.labels.min() >= 0 and wl.labels.max() < 10
    # clipping puts mass at both ends of the pixel range
    assert (wl.x == 0).mean() > 0.01 and (wl.x == 255).mean() > 0.01


def test_connectivity_sampler():
    rng = np.random.default_rng(0)
    c = draw_connectivity(rng, 5000, 6, 7)
    assert (np.sort(c, axis=1)[:, 1:] != np.sort(c, axis=1)[:, :-1]).all()
    with pytest.raises(ValueError):
        draw_connectivity(rng, 1, 7, 6)
    t = draw_tables(rng, 1000, 2)
    assert t.max() < 16 and len(np.unique(t)) == 16


def test_collapsed_routing_reads_at_most_three_wires():
    from paper_2602_07400_amd.workloads import make_workload
    wl = make_workload("c4_collapsed", n=64)
    w_in = wl.config.wires
    for conn, _ in wl.layers:
        assert conn.shape[1] == 6 and conn.min() >= 0 and conn.max() < w_in
        distinct = np.array([len(set(r)) for r in conn[:5000].tolist()])
        assert distinct.max() <= 3 and distinct.min() >= 1
        assert (distinct == 3).mean() > 0.5
        w_in = conn.shape[0]
