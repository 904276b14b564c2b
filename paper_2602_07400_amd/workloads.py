"""Seeded synthetic workloads shaped like the paper's image benchmarks.

This module only draws inputs: pixel batches, threshold ladders, connection
maps and truth tables.  It holds none of the forward pass's arithmetic; the
HIP path and the CPU oracle both receive its arrays byte-identically.

The paper evaluates on MNIST, Fashion-MNIST, CIFAR-10 and CIFAR-100 (Sec. 4
"Data"); none of these datasets is available here, so seeded synthetic arrays
with the same shapes stand in for them: 28x28 grey = 784 features or
32x32x3 = 3072 features (CHW flattening), 10 or 100 classes.

Readings of the paper used here:
* uniform ("linear") thermometer: b equispaced thresholds i/(b+1) of the
  value range (App. A "Initialization"), stored on the raw 0..255 scale as
  floor(255 * i / (b + 1));
* distributive (quantile) thermometer: thresholds are fit once from
  empirical pixel quantiles of a training split (App. A; App. B "MNIST-
  specific encoder collapse"), here per colour channel from a 256-bin
  histogram of a separate seeded training draw, theta_i = min{v : CDF(v) >=
  i/(b+1)};
* fixed random routing drawn once per layer, each node's k inputs distinct
  (Sec. 3 "Connectivity"; App. A "Initialization");
* random truth tables, 2^k entries in the low bits of a uint64 (bits >= 2^k
  are zero);
* collapsed routing (the "collapsed" configurations only): each node's k
  slots are drawn with repetition from a pool of 3 distinct wires of its own,
  so every node reads at most 3 distinct wires.  This stands in for the
  mode-collapsed full-pool router of Sec. 5 "Connectivity", where many slots
  converge on the same wires and a node's table reduces to a function of at
  most 3 effective inputs; it is the workload of table specialization.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import concurrent.futures as cf
import os
import zlib

import numpy as np

__all__ = ["Config", "CONFIGS", "CONFIG_ORDER", "Workload", "make_workload", "draw_connectivity",
           "draw_pooled_connectivity", "draw_tables", "uniform_thresholds"]


@dataclass(frozen=True)
class Config:
    name: str
    n: int                 # batch size (samples)
    d: int                 # input features
    b: int                 # thresholds per feature
    thresholds: str        # "fixed128" | "uniform" | "quantile"
    widths: Tuple[int, ...]
    k: int
    n_classes: int
    pixels: str            # "uniform" | "gaussian_mixture"
    channels: int = 1      # colour channels (quantile fit is per channel)
    description: str = ""
    family: str = ""       # configs of one family share their pixel and threshold draws
    pool: int = 0          # 0: distinct random routing; p > 0: collapsed routing from p wires

    @property
    def seed_key(self) -> str:
        return self.family or self.name

    @property
    def words(self) -> int:
        return (self.n + 63) // 64

    @property
    def wires(self) -> int:
        return self.d * self.b


CONFIGS = {
    "c1_mnist_tiny": Config(
        "c1_mnist_tiny", 4096, 784, 1, "fixed128", (1000, 1000), 6, 10, "uniform", 1,
        "MNIST-shaped tiny net: 4096 x 784 uniform pixels, one threshold at 128, "
        "2 x 1000 nodes, k=6, 10 classes x 100"),
    "c2_fmnist": Config(
        "c2_fmnist", 1 << 20, 784, 7, "uniform", (8000, 8000), 6, 10,
        "gaussian_mixture", 1,
        "Fashion-MNIST-shaped: 2^20 x 784 Gaussian-mixture pixels, 7 uniform "
        "thresholds, 2 x 8000 nodes, k=6, 10 classes x 800"),
    "c3_cifar10": Config(
        "c3_cifar10", 1 << 18, 3072, 3, "quantile", (32000, 32000), 6, 10, "uniform", 3,
        "CIFAR-10-shaped: 2^18 x 3072 uniform pixels, 3 per-channel quantile "
        "thresholds, 2 x 32000 nodes, k=6, 10 classes x 3200"),
    "c4_cifar100_wide": Config(
        "c4_cifar100_wide", 1 << 18, 3072, 7, "uniform", (64000, 64000), 6, 100,
        "uniform", 3,
        "CIFAR-100-shaped wide net: 2^18 x 3072 uniform pixels, 7 uniform "
        "thresholds, 2 x 64000 nodes, k=6, 100 classes x 640"),
}
for _k in (2, 4, 6):
    CONFIGS[f"c5_fanin_k{_k}"] = Config(
        f"c5_fanin_k{_k}", 1 << 18, 3072, 3, "quantile", (64000, 64000), _k, 10,
        "uniform", 3,
        f"fan-in sweep on the CIFAR-10 shape: 2^18 x 3072 uniform pixels, 3 "
        f"per-channel quantile thresholds, 2 x 64000 nodes, k={_k}, 10 classes x 6400",
        "c5_fanin")

# The network shape the paper deploys (Sec. 7 hardware table; App. C.1): its
# MNIST "best-of-space" network with a 4-threshold quantile thermometer on 784
# features (3136 wires), two layers of 4000 nodes of fan-in 4 and a
# 10-class popcount head, timed there at batches of 1024 and 64.  Random
# tables and uniform pixels stand in for the trained checkpoint and MNIST.
CONFIGS["paper_mnist_w4000"] = Config(
    "paper_mnist_w4000", 1024, 784, 4, "quantile", (4000, 4000), 4, 10, "uniform", 1,
    "the paper's deployed MNIST network shape: 784 features, 4 quantile thresholds "
    "(3136 wires), 2 x 4000 nodes, k=4, 10 classes x 400; batch 1024")

# Collapsed routing on the CIFAR-100 wide shape (every node reads at most 3
# distinct wires); the workload table specialization is measured on.
CONFIGS["c4_collapsed"] = Config(
    "c4_collapsed", 1 << 18, 3072, 7, "uniform", (64000, 64000), 6, 100, "uniform", 3,
    "CIFAR-100 wide shape with collapsed routing: each node's 6 slots drawn from 3 "
    "wires of its own", "c4_cifar100_wide", 3)

#: the order the configurations are listed in
CONFIG_ORDER = ["c1_mnist_tiny", "c2_fmnist", "c3_cifar10", "c4_cifar100_wide",
                "c5_fanin_k2", "c5_fanin_k4", "c5_fanin_k6"]

# stream slots of the root SeedSequence
_S_PIXELS, _S_PROTO, _S_TRAIN, _S_LAYERS = 0, 1, 2, 3
_GM_SIGMA = 48.0          # Gaussian-mixture spread (pixels)
_TRAIN_SPLIT = 8192       # samples in the threshold-fitting split


@dataclass
class Workload:
    config: Config
    x: np.ndarray                      # uint8 [n][d]
    thresholds: np.ndarray             # uint8 [d][b]
    layers: List[Tuple[np.ndarray, np.ndarray]]   # [(conn int32 [w][k], tables uint64 [w])]
    labels: Optional[np.ndarray] = None
    seed: int = 0
    dsp_weights: Optional[np.ndarray] = None   # int8 [c][c], quantized head weights

    @property
    def n_classes(self) -> int:
        return self.config.n_classes

    @property
    def n(self) -> int:
        return self.x.shape[0]


def _streams(seed: int, name: str, n_layers: int):
    # slots: pixels, prototypes, training split, (conn, tables) per layer, then
    # the quantized head's weights (appended last, so the others keep their draws)
    root = np.random.SeedSequence([seed, zlib.crc32(name.encode())])
    return root.spawn(_S_LAYERS + 2 * n_layers + 1)


def uniform_thresholds(d: int, b: int) -> np.ndarray:
    """b equispaced thresholds i/(b+1), i = 1..b, on the 0..255 scale."""
    ladder = np.array([(255 * i) // (b + 1) for i in range(1, b + 1)], dtype=np.uint8)
    return np.ascontiguousarray(np.broadcast_to(ladder, (d, b)))


def _quantile_thresholds(train: np.ndarray, b: int, channels: int) -> np.ndarray:
    n, d = train.shape
    per = d // channels
    th = np.empty((d, b), dtype=np.uint8)
    for ch in range(channels):
        vals = train[:, ch * per:(ch + 1) * per].ravel()
        cdf = np.cumsum(np.bincount(vals, minlength=256)) / vals.size
        ladder = [int(np.searchsorted(cdf, i / (b + 1), side="left")) for i in range(1, b + 1)]
        th[ch * per:(ch + 1) * per, :] = np.array(ladder, dtype=np.uint8)
    return th


_CHUNK = 1 << 14           # pixel rows per independently seeded chunk


def _pixel_chunks(n: int, d: int, ss: np.random.SeedSequence, fill) -> np.ndarray:
    """Fill x [n][d] chunk by chunk; chunk i draws from child i of ``ss``, so
    the bytes do not depend on how many threads run the chunks."""
    x = np.empty((n, d), dtype=np.uint8)
    n_chunks = (n + _CHUNK - 1) // _CHUNK
    kids = ss.spawn(n_chunks)

    def run(i):
        s0, s1 = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        fill(np.random.default_rng(kids[i]), x[s0:s1], s0, s1)

    workers = max(1, min(16, os.cpu_count() or 1, n_chunks))
    if workers == 1:
        for i in range(n_chunks):
            run(i)
    else:
        with cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(run, range(n_chunks)))
    return x


def _pixels(cfg: Config, n: int, ss: np.random.SeedSequence, proto_rng: np.random.Generator):
    if cfg.pixels == "uniform":
        def fill(rng, out, s0, s1):
            out[...] = np.frombuffer(rng.bytes(out.size), dtype=np.uint8).reshape(out.shape)
        return _pixel_chunks(n, cfg.d, ss, fill), None
    # Gaussian mixture of class prototypes, clipped to the pixel range
    protos = proto_rng.uniform(0.0, 255.0, size=(cfg.n_classes, cfg.d)).astype(np.float32)
    labels = proto_rng.integers(0, cfg.n_classes, size=n).astype(np.int32)

    def fill(rng, out, s0, s1):
        z = rng.standard_normal(size=out.shape, dtype=np.float32)
        z *= np.float32(_GM_SIGMA)
        z += protos[labels[s0:s1]]
        np.rint(z, out=z)
        np.clip(z, 0.0, 255.0, out=z)
        out[...] = z.astype(np.uint8)
    return _pixel_chunks(n, cfg.d, ss, fill), labels


def draw_connectivity(rng: np.random.Generator, w: int, k: int, w_in: int) -> np.ndarray:
    """Each node draws k distinct input indices uniformly from [0, w_in)."""
    if k > w_in:
        raise ValueError("fan-in larger than the layer input")
    conn = rng.integers(0, w_in, size=(w, k), dtype=np.int64)
    while True:
        s = np.sort(conn, axis=1)
        bad = np.nonzero((s[:, 1:] == s[:, :-1]).any(axis=1))[0] if k > 1 else np.array([], int)
        if bad.size == 0:
            break
        conn[bad] = rng.integers(0, w_in, size=(bad.size, k), dtype=np.int64)
    return conn.astype(np.int32)


def draw_pooled_connectivity(rng: np.random.Generator, w: int, k: int, w_in: int,
                             pool: int) -> np.ndarray:
    """Each node draws `pool` distinct wires of [0, w_in), then its k slots
    uniformly with repetition from them."""
    if pool > w_in:
        raise ValueError("pool larger than the layer input")
    base = draw_connectivity(rng, w, pool, w_in)
    pick = rng.integers(0, pool, size=(w, k))
    return np.take_along_axis(base, pick, axis=1).astype(np.int32)


def draw_tables(rng: np.random.Generator, w: int, k: int) -> np.ndarray:
    """Random 2^k-entry truth tables, entry a = bit a; unused high bits zero."""
    t = rng.integers(0, np.iinfo(np.uint64).max, size=w, dtype=np.uint64, endpoint=True)
    if k < 6:
        t &= np.uint64((1 << (1 << k)) - 1)
    return t


def draw_dsp_weights(rng: np.random.Generator, c: int) -> np.ndarray:
    """c x c weights of the quantized head, uniform on the signed 8-bit grid
    [-127, 127] that trained weights are snapped to."""
    return rng.integers(-127, 128, size=(c, c)).astype(np.int8)


def make_workload(name_or_cfg, seed: int = 0, n: Optional[int] = None) -> Workload:
    """Draw the inputs of one configuration.

    ``n`` overrides the batch size (reduced parity cases); connectivity,
    tables and thresholds do not depend on it.
    """
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    n = cfg.n if n is None else int(n)
    L = len(cfg.widths)
    ss = _streams(seed, cfg.seed_key, L)
    rngs = [np.random.default_rng(q) for q in ss]
    x, labels = _pixels(cfg, n, ss[_S_PIXELS], rngs[_S_PROTO])
    if cfg.thresholds == "fixed128":
        th = np.full((cfg.d, cfg.b), 128, dtype=np.uint8)
    elif cfg.thresholds == "uniform":
        th = uniform_thresholds(cfg.d, cfg.b)
    elif cfg.thresholds == "quantile":
        train, _ = _pixels(cfg, _TRAIN_SPLIT, ss[_S_TRAIN], np.random.default_rng(seed))
        th = _quantile_thresholds(train, cfg.b, cfg.channels)
    else:
        raise ValueError(cfg.thresholds)
    layers = []
    w_in = cfg.wires
    for l, w in enumerate(cfg.widths):
        if cfg.pool:
            conn = draw_pooled_connectivity(rngs[_S_LAYERS + 2 * l], w, cfg.k, w_in, cfg.pool)
        else:
            conn = draw_connectivity(rngs[_S_LAYERS + 2 * l], w, cfg.k, w_in)
        tables = draw_tables(rngs[_S_LAYERS + 2 * l + 1], w, cfg.k)
        layers.append((conn, tables))
        w_in = w
    dsp = draw_dsp_weights(rngs[_S_LAYERS + 2 * L], cfg.n_classes)
    return Workload(cfg, x, th, layers, labels, seed, dsp)
