"""BitLogic CPU oracle -- TEST INFRASTRUCTURE ONLY.

Python front end of ``bitlogic_oracle.c``: a plain per-sample C implementation
of the paper's forward pass (thermometer encoder, LUT layers, GroupSum head and
argmax; Sec. 3 Eq. 1, App. C.1) on unpacked bytes, of the quantized
(DSP-backed) class head on the group sums (Sec. 3; Sec. 5 "Head"), of the
binary-coded encoder (Sec. 3; Sec. 5 "Encoder") and of quantile-threshold
fitting (Sec. 4 "Initialization"; App. B).  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The product library (``paper_2602_07400_amd``) never imports,
links or calls anything here, and the two share no code.

Every function is pinned by ``tests/test_oracle_pins.py`` against closed forms,
textbook truth tables, brute force and invariants; none is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bitlogic_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP over samples)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC",
                               "-Wall", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        lib.oracle_encode.argtypes = [P, i64, i32, P, i32, P]
        lib.oracle_lut_layer.argtypes = [P, i64, i32, P, P, i32, i32, P]
        lib.oracle_groupsum.argtypes = [P, i64, i32, i32, P, P]
        lib.oracle_forward.argtypes = [P, i64, i32, P, i32, i32, P, P, P, P,
                                       i32, P, P, i32]
        lib.oracle_grouped_dsp.argtypes = [P, i64, i32, P, P, P]
        lib.oracle_encode_binary.argtypes = [P, i64, i32, i32, P]
        lib.oracle_fit_quantiles.argtypes = [P, i64, i32, i32, i32, P]
        lib.oracle_forward_binary.argtypes = [P, i64, i32, i32, i32, P, P, P, P, i32, P, P, i32]
        lib.oracle_max_threads.argtypes = []
        for f in (lib.oracle_encode, lib.oracle_lut_layer, lib.oracle_groupsum,
                  lib.oracle_grouped_dsp, lib.oracle_forward, lib.oracle_max_threads,
                  lib.oracle_encode_binary, lib.oracle_fit_quantiles,
                  lib.oracle_forward_binary):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags.c_contiguous
    return a.ctypes.data


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError(f"{what}: oracle status {rc}")


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def encode(x: np.ndarray, thresholds: np.ndarray) -> np.ndarray:
    """x uint8 [n][d], thresholds uint8 [d][b] -> wires uint8 [n][d*b] (0/1)."""
    x = np.ascontiguousarray(x, dtype=np.uint8)
    th = np.ascontiguousarray(thresholds, dtype=np.uint8)
    n, d = x.shape
    assert th.shape[0] == d
    b = th.shape[1]
    e = np.empty((n, d * b), dtype=np.uint8)
    _check(_load().oracle_encode(_ptr(x), n, d, _ptr(th), b, _ptr(e)), "encode")
    return e


def lut_layer(v_in: np.ndarray, conn: np.ndarray, tables: np.ndarray) -> np.ndarray:
    """v_in uint8 [n][w_in] (0/1), conn int32 [w][k], tables uint64 [w] -> uint8 [n][w]."""
    v_in = np.ascontiguousarray(v_in, dtype=np.uint8)
    conn = np.ascontiguousarray(conn, dtype=np.int32)
    tables = np.ascontiguousarray(tables, dtype=np.uint64)
    n, w_in = v_in.shape
    w, k = conn.shape
    out = np.empty((n, w), dtype=np.uint8)
    _check(_load().oracle_lut_layer(_ptr(v_in), n, w_in, _ptr(conn), _ptr(tables),
                                    w, k, _ptr(out)), "lut_layer")
    return out


def groupsum(v: np.ndarray, n_classes: int):
    """v uint8 [n][w] (0/1) -> (scores int32 [n][c], pred int32 [n])."""
    v = np.ascontiguousarray(v, dtype=np.uint8)
    n, w = v.shape
    scores = np.empty((n, n_classes), dtype=np.int32)
    pred = np.empty((n,), dtype=np.int32)
    _check(_load().oracle_groupsum(_ptr(v), n, w, n_classes, _ptr(scores), _ptr(pred)),
           "groupsum")
    return scores, pred


def encode_binary(x: np.ndarray, n_bits: int) -> np.ndarray:
    """Binary-coded encoder: x uint8 [n][d] -> wires uint8 [n][d*b], wire f*b+t = bit t
    of round(x * (2^b - 1) / 255)."""
    x = np.ascontiguousarray(x, dtype=np.uint8)
    n, d = x.shape
    e = np.empty((n, d * n_bits), dtype=np.uint8)
    _check(_load().oracle_encode_binary(_ptr(x), n, d, n_bits, _ptr(e)), "encode_binary")
    return e


def fit_quantiles(x: np.ndarray, n_bits: int, n_groups: int = 1) -> np.ndarray:
    """Quantile thermometer thresholds fitted from x uint8 [n][d]: th uint8 [d][b], one
    ladder per contiguous group of d / n_groups features."""
    x = np.ascontiguousarray(x, dtype=np.uint8)
    n, d = x.shape
    th = np.empty((d, n_bits), dtype=np.uint8)
    _check(_load().oracle_fit_quantiles(_ptr(x), n, d, n_bits, n_groups, _ptr(th)),
           "fit_quantiles")
    return th


def grouped_dsp(counts: np.ndarray, weights: np.ndarray):
    """Quantized head: counts int32 [n][c], weights int8 [c][c] ->
    (logits int64 [n][c], pred int32 [n]); logit i = sum_j weights[i][j] * counts[j]."""
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    q = np.ascontiguousarray(weights, dtype=np.int8)
    n, c = counts.shape
    assert q.shape == (c, c)
    logits = np.empty((n, c), dtype=np.int64)
    pred = np.empty((n,), dtype=np.int32)
    _check(_load().oracle_grouped_dsp(_ptr(counts), n, c, _ptr(q), _ptr(logits), _ptr(pred)),
           "grouped_dsp")
    return logits, pred


def forward(x: np.ndarray, thresholds, layers, n_classes: int,
            n_threads: int = 0, binary_bits: int = 0):
    """Whole forward, per sample.  layers = [(conn int32 [w][k], tables uint64 [w]), ...].
    With binary_bits > 0 the binary-coded encoder replaces the thermometer
    (thresholds is then ignored).

    Returns (scores int32 [n][c], pred int32 [n]).
    """
    x = np.ascontiguousarray(x, dtype=np.uint8)
    n, d = x.shape
    if binary_bits:
        th, b = None, int(binary_bits)
    else:
        th = np.ascontiguousarray(thresholds, dtype=np.uint8)
        b = th.shape[1]
    conns = [np.ascontiguousarray(c, dtype=np.int32) for c, _ in layers]
    tabs = [np.ascontiguousarray(t, dtype=np.uint64) for _, t in layers]
    L = len(layers)
    conn_p = (ctypes.c_void_p * L)(*[_ptr(c) for c in conns])
    tab_p = (ctypes.c_void_p * L)(*[_ptr(t) for t in tabs])
    w_out = (ctypes.c_int32 * L)(*[c.shape[0] for c in conns])
    ks = (ctypes.c_int32 * L)(*[c.shape[1] for c in conns])
    scores = np.empty((n, n_classes), dtype=np.int32)
    pred = np.empty((n,), dtype=np.int32)
    ptrs = [ctypes.cast(conn_p, ctypes.c_void_p), ctypes.cast(tab_p, ctypes.c_void_p),
            ctypes.cast(w_out, ctypes.c_void_p), ctypes.cast(ks, ctypes.c_void_p)]
    if th is None:
        rc = _load().oracle_forward_binary(_ptr(x), n, d, b, L, *ptrs, n_classes, _ptr(scores),
                                           _ptr(pred), n_threads)
    else:
        rc = _load().oracle_forward(_ptr(x), n, d, _ptr(th), b, L, *ptrs, n_classes,
                                    _ptr(scores), _ptr(pred), n_threads)
    _check(rc, "forward")
    return scores, pred
