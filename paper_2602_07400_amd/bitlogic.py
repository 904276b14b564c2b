"""Python binding of libbitlogic (C ABI in include/bitlogic.h).

Argument marshalling only: every step of the forward pass runs in the HIP
kernels of ``libbitlogic.so``.  Tensors are torch tensors on the GPU; their
``data_ptr()`` is handed to the C ABI together with the current HIP stream.
Packed bit tensors are ``torch.int64`` (the same 64 bits the C side reads as
``uint64``); ``torch.uint64`` tensors are accepted too.

If the shared library has not been built, every call raises: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

__all__ = [
    "BitlogicError", "bitlogic_encode", "bitlogic_lut_layer", "bitlogic_groupsum_head",
    "bitlogic_forward", "bitlogic_forward_timed", "bitlogic_forward_workspace_bytes",
    "bitlogic_forward_plan", "bitlogic_grouped_dsp_head", "bitlogic_forward_grouped_dsp",
    "bitlogic_encode_binary", "bitlogic_fit_quantile_thresholds", "bitlogic_network_forward",
    "bitlogic_network_forward_noalloc", "NOALLOC_SCRATCH_BYTES",
    "bitlogic_groupsum_head_workspace_bytes", "bitlogic_status_string", "bitlogic_version",
    "BitlogicModel", "bitlogic_specialize_layer", "bitlogic_specialize_network", "library_path",
    "load_library", "words",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libbitlogic.so")

OK = 0
_lib = None


class BitlogicError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"bitlogic status {status} ({bitlogic_status_string(status)}): {detail}")


class _ForwardInfo(ctypes.Structure):
    _fields_ = [("workspace_bytes", ctypes.c_size_t), ("slab_words", ctypes.c_int32),
                ("fused_head", ctypes.c_int32), ("head_splits", ctypes.c_int32),
                ("head_planes", ctypes.c_int32), ("jump_layers", ctypes.c_uint32)]


class _Layer(ctypes.Structure):
    _fields_ = [("conn", ctypes.c_void_p), ("tables", ctypes.c_void_p),
                ("w_out", ctypes.c_int32), ("k", ctypes.c_int32)]


ENCODER_THERMOMETER, ENCODER_BINARY = 0, 1
HEAD_GROUPSUM, HEAD_GROUPED_DSP = 0, 1


class _Network(ctypes.Structure):
    _fields_ = [("n_features", ctypes.c_int32), ("encoder", ctypes.c_int32),
                ("n_bits", ctypes.c_int32), ("thresholds", ctypes.c_void_p),
                ("layers", ctypes.c_void_p), ("n_layers", ctypes.c_int32),
                ("n_classes", ctypes.c_int32), ("head", ctypes.c_int32),
                ("head_weights", ctypes.c_void_p), ("pass_fanin", ctypes.c_void_p)]


MAX_FANIN = 6
SPECIALIZE_PASS = 32          # nodes per entry of a specialized layer's fan-in array


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libbitlogic.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"{_LIB_PATH} is missing: build it with __graft_entry__.build() "
            "(hipcc --offload-arch=gfx950); there is no fallback path")
    lib = ctypes.CDLL(_LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "bitlogic_encode": ([P, i64, i32, P, i32, P, P], ctypes.c_int),
        "bitlogic_lut_layer": ([P, i32, i64, P, P, i32, i32, P, P], ctypes.c_int),
        "bitlogic_groupsum_head_workspace_bytes": ([i32, i64, i32], sz),
        "bitlogic_groupsum_head": ([P, i32, i64, i32, P, P, P, sz, P], ctypes.c_int),
        "bitlogic_forward_workspace_bytes": ([i64, i32, i32, P, i32, i32], sz),
        "bitlogic_forward_plan": ([i64, i32, i32, P, i32, i32, P], ctypes.c_int),
        "bitlogic_grouped_dsp_head": ([P, i64, i32, P, P, P, P], ctypes.c_int),
        "bitlogic_encode_binary": ([P, i64, i32, i32, P, P], ctypes.c_int),
        "bitlogic_fit_quantile_thresholds_workspace_bytes": ([i32], sz),
        "bitlogic_fit_quantile_thresholds": ([P, i64, i32, i32, i32, P, P, sz, P], ctypes.c_int),
        "bitlogic_network_workspace_bytes": ([P, i64], sz),
        "bitlogic_network_plan": ([P, i64, P], ctypes.c_int),
        "bitlogic_network_forward": ([P, P, i64, P, P, P, sz, P, P, i32], ctypes.c_int),
        "bitlogic_network_forward_noalloc": ([P, P, i64, P, P, P], ctypes.c_int),
        "bitlogic_forward_grouped_dsp": ([P, i64, i32, P, i32, P, i32, i32, P, P, P, P, sz, P],
                                         ctypes.c_int),
        "bitlogic_forward": ([P, i64, i32, P, i32, P, i32, i32, P, P, P, sz, P], ctypes.c_int),
        "bitlogic_forward_timed": ([P, i64, i32, P, i32, P, i32, i32, P, P, P, sz, P, P, i32],
                                   ctypes.c_int),
        "bitlogic_specialize_layer": ([P, P, i32, i32, i32, P, P, P], ctypes.c_int),
        "bitlogic_specialize_network": ([i32, P, P, P, P, i32, i32, ctypes.c_double, P, P, P,
                                         P, P, P], ctypes.c_int),
        "bitlogic_probe_valu": ([P, i32, i32, ctypes.c_uint32, P], ctypes.c_int),
        "bitlogic_probe_hbm": ([i32, P, P, i64, i32, i32, P], ctypes.c_int),
        "bitlogic_probe_valu_op": ([i32, P, i32, i32, ctypes.c_uint32, P], ctypes.c_int),
        "bitlogic_probe_gather": ([P, i64, i32, i32, i32, i32, i32, ctypes.c_uint32, P, P, P],
                                  ctypes.c_int),
        "bitlogic_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "bitlogic_last_error": ([], ctypes.c_char_p),
        "bitlogic_version": ([], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def bitlogic_status_string(status: int) -> str:
    return load_library().bitlogic_status_string(int(status)).decode()


def bitlogic_version() -> int:
    return int(load_library().bitlogic_version())


def _check(rc: int) -> None:
    if rc != OK:
        raise BitlogicError(rc, load_library().bitlogic_last_error().decode())


def words(n_samples: int) -> int:
    return (int(n_samples) + 63) // 64


def _stream(stream, device) -> int:
    if stream is None:
        return torch.cuda.current_stream(device).cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dev(t: torch.Tensor, name: str, dtypes) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


_U8 = (torch.uint8,)
_I32 = (torch.int32,)
_U64 = (torch.int64, torch.uint64)


def bitlogic_encode(x: torch.Tensor, thresholds: torch.Tensor,
                    bits_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """x uint8 [N][d], thresholds uint8 [d][b] -> packed wires int64 [d*b][ceil(N/64)]."""
    n, d = x.shape
    b = thresholds.shape[1]
    if bits_out is None:
        bits_out = _empty((d * b, words(n)), torch.int64, x.device, stream)
    _check(load_library().bitlogic_encode(
        _dev(x, "x", _U8), n, d, _dev(thresholds, "thresholds", _U8), b,
        _dev(bits_out, "bits_out", _U64), _stream(stream, x.device)))
    return bits_out


def bitlogic_lut_layer(bits_in: torch.Tensor, conn: torch.Tensor, tables: torch.Tensor,
                       bits_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """bits_in [w_in][W], conn int32 [w][k], tables [w] -> bits_out [w][W]."""
    w_in, n_words = bits_in.shape
    w, k = conn.shape
    if bits_out is None:
        bits_out = _empty((w, n_words), torch.int64, bits_in.device, stream)
    _check(load_library().bitlogic_lut_layer(
        _dev(bits_in, "bits_in", _U64), w_in, n_words, _dev(conn, "conn", _I32),
        _dev(tables, "tables", _U64), w, k, _dev(bits_out, "bits_out", _U64),
        _stream(stream, bits_in.device)))
    return bits_out


def bitlogic_groupsum_head_workspace_bytes(w: int, n_samples: int, n_classes: int) -> int:
    return int(load_library().bitlogic_groupsum_head_workspace_bytes(w, n_samples, n_classes))


def _on_stream(t: Optional[torch.Tensor], handle: int, device) -> Optional[torch.Tensor]:
    """Tell torch's caching allocator that a tensor this module allocated is used
    on the HIP stream `handle`, when that is not the current stream: its memory
    is then not handed out again before the stream's work on it is done."""
    if t is not None and handle != torch.cuda.current_stream(device).cuda_stream:
        t.record_stream(torch.cuda.ExternalStream(handle, device=device))
    return t


def _empty(shape, dtype, device, stream) -> torch.Tensor:
    """An output this module allocates for a call on `stream` (see _on_stream)."""
    return _on_stream(torch.empty(shape, dtype=dtype, device=device), _stream(stream, device),
                      device)


def _workspace(nbytes: int, device, given: Optional[torch.Tensor],
               handle: Optional[int] = None) -> Tuple[int, int]:
    if given is not None:
        return _dev(given, "workspace", (torch.uint8,)), given.numel()
    if nbytes == 0:
        return 0, 0
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
    if handle is not None:
        _on_stream(buf, handle, device)
    _workspace.keep = buf        # kept alive until the next call allocates one
    return buf.data_ptr(), nbytes


def bitlogic_groupsum_head(bits: torch.Tensor, n_samples: int, n_classes: int,
                           scores: Optional[torch.Tensor] = None,
                           argmax: Optional[torch.Tensor] = None,
                           workspace: Optional[torch.Tensor] = None, stream=None,
                           want_scores: bool = True):
    """bits [w][W] -> (scores int32 [N][c] or None, argmax int32 [N])."""
    w = bits.shape[0]
    dev = bits.device
    if scores is None and want_scores:
        scores = _empty((n_samples, n_classes), torch.int32, dev, stream)
    if argmax is None:
        argmax = _empty((n_samples,), torch.int32, dev, stream)
    ws_ptr, ws_bytes = _workspace(bitlogic_groupsum_head_workspace_bytes(w, n_samples, n_classes),
                                  dev, workspace, _stream(stream, dev))
    _check(load_library().bitlogic_groupsum_head(
        _dev(bits, "bits", _U64), w, n_samples, n_classes,
        _dev(scores, "scores", _I32) if scores is not None else None,
        _dev(argmax, "argmax", _I32), ws_ptr, ws_bytes, _stream(stream, dev)))
    return scores, argmax


def _layer_array(layers: Sequence[Tuple[torch.Tensor, torch.Tensor]]):
    arr = (_Layer * len(layers))()
    for l, (conn, tables) in enumerate(layers):
        arr[l].conn = _dev(conn, f"conn[{l}]", _I32)
        arr[l].tables = _dev(tables, f"tables[{l}]", _U64)
        arr[l].w_out = conn.shape[0]
        arr[l].k = conn.shape[1]
    return arr


def bitlogic_forward_workspace_bytes(n_samples: int, n_features: int, n_thresholds: int,
                                     layers, n_classes: int) -> int:
    arr = _layer_array(layers)
    return int(load_library().bitlogic_forward_workspace_bytes(
        n_samples, n_features, n_thresholds, ctypes.cast(arr, ctypes.c_void_p), len(layers),
        n_classes))


def bitlogic_forward_plan(n_samples: int, n_features: int, n_thresholds: int,
                          layers, n_classes: int) -> dict:
    """How bitlogic_forward runs this shape: workspace size, slab width, whether
    the last layer is fused with the head, and the head's counter layout."""
    arr = _layer_array(layers)
    info = _ForwardInfo()
    _check(load_library().bitlogic_forward_plan(
        n_samples, n_features, n_thresholds, ctypes.cast(arr, ctypes.c_void_p), len(layers),
        n_classes, ctypes.byref(info)))
    return {"workspace_bytes": int(info.workspace_bytes), "slab_words": int(info.slab_words),
            "fused_head": bool(info.fused_head), "head_splits": int(info.head_splits),
            "head_planes": int(info.head_planes)}


_I8 = (torch.int8,)


def bitlogic_encode_binary(x: torch.Tensor, n_bits: int,
                           bits_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Binary-coded encoder: pixels uint8 [N][d] -> packed int64 [d*n_bits][ceil(N/64)];
    wire f*n_bits+t = bit t of round(x * (2^n_bits - 1) / 255)."""
    n, d = x.shape
    if bits_out is None:
        bits_out = _empty((d * n_bits, words(n)), torch.int64, x.device, stream)
    _check(load_library().bitlogic_encode_binary(_dev(x, "x", _U8), n, d, int(n_bits),
                                                 _dev(bits_out, "bits_out", _U64),
                                                 _stream(stream, x.device)))
    return bits_out


def bitlogic_fit_quantile_thresholds(x: torch.Tensor, n_thresholds: int, n_groups: int = 1,
                                     out: Optional[torch.Tensor] = None,
                                     workspace: Optional[torch.Tensor] = None,
                                     stream=None) -> torch.Tensor:
    """Quantile thermometer thresholds fitted from pixels uint8 [N][d]: uint8
    [d][n_thresholds], one ladder per contiguous group of d / n_groups features."""
    n, d = x.shape
    dev = x.device
    if out is None:
        out = _empty((d, n_thresholds), torch.uint8, dev, stream)
    lib = load_library()
    need = int(lib.bitlogic_fit_quantile_thresholds_workspace_bytes(int(n_groups)))
    ws_ptr, ws_bytes = _workspace(max(need, 8), dev, workspace, _stream(stream, dev))
    _check(lib.bitlogic_fit_quantile_thresholds(_dev(x, "x", _U8), n, d, int(n_thresholds),
                                                int(n_groups), _dev(out, "out", _U8), ws_ptr,
                                                ws_bytes, _stream(stream, dev)))
    return out


def bitlogic_grouped_dsp_head(counts: torch.Tensor, weights: torch.Tensor,
                              logits: Optional[torch.Tensor] = None,
                              argmax: Optional[torch.Tensor] = None, stream=None,
                              want_logits: bool = True):
    """Quantized head: counts int32 [N][c] (0..65535), weights int8 [c][c] ->
    (logits int32 [N][c], argmax int32 [N]); logit i = sum_j weights[i][j] * counts[j]."""
    n, c = counts.shape
    dev = counts.device
    if tuple(weights.shape) != (c, c):
        raise ValueError(f"weights must be [{c}][{c}]")
    if logits is None and want_logits:
        logits = _empty((n, c), torch.int32, dev, stream)
    if argmax is None:
        argmax = _empty((n,), torch.int32, dev, stream)
    _check(load_library().bitlogic_grouped_dsp_head(
        _dev(counts, "counts", _I32), n, c, _dev(weights, "weights", _I8),
        _dev(logits, "logits", _I32) if logits is not None else None,
        _dev(argmax, "argmax", _I32), _stream(stream, dev)))
    return logits, argmax


def bitlogic_forward_grouped_dsp(x: torch.Tensor, thresholds: torch.Tensor,
                                 layers: Sequence[Tuple[torch.Tensor, torch.Tensor]],
                                 n_classes: int, weights: torch.Tensor,
                                 logits: Optional[torch.Tensor] = None,
                                 argmax: Optional[torch.Tensor] = None,
                                 workspace: Optional[torch.Tensor] = None, stream=None,
                                 want_logits: bool = True):
    """Whole forward with the quantized head: pixels uint8 [N][d] ->
    (logits int32 [N][c], argmax int32 [N])."""
    n, d = x.shape
    b = thresholds.shape[1]
    dev = x.device
    arr = _layer_array(layers)
    lib = load_library()
    need = int(lib.bitlogic_forward_workspace_bytes(
        n, d, b, ctypes.cast(arr, ctypes.c_void_p), len(arr), n_classes))
    if logits is None and want_logits:
        logits = _empty((n, n_classes), torch.int32, dev, stream)
    if argmax is None:
        argmax = _empty((n,), torch.int32, dev, stream)
    ws_ptr, ws_bytes = _workspace(need, dev, workspace, _stream(stream, dev))
    _check(lib.bitlogic_forward_grouped_dsp(
        _dev(x, "x", _U8), n, d, _dev(thresholds, "thresholds", _U8), b,
        ctypes.cast(arr, ctypes.c_void_p), len(arr), n_classes, _dev(weights, "weights", _I8),
        _dev(logits, "logits", _I32) if logits is not None else None,
        _dev(argmax, "argmax", _I32), ws_ptr, ws_bytes, _stream(stream, dev)))
    return logits, argmax


def _forward(x, thresholds, layers, n_classes, scores, argmax, workspace, stream, want_scores,
             events):
    n, d = x.shape
    b = thresholds.shape[1]
    dev = x.device
    arr = _layer_array(layers)
    lib = load_library()
    need = int(lib.bitlogic_forward_workspace_bytes(
        n, d, b, ctypes.cast(arr, ctypes.c_void_p), len(arr), n_classes))
    if scores is None and want_scores:
        scores = _empty((n, n_classes), torch.int32, dev, stream)
    if argmax is None:
        argmax = _empty((n,), torch.int32, dev, stream)
    ws_ptr, ws_bytes = _workspace(need, dev, workspace, _stream(stream, dev))
    args = [_dev(x, "x", _U8), n, d, _dev(thresholds, "thresholds", _U8), b,
            ctypes.cast(arr, ctypes.c_void_p), len(arr), n_classes,
            _dev(scores, "scores", _I32) if scores is not None else None,
            _dev(argmax, "argmax", _I32), ws_ptr, ws_bytes, _stream(stream, dev)]
    if events is None:
        _check(lib.bitlogic_forward(*args))
    else:
        handles = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
        _check(lib.bitlogic_forward_timed(*args, ctypes.cast(handles, ctypes.c_void_p),
                                          len(events)))
    return scores, argmax


def bitlogic_forward(x: torch.Tensor, thresholds: torch.Tensor,
                     layers: Sequence[Tuple[torch.Tensor, torch.Tensor]], n_classes: int,
                     scores: Optional[torch.Tensor] = None,
                     argmax: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None,
                     want_scores: bool = True):
    """Whole forward: pixels uint8 [N][d] -> (scores int32 [N][c], argmax int32 [N])."""
    return _forward(x, thresholds, layers, n_classes, scores, argmax, workspace, stream,
                    want_scores, None)


def bitlogic_forward_timed(x: torch.Tensor, thresholds: torch.Tensor,
                           layers: Sequence[Tuple[torch.Tensor, torch.Tensor]], n_classes: int,
                           events: Sequence["torch.cuda.Event"],
                           scores: Optional[torch.Tensor] = None,
                           argmax: Optional[torch.Tensor] = None,
                           workspace: Optional[torch.Tensor] = None, stream=None,
                           want_scores: bool = True):
    """bitlogic_forward with torch.cuda.Events recorded at the stage boundaries
    (len(layers) + 3 events, created with enable_timing=True and recorded once
    beforehand so that their HIP handles exist)."""
    return _forward(x, thresholds, layers, n_classes, scores, argmax, workspace, stream,
                    want_scores, list(events))


def bitlogic_specialize_layer(conn, tables, w_in: int):
    """Table specialization of one layer on the host (bitlogic_specialize_layer):
    conn int32 [w][k], tables uint64 [w] -> (k_eff int32 [w], conn_eff int32
    [w][k] with slots past k_eff zero, tables_eff uint64 [w])."""
    conn = np.ascontiguousarray(conn, dtype=np.int32)
    tables = np.ascontiguousarray(tables, dtype=np.uint64)
    if conn.ndim != 2 or tables.shape != (conn.shape[0],):
        raise ValueError("conn [w][k] and tables [w] expected")
    w, k = conn.shape
    k_eff = np.zeros(w, dtype=np.int32)
    conn_eff = np.zeros_like(conn)
    tables_eff = np.zeros_like(tables)
    _check(load_library().bitlogic_specialize_layer(
        conn.ctypes.data, tables.ctypes.data, w, k, int(w_in), k_eff.ctypes.data,
        conn_eff.ctypes.data, tables_eff.ctypes.data))
    return k_eff, conn_eff, tables_eff


def bitlogic_specialize_network(layers, w_in: int, n_classes: int, min_gain: float = 0.0):
    """Table specialization of a whole network on the host
    (bitlogic_specialize_network): layers [(conn int32 [w][k], tables uint64
    [w])] -> [(conn, tables, fanin uint8 [ceil(w / 32)] or None, order int32
    [w])] per layer.  A specialized layer has its nodes reordered by effective
    fan-in and the largest effective fan-in as its width; a layer that would
    save less than min_gain of its multiplexers is kept (fanin None)."""
    conns = [np.ascontiguousarray(c, dtype=np.int32) for c, _ in layers]
    tabs = [np.ascontiguousarray(t, dtype=np.uint64) for _, t in layers]
    L = len(layers)
    outs = [(np.zeros_like(c), np.zeros_like(t),
             np.zeros((c.shape[0] + SPECIALIZE_PASS - 1) // SPECIALIZE_PASS, np.uint8),
             np.zeros(c.shape[0], np.int32)) for c, t in zip(conns, tabs)]
    arr = lambda xs, ty: (ty * L)(*[x.ctypes.data for x in xs])
    P = ctypes.c_void_p
    k_out = (ctypes.c_int32 * L)()
    applied = (ctypes.c_int32 * L)()
    _check(load_library().bitlogic_specialize_network(
        int(w_in), arr(conns, P), arr(tabs, P),
        (ctypes.c_int32 * L)(*[c.shape[0] for c in conns]),
        (ctypes.c_int32 * L)(*[c.shape[1] for c in conns]), L, int(n_classes),
        float(min_gain), k_out, applied,
        arr([o[0] for o in outs], P), arr([o[1] for o in outs], P),
        arr([o[2] for o in outs], P), arr([o[3] for o in outs], P)))
    res = []
    for (c, t, f, o), kn, a in zip(outs, k_out, applied):
        w = c.shape[0]
        res.append((np.ascontiguousarray(c.reshape(-1)[:w * kn].reshape(w, kn)), t,
                    f if a else None, o))
    return res


@dataclass
class BitlogicModel:
    """A network resident in device memory: encoder (thermometer thresholds, or
    the binary code width), per-layer conn/tables, and the class head."""
    thresholds: Optional[torch.Tensor]
    layers: List[Tuple[torch.Tensor, torch.Tensor]]
    n_classes: int
    n_features: int = 0
    encoder: int = ENCODER_THERMOMETER
    n_bits: int = 0
    head: int = HEAD_GROUPSUM
    head_weights: Optional[torch.Tensor] = None
    # specialized network: per layer the fan-in of each run of 32 nodes
    # (device), the node count per effective fan-in 0..6 and the original
    # node at each position
    pass_fanin: Optional[List[torch.Tensor]] = None
    fanin_histogram: Optional[list] = None
    order: Optional[list] = None

    def __post_init__(self):
        if self.thresholds is not None and self.encoder == ENCODER_THERMOMETER:
            self.n_features, self.n_bits = (int(v) for v in self.thresholds.shape)

    @classmethod
    def from_numpy(cls, thresholds, layers, n_classes: int, device="cuda",
                   encoder: str = "thermometer", n_features: Optional[int] = None,
                   n_bits: Optional[int] = None, head_weights=None,
                   specialize=False) -> "BitlogicModel":
        """Copy a host model to the GPU, checking every connection index.
        encoder "thermometer" takes thresholds uint8 [d][b]; "binary" takes
        n_features and n_bits (thresholds None).  head_weights int8 [c][c]
        selects the quantized head.  specialize=True evaluates the network
        from its specialized tables (bitlogic_specialize_network: tied and
        ignored inputs removed, nodes ordered by effective fan-in) wherever a
        layer saves at least 10% of its multiplexers; a float sets that
        fraction (0.0: every layer)."""
        if encoder == "thermometer":
            th = np.ascontiguousarray(thresholds, dtype=np.uint8)
            if th.ndim != 2:
                raise ValueError("thresholds must be [d][b]")
            d, b = th.shape
            th_dev, kind = torch.from_numpy(th).to(device), ENCODER_THERMOMETER
        elif encoder == "binary":
            if n_features is None or n_bits is None:
                raise ValueError("the binary encoder needs n_features and n_bits")
            d, b = int(n_features), int(n_bits)
            th_dev, kind = None, ENCODER_BINARY
        else:
            raise ValueError(f"unknown encoder {encoder!r}")
        w_in = d * b
        dev_layers, host_layers = [], []
        for l, (conn, tables) in enumerate(layers):
            conn = np.ascontiguousarray(conn, dtype=np.int32)
            tables = np.ascontiguousarray(tables, dtype=np.uint64)
            if conn.ndim != 2 or tables.shape != (conn.shape[0],):
                raise ValueError(f"layer {l}: conn [w][k] and tables [w] expected")
            if conn.size and (conn.min() < 0 or conn.max() >= w_in):
                raise ValueError(f"layer {l}: connection index outside [0, {w_in})")
            host_layers.append((conn, tables))
            w_in = conn.shape[0]
        if w_in % n_classes != 0:
            raise ValueError("last width must be a multiple of n_classes")
        fanin = hist = order = None
        if specialize is not False and specialize is not None:
            gain = 0.1 if specialize is True else float(specialize)
            spec = bitlogic_specialize_network(host_layers, d * b, n_classes, gain)
            hist, w_prev = [], d * b
            for (conn, tables), sp in zip(host_layers, spec):
                k_eff, _, _ = bitlogic_specialize_layer(conn, tables, w_prev)
                hist.append(None if sp[2] is None else
                            np.bincount(k_eff, minlength=MAX_FANIN + 1))
                w_prev = conn.shape[0]
            host_layers = [(c, t) for c, t, _, _ in spec]
            fanin = [None if f is None else torch.from_numpy(f).to(device)
                     for _, _, f, _ in spec]
            order = [o for _, _, _, o in spec]
            if all(f is None for f in fanin):
                fanin = None
        for conn, tables in host_layers:
            dev_layers.append((torch.from_numpy(conn).to(device),
                               torch.from_numpy(tables.view(np.int64)).to(device)))
        hw, head = None, HEAD_GROUPSUM
        if head_weights is not None:
            q = np.ascontiguousarray(head_weights, dtype=np.int8)
            if q.shape != (n_classes, n_classes):
                raise ValueError("head_weights must be [c][c]")
            hw, head = torch.from_numpy(q).to(device), HEAD_GROUPED_DSP
        return cls(th_dev, dev_layers, int(n_classes), d, kind, b, head, hw, fanin, hist, order)

    def _fanin_array(self):
        if not self.pass_fanin:
            return None, None
        ptrs = (ctypes.c_void_p * len(self.layers))(
            *[None if f is None else _dev(f, "pass_fanin", (torch.uint8,))
              for f in self.pass_fanin])
        return ctypes.cast(ptrs, ctypes.c_void_p), ptrs

    def _net(self):
        arr = _layer_array(self.layers)
        net = _Network()
        net.n_features, net.encoder, net.n_bits = self.n_features, self.encoder, self.n_bits
        net.thresholds = (_dev(self.thresholds, "thresholds", _U8)
                          if self.thresholds is not None else None)
        net.layers = ctypes.cast(arr, ctypes.c_void_p)
        net.n_layers = len(self.layers)
        net.n_classes = self.n_classes
        net.head = self.head
        net.head_weights = (_dev(self.head_weights, "head_weights", _I8)
                            if self.head_weights is not None else None)
        net.pass_fanin, keep = self._fanin_array()
        return net, (arr, keep)

    def workspace_bytes(self, n_samples: int) -> int:
        net, keep = self._net()
        return int(load_library().bitlogic_network_workspace_bytes(ctypes.byref(net),
                                                                   n_samples))

    def plan(self, n_samples: int) -> dict:
        net, keep = self._net()
        info = _ForwardInfo()
        _check(load_library().bitlogic_network_plan(ctypes.byref(net), n_samples,
                                                    ctypes.byref(info)))
        return {"workspace_bytes": int(info.workspace_bytes), "slab_words": int(info.slab_words),
                "fused_head": bool(info.fused_head), "head_splits": int(info.head_splits),
                "head_planes": int(info.head_planes),
                "jump_layers": [l for l in range(min(len(self.layers), 32))
                                if (int(info.jump_layers) >> l) & 1]}

    def forward(self, x: torch.Tensor, out: Optional[torch.Tensor] = None,
                argmax: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None, events=None, want_scores: bool = True):
        """pixels uint8 [N][d] -> (scores or logits int32 [N][c], argmax int32 [N])."""
        return bitlogic_network_forward(self, x, out, argmax, workspace, stream, events,
                                        want_scores)


def bitlogic_network_forward(model: BitlogicModel, x: torch.Tensor,
                             out: Optional[torch.Tensor] = None,
                             argmax: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None, stream=None,
                             events=None, want_scores: bool = True):
    """Forward of a BitlogicModel through bitlogic_network_forward."""
    n, d = x.shape
    if d != model.n_features:
        raise ValueError(f"x has {d} features, the model {model.n_features}")
    dev = x.device
    net, keep = model._net()
    lib = load_library()
    need = int(lib.bitlogic_network_workspace_bytes(ctypes.byref(net), n))
    if out is None and want_scores:
        out = _empty((n, model.n_classes), torch.int32, dev, stream)
    if argmax is None:
        argmax = _empty((n,), torch.int32, dev, stream)
    ws_ptr, ws_bytes = _workspace(need, dev, workspace, _stream(stream, dev))
    if events is None:
        ev_ptr, n_ev = None, 0
    else:
        handles = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
        ev_ptr, n_ev = ctypes.cast(handles, ctypes.c_void_p), len(events)
    _check(lib.bitlogic_network_forward(
        ctypes.byref(net), _dev(x, "x", _U8), n,
        _dev(out, "out", _I32) if out is not None else None, _dev(argmax, "argmax", _I32),
        ws_ptr, ws_bytes, _stream(stream, dev), ev_ptr, n_ev))
    return out, argmax


# bitlogic_network_forward_noalloc's static scratch per GPU (the header's
# BITLOGIC_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 64 << 20


def bitlogic_network_forward_noalloc(model: BitlogicModel, x: torch.Tensor, out: torch.Tensor,
                                     argmax: torch.Tensor, stream=None):
    """Forward of a BitlogicModel through bitlogic_network_forward_noalloc: the
    library's static scratch replaces the workspace.  out (int32 [N][c] or
    None) and argmax (int32 [N] or None) are the caller's buffers; nothing is
    allocated here or in the library."""
    n, d = x.shape
    if d != model.n_features:
        raise ValueError(f"x has {d} features, the model {model.n_features}")
    net, keep = model._net()
    _check(load_library().bitlogic_network_forward_noalloc(
        ctypes.byref(net), _dev(x, "x", _U8), n,
        _dev(out, "out", _I32) if out is not None else None,
        _dev(argmax, "argmax", _I32) if argmax is not None else None, _stream(stream, x.device)))
    return out, argmax


# ---------------------------------------------------------------- peak probes

PROBE_THREADS = 256
PROBE_CHAINS = 8


def bitlogic_probe_valu(out: torch.Tensor, blocks: int, iters: int, seed: int = 0,
                        stream=None) -> int:
    """Integer VALU probe into out (int32 [blocks * 256] on the GPU); returns
    the number of 32-bit lane-ops it performs (blocks * 256 * iters * 8)."""
    if out.numel() < blocks * PROBE_THREADS:
        raise ValueError("out needs blocks * 256 words")
    _check(load_library().bitlogic_probe_valu(_dev(out, "out", _I32), int(blocks), int(iters),
                                              int(seed) & 0xFFFFFFFF,
                                              _stream(stream, out.device)))
    return int(blocks) * PROBE_THREADS * int(iters) * PROBE_CHAINS


PROBE_HBM_COPY, PROBE_HBM_READ, PROBE_HBM_WRITE = 0, 1, 2


def bitlogic_probe_hbm(mode: int, src: Optional[torch.Tensor], dst: torch.Tensor,
                       nbytes: Optional[int] = None, unroll: int = 4, blocks: int = 0,
                       stream=None) -> int:
    """HBM streaming probe (include/bitlogic.h): copy src into dst, read src
    (dst[0:16] receives the XOR of its 16-byte pieces) or write dst's
    pattern; returns the HBM bytes it moves (read + written)."""
    for t, name in ((src, "src"), (dst, "dst")):
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous GPU tensor")
    size = lambda t: t.numel() * t.element_size()
    if nbytes is None:
        nbytes = size(dst) if mode == PROBE_HBM_WRITE else size(src)
    if mode != PROBE_HBM_WRITE and nbytes > size(src):
        raise ValueError("src is smaller than nbytes")
    if mode != PROBE_HBM_READ and nbytes > size(dst):
        raise ValueError("dst is smaller than nbytes")
    if mode == PROBE_HBM_READ and size(dst) < 16:
        raise ValueError("the read probe writes 16 bytes")
    dev = dst.device
    _check(load_library().bitlogic_probe_hbm(
        int(mode), src.data_ptr() if src is not None else None, dst.data_ptr(), int(nbytes),
        int(unroll), int(blocks), _stream(stream, dev)))
    return (2 if mode == PROBE_HBM_COPY else 1) * int(nbytes)


PROBE_OP_MUX, PROBE_OP_MUX_BANK, PROBE_OP_BFE = 0, 1, 2


def bitlogic_probe_valu_op(op: int, out: torch.Tensor, blocks: int, iters: int, seed: int = 0,
                           stream=None) -> int:
    """Instruction-rate probe (include/bitlogic.h) into out (int32 [blocks * 256]
    on the GPU); returns the wave instructions it issues."""
    if out.numel() < blocks * PROBE_THREADS:
        raise ValueError("out needs blocks * 256 words")
    _check(load_library().bitlogic_probe_valu_op(int(op), _dev(out, "out", _I32), int(blocks),
                                                 int(iters), int(seed) & 0xFFFFFFFF,
                                                 _stream(stream, out.device)))
    return int(blocks) * 4 * int(iters) * 64


def bitlogic_probe_gather(rows: torch.Tensor, lanes_per_row: int, valu_per_pass: int,
                          blocks: int, passes: int, out: torch.Tensor,
                          sink: Optional[torch.Tensor] = None, waves_per_simd: int = 0,
                          seed: int = 0, stream=None) -> int:
    """Gather probe (include/bitlogic.h) over rows (a contiguous GPU tensor of
    n_rows * 128 bytes); returns the 128-byte rows it gathers."""
    nbytes = rows.numel() * rows.element_size()
    if nbytes % 128:
        raise ValueError("rows must be whole 128-byte rows")
    if out.numel() < blocks * PROBE_THREADS:
        raise ValueError("out needs blocks * 256 words")
    if sink is not None and sink.numel() * sink.element_size() < blocks * passes * 8192:
        raise ValueError("sink needs blocks * passes * 8 KB")
    _check(load_library().bitlogic_probe_gather(
        rows.data_ptr(), nbytes // 128, int(lanes_per_row), int(valu_per_pass), int(blocks),
        int(passes), int(waves_per_simd), int(seed) & 0xFFFFFFFF, _dev(out, "out", _I32),
        sink.data_ptr() if sink is not None else None, _stream(stream, out.device)))
    return int(blocks) * int(passes) * 64 * 6
