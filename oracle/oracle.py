"""ctypes front end of the CPU oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
module.  Inputs are widened to float64 exactly (bf16 bit patterns and float32
are both exact in float64) and handed to the C oracle in ``gdn_oracle.c``.

Any object with the attributes of a workload (B, T, Hk, Hv, dk, dv, parent,
q, k, v, alpha, beta, S0, conv_w, conv_state, accepted) can be passed.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

_lib = None


class _Dims(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("T", ctypes.c_int), ("Hk", ctypes.c_int),
                ("Hv", ctypes.c_int), ("dk", ctypes.c_int), ("dv", ctypes.c_int),
                ("scale", ctypes.c_double)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b  # noqa: WPS433
            _b.build()
        _lib = ctypes.CDLL(LIB_PATH)
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def widen(a: np.ndarray) -> np.ndarray:
    """float64 copy of an input: bf16 bit patterns (uint16) or floats."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return np.ascontiguousarray((a.astype(np.uint32) << np.uint32(16)).view(np.float32),
                                    dtype=np.float64)
    return np.ascontiguousarray(a, dtype=np.float64)


def _dims(w, scale: float = 0.0) -> _Dims:
    return _Dims(w.B, w.T, w.Hk, w.Hv, w.dk, w.dv, float(scale))


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (timing only)."""
    lib().oracle_set_num_threads(ctypes.c_int(int(n)))


def tree_status(parent_row: np.ndarray) -> int:
    p = np.ascontiguousarray(parent_row, dtype=np.int32)
    return int(lib().oracle_tree_status(ctypes.c_int(p.shape[0]), _p(p)))


def prepare(parent: np.ndarray) -> dict:
    """Tree metadata for parent [B][T] (see oracle_prepare)."""
    parent = np.ascontiguousarray(parent, dtype=np.int32)
    B, T = parent.shape
    W = (T + 63) // 64
    depth = np.zeros((B, T), np.int32)
    order = np.zeros((B, T), np.int32)
    anc = np.zeros((B, T, W), np.uint64)
    nvalid = np.zeros(B, np.int32)
    status = np.zeros(B, np.int32)
    lib().oracle_prepare(ctypes.c_int(B), ctypes.c_int(T), _p(parent), _p(depth), _p(order),
                         _p(anc), _p(nvalid), _p(status))
    return dict(depth=depth, order=order, anc=anc, nvalid=nvalid, status=status)


def _inputs(w):
    return (np.ascontiguousarray(w.parent, dtype=np.int32), widen(w.q), widen(w.k), widen(w.v),
            widen(w.alpha), widen(w.beta), widen(w.conv_w), widen(w.conv_state), widen(w.S0))


def features(w) -> np.ndarray:
    """Post-conv, post-SiLU, q/k-normalised features [B][T][C] (float64)."""
    parent, q, k, v, _a, _b, cw, cs, _s = _inputs(w)
    C = 2 * w.Hk * w.dk + w.Hv * w.dv
    feat = np.zeros((w.B, w.T, C), np.float64)
    d = _dims(w)
    lib().oracle_features(ctypes.byref(d), _p(parent), _p(q), _p(k), _p(v), _p(cw), _p(cs),
                          _p(feat))
    return feat


def verify(w, node_mask: np.ndarray | None = None, scale: float = 0.0) -> np.ndarray:
    """Per-node outputs [B][T][Hv][dv] (float64); see oracle_verify."""
    parent, q, k, v, a, b, cw, cs, s0 = _inputs(w)
    out = np.zeros((w.B, w.T, w.Hv, w.dv), np.float64)
    d = _dims(w, scale)
    mask = None
    if node_mask is not None:
        mask = np.ascontiguousarray(node_mask, dtype=np.uint8)
        assert mask.shape == (w.B, w.T)
    lib().oracle_verify(ctypes.byref(d), _p(parent), _p(q), _p(k), _p(v), _p(a), _p(b), _p(cw),
                        _p(cs), _p(s0), _p(mask) if mask is not None else None, _p(out))
    return out


def commit(w, accepted: np.ndarray | None = None, S: np.ndarray | None = None,
           conv_state: np.ndarray | None = None):
    """Committed (S, conv_state, status) in float64; see oracle_commit.

    S and conv_state default to the workload's S0 / conv_state."""
    parent, q, k, v, a, b, cw, cs, s0 = _inputs(w)
    acc = np.ascontiguousarray(w.accepted if accepted is None else accepted, dtype=np.int32)
    Sx = s0.copy() if S is None else widen(S).copy()
    csx = cs.copy() if conv_state is None else widen(conv_state).copy()
    status = np.zeros(w.B, np.int32)
    d = _dims(w)
    lib().oracle_commit(ctypes.byref(d), _p(parent), _p(acc), _p(q), _p(k), _p(v), _p(a), _p(b),
                        _p(cw), _p(csx), _p(Sx), _p(status))
    return Sx, csx, status
