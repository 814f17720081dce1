"""fp64 CPU oracle for Fibonacci-offset sparse attention (Python side).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and the CPU-baseline
leg of bench.py import this package.  It shares no code with the HIP library.

The numerical work is in fibattn_oracle.c (plain C, float64, one query at a time);
this module marshals numpy arrays to it and holds the oracle's own copy of the
per-layer alpha schedules (Section 2, "The per-layer scalar").
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int)
_fp = ctypes.POINTER(ctypes.c_float)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from oracle.build import build
        build()
    lib = ctypes.CDLL(LIB_PATH)
    i, f, d = ctypes.c_int, ctypes.c_float, ctypes.c_double
    lib.oracle_rungs.argtypes = [f, _ip, i, i, _ip, _fp, _ip, _fp]
    lib.oracle_rungs.restype = i
    lib.oracle_forward.argtypes = [i, i, i, i, i, i, _ip, i, f, _dp, _dp, _dp, _dp, _dp]
    lib.oracle_forward.restype = i
    lib.oracle_backward.argtypes = [i, i, i, i, i, i, _ip, i, f, _dp, _dp, _dp, _dp, _dp, _dp, _dp, _dp, _dp]
    lib.oracle_backward.restype = i
    lib.oracle_forward_table.argtypes = [i, i, i, i, i, i, i, _ip, _dp, _ip, _dp, _dp, _dp, _dp, _dp]
    lib.oracle_forward_table.restype = None
    lib.oracle_backward_table.argtypes = [i, i, i, i, i, i, i, _ip, _dp, _ip, _dp, _dp, _dp, _dp, _dp, _dp, _dp, _dp, _dp]
    lib.oracle_backward_table.restype = None
    lib.oracle_rope.argtypes = [i, i, i, i, d, i, _dp, _dp]
    lib.oracle_rope.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = i
    _lib = lib
    return lib


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # torch tensor
        x = x.detach().cpu().double().numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a: np.ndarray, t=_dp):
    return a.ctypes.data_as(t)


def _base(base) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(base, dtype=np.int32).reshape(-1))


def _heads(q, k):
    """(B, H, Hkv, T, D) of q [B, H, T, D] and k [B, Hkv, T, D], H a multiple of Hkv."""
    B, H, T, D = q.shape
    if k.ndim != 4 or k.shape[0] != B or k.shape[2:] != (T, D) or k.shape[1] < 1 or H % k.shape[1]:
        raise ValueError(f"k shape {k.shape} does not group q shape {q.shape}")
    return B, H, k.shape[1], T, D


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def rungs(alpha: float, base, W: int):
    """Rung table after inclusion and dedupe: list of (d0, w, f, d) with w, d float32."""
    lib = _load()
    b = _base(base)
    K = b.size
    d0 = np.zeros(64, np.int32); f = np.zeros(64, np.int32)
    w = np.zeros(64, np.float32); d = np.zeros(64, np.float32)
    n = lib.oracle_rungs(ctypes.c_float(np.float32(alpha)), _ptr(b, _ip), K, W,
                         _ptr(d0, _ip), _ptr(w, _fp), _ptr(f, _ip), _ptr(d, _fp))
    if n < 0:
        raise ValueError("bad rung-table input")
    return [(int(d0[a]), np.float32(w[a]), int(f[a]), np.float32(d[a])) for a in range(n)]


def forward(q, k, v, W: int, base, alpha: float):
    """o [B,H,T,D] and lse [B,H,T] in float64 (Section 2); k, v may have fewer heads
    (grouped heads: [B,Hkv,T,D])."""
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, Hkv, T, D = _heads(q, k)
    b = _base(base)
    o = np.empty_like(q)
    lse = np.empty((B, H, T), np.float64)
    rc = lib.oracle_forward(B, H, Hkv, T, D, W, _ptr(b, _ip), b.size, ctypes.c_float(np.float32(alpha)),
                            _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError("bad oracle input")
    return o, lse


def backward(q, k, v, dO, W: int, base, alpha: float):
    """dq [B,H,T,D], dk, dv (shaped like k, v), dalpha and the L1 mass of its terms,
    in float64."""
    lib = _load()
    q, k, v, dO = _f64(q), _f64(k), _f64(v), _f64(dO)
    B, H, Hkv, T, D = _heads(q, k)
    b = _base(base)
    dq = np.empty_like(q); dk = np.empty_like(k); dv = np.empty_like(k)
    da = ctypes.c_double(0.0); l1 = ctypes.c_double(0.0)
    rc = lib.oracle_backward(B, H, Hkv, T, D, W, _ptr(b, _ip), b.size, ctypes.c_float(np.float32(alpha)),
                             _ptr(q), _ptr(k), _ptr(v), _ptr(dO), _ptr(dq), _ptr(dk), _ptr(dv),
                             ctypes.byref(da), ctypes.byref(l1))
    if rc != 0:
        raise ValueError("bad oracle input")
    return dq, dk, dv, da.value, l1.value


def forward_table(q, k, v, W: int, d0, w, f):
    """Forward on an explicit rung table (w in float64); used for finite differences in alpha."""
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, Hkv, T, D = _heads(q, k)
    d0 = _base(d0); f = _base(f); w = np.ascontiguousarray(w, np.float64)
    o = np.empty_like(q)
    lse = np.empty((B, H, T), np.float64)
    lib.oracle_forward_table(B, H, Hkv, T, D, W, d0.size, _ptr(d0, _ip), _ptr(w), _ptr(f, _ip),
                             _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse))
    return o, lse


def backward_table(q, k, v, dO, W: int, d0, w, f):
    lib = _load()
    q, k, v, dO = _f64(q), _f64(k), _f64(v), _f64(dO)
    B, H, Hkv, T, D = _heads(q, k)
    d0 = _base(d0); f = _base(f); w = np.ascontiguousarray(w, np.float64)
    dq = np.empty_like(q); dk = np.empty_like(k); dv = np.empty_like(k)
    da = ctypes.c_double(0.0); l1 = ctypes.c_double(0.0)
    lib.oracle_backward_table(B, H, Hkv, T, D, W, d0.size, _ptr(d0, _ip), _ptr(w), _ptr(f, _ip),
                              _ptr(q), _ptr(k), _ptr(v), _ptr(dO), _ptr(dq), _ptr(dk), _ptr(dv),
                              ctypes.byref(da), ctypes.byref(l1))
    return dq, dk, dv, da.value, l1.value


def rope(x, rope_base: float = 10000.0, transpose: bool = False):
    """RoPE at true positions (rotate-half, float64 angles); transpose applies R^T."""
    lib = _load()
    x = _f64(x)
    B, H, T, D = x.shape
    y = np.empty_like(x)
    lib.oracle_rope(B, H, T, D, float(rope_base), int(bool(transpose)), _ptr(x), _ptr(y))
    return y


# --- the oracle's own copy of the alpha schedules (Section 2) ---------------------

def alpha_from_theta(theta) -> np.ndarray:
    """alpha = 0.5 + sigmoid(theta) in float64, rounded once to float32."""
    t = np.asarray(theta, dtype=np.float64)
    return (0.5 + 1.0 / (1.0 + np.exp(-t))).astype(np.float32)


def alpha_schedule(kind: str, L: int = 16, theta=None) -> np.ndarray:
    """'fixed', 'linear' (0.5 + l/(L-1)), 'coprime' (linear values at 7*l mod L) or 'learned'."""
    if kind == "fixed":
        return np.ones(L, np.float32)
    if kind == "linear":
        return np.array([0.5 + l / (L - 1) for l in range(L)], np.float64).astype(np.float32)
    if kind == "coprime":
        return np.array([0.5 + ((7 * l) % L) / (L - 1) for l in range(L)], np.float64).astype(np.float32)
    if kind == "learned":
        return alpha_from_theta(theta)
    raise ValueError(kind)
