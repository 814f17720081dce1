"""Offset base tables and per-layer alpha schedules (host side).

Section 2: every rung distance is d_k = alpha * f_k, with alpha = 0.5 + sigmoid(theta)
in [0.5, 1.5] and one alpha per layer.  The paper studies four ways of setting it
over L = 16 layers (fixed, learned, linear stagger, coprime stagger) and two bases
(Fibonacci, K = 15, and a reach-matched power-of-2 control).

Each alpha is computed in float64 and rounded once to float32; the float32 value is
what the kernels and the oracle receive.
"""
from __future__ import annotations

import numpy as np

# Section 2, "Attended set": the Fibonacci base, K = 15 (f_15 = 987, about the
# training length 1024).
FIB15 = (1, 2, 3, 5, 8, 13, 21, 34, 55, 89, 144, 233, 377, 610, 987)
# Section 2, "Control base": a power-of-2 base with the same reach; at T = 1024 the
# workloads take 1, 2, 4, ..., 1024 (K = 11).
POW2_11 = tuple(1 << j for j in range(11))


def alpha_from_theta(theta) -> np.ndarray:
    """alpha = 0.5 + sigmoid(theta), evaluated in float64, rounded to float32."""
    t = np.asarray(theta, dtype=np.float64)
    return (0.5 + 1.0 / (1.0 + np.exp(-t))).astype(np.float32)


def alpha_fixed(L: int = 16) -> np.ndarray:
    """'Fixed' schedule: alpha = 1 in every layer (integer offsets)."""
    return np.ones(L, dtype=np.float32)


def alpha_linear_stagger(L: int = 16) -> np.ndarray:
    """'Staggered (linear)': alpha_l = 0.5 + l/(L-1), a ramp from 0.5 to 1.5."""
    l = np.arange(L, dtype=np.float64)
    return (0.5 + l / (L - 1)).astype(np.float32)


def alpha_coprime_stagger(L: int = 16, S: int = 7) -> np.ndarray:
    """'Staggered (coprime / HDC)': the linear-stagger values reassigned by l -> S*l mod L.

    For L = 16, S = 7 the map is its own inverse (7*7 = 49 = 1 mod 16), so reading
    the reassignment as either direction gives the same table."""
    lin = np.arange(L, dtype=np.float64)
    src = (S * np.arange(L)) % L
    return (0.5 + lin[src] / (L - 1)).astype(np.float32)


def integer_base(alpha, base) -> tuple:
    """Static offsets rounded to integers, as a base table for alpha = 1.

    Section 2 runs the static schedules on integer offsets (a boolean mask) without
    giving the rounding rule.  The reading taken here: d_k = fl32(alpha * f_k) (the
    float32 product every rung table uses), rounded half to even, dropping 0 and
    repeats.  Passing the result with alpha = 1 selects the integer-offset kernels,
    which never read a second row."""
    a = np.float32(alpha)
    d = np.rint(np.asarray(base, dtype=np.float32) * a).astype(np.int64)
    return tuple(int(x) for x in np.unique(d[d > 0]))
