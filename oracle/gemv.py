"""Exactly rounded fp64 reference of the decode-step product y = W x.

TEST INFRASTRUCTURE ONLY (see the package header).

Each product of a bf16 or float16 weight (8 or 11 significant bits) and a
float32, bf16 or float16 activation (at most 24 significant bits) is exact in
float64; ``math.fsum``
then returns the correctly rounded sum, so y_ref is the exact dot product
rounded once. ``den`` is the same sum of |w x|, the scale of the relative
error metric |y - y_ref| / (den + 1e-30).
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np


def bf16_to_f64(w_bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact: bf16 is the top half of a float32)."""
    u = np.asarray(w_bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def fp16_to_f64(w_bits: np.ndarray) -> np.ndarray:
    """float16 bit patterns -> float64 (exact)."""
    return np.asarray(w_bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def x_to_f64(x: np.ndarray) -> np.ndarray:
    """Activations as float64: float32 or float16 values, or uint16 arrays
    holding bf16 bits."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_to_f64(x)
    return x.astype(np.float64)


def gemv_rows(w_bits: np.ndarray, x: np.ndarray, rows=None, weights: str = "bf16") -> Tuple[np.ndarray, np.ndarray]:
    """y_ref[b, r] and den[b, r] for the selected rows (all rows if None).

    w_bits: uint16 [R, K] bf16 (weights="bf16") or float16 ("fp16") bits;
    x: [B, K] float32, float16, or bf16 bits."""
    to_f64 = fp16_to_f64 if weights == "fp16" else bf16_to_f64
    W = np.asarray(w_bits)
    X = x_to_f64(x)
    if X.ndim == 1:
        X = X[None, :]
    rows = range(W.shape[0]) if rows is None else list(rows)
    B = X.shape[0]
    y = np.zeros((B, len(rows)), dtype=np.float64)
    den = np.zeros((B, len(rows)), dtype=np.float64)
    for i, r in enumerate(rows):
        wr = to_f64(W[r])
        for b in range(B):
            p = wr * X[b]                       # exact products
            y[b, i] = math.fsum(p.tolist())
            den[b, i] = math.fsum(np.abs(p).tolist())
    return y, den


def rel_err(y: np.ndarray, y_ref: np.ndarray, den: np.ndarray) -> np.ndarray:
    """Per-output error |y - y_ref| / (sum |w x| + 1e-30)."""
    return np.abs(np.asarray(y, np.float64) - y_ref) / (den + 1e-30)
