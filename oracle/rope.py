"""Rotary position encoding, float64 (oracle; test infrastructure only).

Sec. 3.3: position ids advance with every token fed to the model, whatever
is evicted, so every cached key keeps the rotation of its original position
and is never re-encoded.  The paper does not name the rotary variant; this
oracle uses the rotate-half form with per-pair frequency theta**(-2i/D):

    x'[i]       = x[i] cos(a_i) - x[i+D/2] sin(a_i)
    x'[i+D/2]   = x[i+D/2] cos(a_i) + x[i] sin(a_i),   a_i = pos * theta**(-2i/D)

for i < D/2.  Parity of the variant itself is unpinned (a reading).
"""
from __future__ import annotations

import numpy as np


def inverse_frequencies(head_dim: int, theta: float) -> np.ndarray:
    """theta ** (-2 i / D) for i = 0 .. D/2 - 1, float64."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * i / head_dim)


def rotate(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate ``x[..., D]`` by the angles of ``pos`` (shape ``x.shape[:-2]`` or
    ``x.shape[:-1]``; a trailing head axis is broadcast).  Returns float64."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    p = np.asarray(pos, dtype=np.float64)
    while p.ndim < x.ndim - 1:
        p = p[..., None]
    ang = p[..., None] * inverse_frequencies(D, theta)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)
