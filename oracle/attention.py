"""Causal grouped-query softmax attention, float64 (oracle; test infrastructure only).

The unit's new rows attend over the resident KV cache (Sec. 3.1: each unit is
processed by the language model; Sec. 3.3: the resident cache after eviction).
For query row i and query head h, with KV head g = floor(h / (Hq / Hkv))
(contiguous head groups; the paper does not state the grouping):

    s_j = scale * <q_i,h , k_j,g>        over resident keys j with pos_j <= pos_i
    o_i,h = sum_j exp(s_j - max s) v_j,g / sum_j exp(s_j - max s)

q and k are already rotated to their own positions.  This is the textbook
definition; the only library step is the matrix product.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def attend(q_rot: np.ndarray, k_rot: np.ndarray, v: np.ndarray,
           q_pos: np.ndarray, k_pos: np.ndarray, scale: float,
           visible: Optional[np.ndarray] = None) -> np.ndarray:
    """q_rot ``[n][Hq][D]``, k_rot and v ``[R][Hkv][D]``, positions ``[n]`` and ``[R]``.

    ``visible`` (bool ``[R]``) additionally hides keys (used to express
    "full history with evicted rows masked").  Returns o ``[n][Hq][D]`` float64.
    A query with no visible key gets a zero output (never happens for a query
    that is itself resident, since it sees its own key).
    """
    q_rot = np.asarray(q_rot, np.float64)
    k_rot = np.asarray(k_rot, np.float64)
    v = np.asarray(v, np.float64)
    n, Hq, D = q_rot.shape
    Hkv = k_rot.shape[1]
    group = Hq // Hkv
    mask = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]      # [n][R]
    if visible is not None:
        mask = mask & np.asarray(visible, bool)[None, :]
    out = np.zeros((n, Hq, D), np.float64)
    for h in range(Hq):
        g = h // group
        s = scale * (q_rot[:, h, :] @ k_rot[:, g, :].T)                   # [n][R]
        s = np.where(mask, s, -np.inf)
        m = np.max(s, axis=1, keepdims=True)
        m = np.where(np.isfinite(m), m, 0.0)
        e = np.where(mask, np.exp(s - m), 0.0)
        denom = e.sum(axis=1, keepdims=True)
        num = e @ v[:, g, :]
        out[:, h, :] = np.divide(num, denom, out=np.zeros_like(num), where=denom > 0)
    return out
