"""Metadata-only policy passes and state reconstruction (oracle; test infrastructure only).

Eviction depends only on row metadata (segment class, unit id) and the
resident count, never on K/V values (Sec. 3.3 counts positions), so a whole
stream's eviction history can be replayed without attention.  The resident
state after any step is then fully determined, which lets a test resume a
long stream at unit k by regenerating only the surviving rows' values.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from synth.streams import StreamSpec, WorkloadConfig, step_values

from .cache import OracleCache
from .policy import plan_eviction


@dataclass
class StepTrace:
    n_pre: int
    n_post: int
    units: List[int]
    budget_unmet: bool
    moved: int                 # survivors at or after the first evicted slot


@dataclass
class StreamTrace:
    steps: List[StepTrace] = field(default_factory=list)
    peak: int = 0
    # layout after the last replayed step, and where each row came from
    pos: Optional[np.ndarray] = None
    seg: Optional[np.ndarray] = None
    unit: Optional[np.ndarray] = None
    src_step: Optional[np.ndarray] = None
    src_row: Optional[np.ndarray] = None


def replay_metadata(spec: StreamSpec, budget: int, window: int,
                    n_steps: Optional[int] = None, evict: bool = True) -> StreamTrace:
    """Run the eviction policy over the first ``n_steps`` steps of a stream."""
    n_steps = len(spec.steps) if n_steps is None else n_steps
    if not evict:
        return _replay_no_eviction(spec, n_steps)
    pos = np.zeros(0, np.int64)
    seg = np.zeros(0, np.uint8)
    unit = np.zeros(0, np.int64)
    src_step = np.zeros(0, np.int64)
    src_row = np.zeros(0, np.int64)
    cur = -1
    tr = StreamTrace()
    for i in range(n_steps):
        st = spec.steps[i]
        n = st.n
        pos = np.concatenate([pos, st.pos.astype(np.int64)])
        seg = np.concatenate([seg, st.seg])
        unit = np.concatenate([unit, np.full(n, st.unit, np.int64)])
        src_step = np.concatenate([src_step, np.full(n, i, np.int64)])
        src_row = np.concatenate([src_row, np.arange(n, dtype=np.int64)])
        cur = max(cur, st.unit)
        tr.peak = max(tr.peak, pos.shape[0])
        if not evict or not st.evict:
            # Sec. 3.3 checks the budget after each duplex unit: a step that does
            # not end its unit (a side-channel chunk or token) is not checked
            tr.steps.append(StepTrace(pos.shape[0], pos.shape[0], [], False, 0))
            continue
        plan = plan_eviction(seg, unit, budget, window, cur)
        keep = ~plan.evict_mask
        if plan.evict_mask.any():
            first = int(np.argmax(plan.evict_mask))
            moved = int(keep[first:].sum())
        else:
            moved = 0
        tr.steps.append(StepTrace(plan.n_pre, plan.n_post, plan.units, plan.budget_unmet, moved))
        pos, seg, unit = pos[keep], seg[keep], unit[keep]
        src_step, src_row = src_step[keep], src_row[keep]
    tr.pos, tr.seg, tr.unit, tr.src_step, tr.src_row = pos, seg, unit, src_step, src_row
    return tr


def _replay_no_eviction(spec: StreamSpec, n_steps: int) -> StreamTrace:
    """Without eviction every appended row stays: the layout is the concatenation."""
    tr = StreamTrace()
    steps = spec.steps[:n_steps]
    total = 0
    for st in steps:
        total += st.n
        tr.steps.append(StepTrace(total, total, [], False, 0))
    tr.peak = total
    if steps:
        tr.pos = np.concatenate([st.pos.astype(np.int64) for st in steps])
        tr.seg = np.concatenate([st.seg for st in steps])
        tr.unit = np.concatenate([np.full(st.n, st.unit, np.int64) for st in steps])
        tr.src_step = np.concatenate([np.full(st.n, i, np.int64) for i, st in enumerate(steps)])
        tr.src_row = np.concatenate([np.arange(st.n, dtype=np.int64) for st in steps])
    else:
        tr.pos = np.zeros(0, np.int64)
        tr.seg = np.zeros(0, np.uint8)
        tr.unit = tr.src_step = tr.src_row = np.zeros(0, np.int64)
    return tr


def resume(cfg: WorkloadConfig, seed: int, spec: StreamSpec, budget: int, window: int,
           n_steps: int, layers: Sequence[int], evict: bool = True,
           values: Optional[Callable[[int], Dict[str, np.ndarray]]] = None) -> OracleCache:
    """Oracle cache holding the state of ``spec`` after its first ``n_steps`` steps.

    The surviving rows are re-appended in cache order with their original
    positions (so their keys get the rotation of those positions), with
    values regenerated from the seeded generator for ``layers``.  With
    ``evict`` false the stream is replayed without eviction (a control run).
    ``values(step_index)`` may supply a step's generated values (arrays ``k``,
    ``v`` of shape ``[len(layers)][n][Hkv][D]``) instead of regenerating them.
    """
    tr = replay_metadata(spec, budget, window, n_steps, evict=evict)
    cache = OracleCache(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, layers,
                        theta=cfg.rope_theta, scale=cfg.scale)
    # regenerate each surviving row's values from its source step
    k = {l: np.zeros((tr.pos.shape[0], cfg.n_kv_heads, cfg.head_dim)) for l in layers}
    v = {l: np.zeros((tr.pos.shape[0], cfg.n_kv_heads, cfg.head_dim)) for l in layers}
    steps = tr.src_step
    starts = np.flatnonzero(np.r_[True, steps[1:] != steps[:-1]])
    ends = np.r_[starts[1:], steps.shape[0]]
    for a, b in zip(starts, ends):
        st = spec.steps[int(steps[a])]
        vals = values(int(steps[a])) if values is not None else \
            step_values(cfg, seed, spec.stream, st.key, st.n, layers)
        rows = tr.src_row[a:b]
        for i, l in enumerate(layers):
            k[l][a:b] = vals["k"][i][rows]
            v[l][a:b] = vals["v"][i][rows]
    cache.load_rows(tr.seg, tr.pos, tr.unit, k, v, step_rows=0)
    cache.peak = tr.peak
    # the newest unit and position may belong to rows that were just evicted
    if n_steps:
        cache.cur = max(st.unit for st in spec.steps[:n_steps])
        cache.last_pos = int(spec.steps[n_steps - 1].pos[-1])
    cache.step_rows = 0
    return cache

