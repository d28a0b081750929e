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
from .policy import EvictRule, compaction_indices, plan_by_rule


@dataclass
class StepTrace:
    n_pre: int
    n_post: int
    units: List[int]
    budget_unmet: bool
    moved: int                 # survivors at or after the first evicted slot: the rows an
                               # in-place order-preserving compaction would shift
    settled: int = 0           # survivors that join the retained prefix at this step (below)
    evict_mask: Optional[np.ndarray] = None   # bool [n_pre] (with record_masks)
    new_slot: Optional[np.ndarray] = None     # int32 [n_pre] (with record_masks)


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


class MetadataReplay:
    """The eviction policy over a stream's steps, one step at a time.

    Besides the plan of each step it reports ``settled``: once a step has
    evicted units up to u, every resident row of a unit <= u is non-evictable
    for good (whole units go oldest first), so those rows form a retained
    prefix of the cache that no later eviction touches; ``settled`` counts the
    surviving rows of units <= u that were not already in that prefix (rows
    retained from the units just evicted, and rows appended since the
    previous eviction under a unit id it had already reached).  A cache that
    keeps that prefix in a region of its own copies exactly these rows into
    it when it compacts.  Under the row and sink+recent variants of the rule
    (which can stop inside a unit) the prefix ends at the newest evicted row
    instead: ``settled`` then counts the survivors older than that row that
    were not already in it.
    """

    def __init__(self, spec: StreamSpec, budget: int, window: int, record_masks: bool = False,
                 rule: Optional[EvictRule] = None):
        self.spec, self.budget, self.window = spec, budget, window
        self.rule = rule or EvictRule()
        self.record_masks = record_masks
        self.i = 0
        self.pos = np.zeros(0, np.int64)
        self.seg = np.zeros(0, np.uint8)
        self.unit = np.zeros(0, np.int64)
        self.src_step = np.zeros(0, np.int64)
        self.src_row = np.zeros(0, np.int64)
        self.in_prefix = np.zeros(0, bool)
        self.cur = -1
        self.peak = 0

    def step(self) -> StepTrace:
        st = self.spec.steps[self.i]
        n = st.n
        self.pos = np.concatenate([self.pos, st.pos.astype(np.int64)])
        self.seg = np.concatenate([self.seg, st.seg])
        self.unit = np.concatenate([self.unit, np.full(n, st.unit, np.int64)])
        self.src_step = np.concatenate([self.src_step, np.full(n, self.i, np.int64)])
        self.src_row = np.concatenate([self.src_row, np.arange(n, dtype=np.int64)])
        self.in_prefix = np.concatenate([self.in_prefix, np.zeros(n, bool)])
        self.i += 1
        self.cur = max(self.cur, st.unit)
        self.peak = max(self.peak, self.pos.shape[0])
        R = self.pos.shape[0]
        if not st.evict:
            # Sec. 3.3 checks the budget after each duplex unit: a step that does
            # not end its unit (a side-channel chunk or token) is not checked
            tr = StepTrace(R, R, [], False, 0)
            if self.record_masks:
                tr.evict_mask = np.zeros(R, bool)
                tr.new_slot = np.arange(R, dtype=np.int32)
            return tr
        plan = plan_by_rule(self.rule, self.seg, self.unit, self.budget, self.window, self.cur)
        keep = ~plan.evict_mask
        moved = int(keep[int(np.argmax(plan.evict_mask)):].sum()) if plan.evict_mask.any() else 0
        settled = 0
        if plan.units:
            if self.rule.kind == "unit":
                older = self.unit <= max(plan.units)
            else:
                # the other rules can stop inside a unit: the retained prefix ends
                # at the newest evicted row
                older = np.arange(keep.shape[0]) < int(np.flatnonzero(plan.evict_mask)[-1])
            joins = keep & older & ~self.in_prefix
            settled = int(joins.sum())
            self.in_prefix |= joins
        tr = StepTrace(plan.n_pre, plan.n_post, plan.units, plan.budget_unmet, moved, settled)
        if self.record_masks:
            tr.evict_mask = plan.evict_mask
            tr.new_slot = compaction_indices(plan.evict_mask)
        self.pos, self.seg, self.unit = self.pos[keep], self.seg[keep], self.unit[keep]
        self.src_step, self.src_row = self.src_step[keep], self.src_row[keep]
        self.in_prefix = self.in_prefix[keep]
        return tr


def replay_metadata(spec: StreamSpec, budget: int, window: int,
                    n_steps: Optional[int] = None, evict: bool = True,
                    record_masks: bool = False, rule: Optional[EvictRule] = None) -> StreamTrace:
    """Run the eviction policy (``rule``: Sec. 3.3's by default) over the first
    ``n_steps`` steps of a stream.  With ``record_masks`` every step also
    carries its eviction mask and compaction indices (memory grows with steps
    x resident rows)."""
    n_steps = len(spec.steps) if n_steps is None else n_steps
    if not evict:
        return _replay_no_eviction(spec, n_steps)
    rp = MetadataReplay(spec, budget, window, record_masks=record_masks, rule=rule)
    tr = StreamTrace()
    for _ in range(n_steps):
        tr.steps.append(rp.step())
    tr.peak = rp.peak
    tr.pos, tr.seg, tr.unit, tr.src_step, tr.src_row = rp.pos, rp.seg, rp.unit, rp.src_step, rp.src_row
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
           values: Optional[Callable[[int], Dict[str, np.ndarray]]] = None,
           rule: Optional[EvictRule] = None) -> OracleCache:
    """Oracle cache holding the state of ``spec`` after its first ``n_steps`` steps.

    The surviving rows are re-appended in cache order with their original
    positions (so their keys get the rotation of those positions), with
    values regenerated from the seeded generator for ``layers``.  With
    ``evict`` false the stream is replayed without eviction (a control run).
    ``values(step_index)`` may supply a step's generated values (arrays ``k``,
    ``v`` of shape ``[len(layers)][n][Hkv][D]``) instead of regenerating them.
    """
    tr = replay_metadata(spec, budget, window, n_steps, evict=evict, rule=rule)
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

