"""One stream's resident KV cache, float64 (oracle; test infrastructure only).

Per step of a stream (a listening unit or one decode token) the paper's
method does, in this order:

1. append the step's rows, each key rotated at its own position id
   (Sec. 3.3: positions advance with every fed token and kept keys are never
   re-encoded);
2. run attention for the step's new rows over the resident cache
   (Sec. 3.1: the unit is processed by the language model);
3. after the unit, evict under the budget and compact (Sec. 3.3).

Rows are stored in cache order (the order they were appended); compaction
keeps survivors in that order.  The cache can also keep the full history of
every row ever appended, to express "full-history attention with the
evicted rows masked".
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Iterable, Optional, Sequence

import numpy as np

from synth.streams import SEG_PREFIX, SEG_RESPONSE

from . import rope
from .attention import attend
from .policy import EvictionPlan, EvictRule, compaction_indices, plan_by_rule


class OracleError(ValueError):
    pass


@dataclass
class EvictRecord:
    plan: EvictionPlan
    new_slot: np.ndarray      # int32 [n_pre]
    pos: np.ndarray           # layout after compaction
    seg: np.ndarray
    unit: np.ndarray

    @property
    def n_evicted(self) -> int:
        return self.plan.n_pre - self.plan.n_post


class OracleCache:
    def __init__(self, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 layers: Iterable[int] = (0,), theta: float = 1.0e6,
                 scale: Optional[float] = None, keep_history: bool = False):
        self.Hq, self.Hkv, self.D = n_q_heads, n_kv_heads, head_dim
        self.layers = list(layers)
        self.theta = theta
        self.scale = 1.0 / np.sqrt(head_dim) if scale is None else scale
        self.pos = np.zeros(0, np.int64)
        self.seg = np.zeros(0, np.uint8)
        self.unit = np.zeros(0, np.int64)
        self.k: Dict[int, np.ndarray] = {l: np.zeros((0, n_kv_heads, head_dim)) for l in self.layers}
        self.v: Dict[int, np.ndarray] = {l: np.zeros((0, n_kv_heads, head_dim)) for l in self.layers}
        self.cur: Optional[int] = None
        self.last_pos: Optional[int] = None
        self.peak = 0
        self.step_rows = 0
        self.keep_history = keep_history
        if keep_history:
            self.h_pos = np.zeros(0, np.int64)
            self.h_resident = np.zeros(0, bool)
            self.h_k = {l: np.zeros((0, n_kv_heads, head_dim)) for l in self.layers}
            self.h_v = {l: np.zeros((0, n_kv_heads, head_dim)) for l in self.layers}

    @property
    def resident(self) -> int:
        return int(self.pos.shape[0])

    # -- 1. append -------------------------------------------------------------
    def append(self, seg: Sequence[int], pos: Sequence[int], unit: int,
               k: Optional[Dict[int, np.ndarray]] = None,
               v: Optional[Dict[int, np.ndarray]] = None) -> None:
        """Append one step's rows.  ``k``/``v`` map layer -> ``[n][Hkv][D]`` pre-rotation."""
        seg = np.asarray(seg, np.uint8)
        pos = np.asarray(pos, np.int64)
        n = int(seg.shape[0])
        if n == 0 or pos.shape[0] != n:
            raise OracleError("a step appends at least one row, with one position per row")
        if np.any(seg > SEG_RESPONSE):
            raise OracleError("unknown segment class")
        if np.any(np.diff(pos) <= 0) or (self.last_pos is not None and pos[0] <= self.last_pos):
            raise OracleError("positions must strictly increase")
        if self.cur is not None and unit < self.cur:
            raise OracleError("unit ids must not decrease")
        if unit >= 0 and np.any(seg == SEG_PREFIX):
            raise OracleError("prefix rows belong to unit -1")
        self.pos = np.concatenate([self.pos, pos])
        self.seg = np.concatenate([self.seg, seg])
        self.unit = np.concatenate([self.unit, np.full(n, unit, np.int64)])
        for l in self.layers:
            kr = rope.rotate(np.asarray(k[l], np.float64), pos, self.theta)
            vv = np.asarray(v[l], np.float64)
            self.k[l] = np.concatenate([self.k[l], kr])
            self.v[l] = np.concatenate([self.v[l], vv])
            if self.keep_history:
                self.h_k[l] = np.concatenate([self.h_k[l], kr])
                self.h_v[l] = np.concatenate([self.h_v[l], vv])
        if self.keep_history:
            self.h_pos = np.concatenate([self.h_pos, pos])
            self.h_resident = np.concatenate([self.h_resident, np.ones(n, bool)])
        self.cur = unit if self.cur is None else max(self.cur, unit)
        self.last_pos = int(pos[-1])
        self.peak = max(self.peak, self.resident)
        self.step_rows = n

    def load_rows(self, seg: Sequence[int], pos: Sequence[int], unit: Sequence[int],
                  k: Dict[int, np.ndarray], v: Dict[int, np.ndarray], step_rows: int) -> None:
        """Set the resident state in one go: rows in cache order with their own
        unit ids, keys rotated by their original positions (Sec. 3.3), exactly
        what appending them step by step would store.  ``step_rows`` is the
        row count of the newest step (the rows queries may come from)."""
        seg = np.asarray(seg, np.uint8)
        pos = np.asarray(pos, np.int64)
        unit = np.asarray(unit, np.int64)
        if self.resident:
            raise OracleError("load_rows fills an empty cache")
        if np.any(np.diff(pos) <= 0):
            raise OracleError("positions must strictly increase")
        if np.any(seg > SEG_RESPONSE) or np.any(np.diff(unit) < 0):
            raise OracleError("unknown segment class or decreasing unit ids")
        self.pos, self.seg, self.unit = pos.copy(), seg.copy(), unit.copy()
        for l in self.layers:
            self.k[l] = rope.rotate(np.asarray(k[l], np.float64), pos, self.theta)
            self.v[l] = np.asarray(v[l], np.float64).copy()
        if pos.shape[0]:
            self.cur = int(unit.max())
            self.last_pos = int(pos[-1])
        self.peak = max(self.peak, self.resident)
        self.step_rows = int(step_rows)

    # -- 2. attention ------------------------------------------------------------
    def attention(self, layer: int, q: np.ndarray, n_q: Optional[int] = None) -> np.ndarray:
        """Attention of the last ``n_q`` appended rows (queries ``q[n_q][Hq][D]``,
        pre-rotation) over the resident cache of ``layer``."""
        q = np.asarray(q, np.float64)
        n_q = q.shape[0] if n_q is None else n_q
        if n_q > self.step_rows:
            raise OracleError("queries must be rows of the current step")
        q_pos = self.pos[self.resident - n_q:]
        q_rot = rope.rotate(q, q_pos, self.theta)
        return attend(q_rot, self.k[layer], self.v[layer], q_pos, self.pos, self.scale)

    def attention_full_history(self, layer: int, q: np.ndarray) -> np.ndarray:
        """Same queries over every row ever appended, evicted rows masked out."""
        if not self.keep_history:
            raise OracleError("history not kept")
        q = np.asarray(q, np.float64)
        n_q = q.shape[0]
        q_pos = self.pos[self.resident - n_q:]
        q_rot = rope.rotate(q, q_pos, self.theta)
        return attend(q_rot, self.h_k[layer], self.h_v[layer], q_pos, self.h_pos,
                      self.scale, visible=self.h_resident)

    # -- 3. evict and compact ----------------------------------------------------
    def evict(self, budget: int, window: int, rule: Optional[EvictRule] = None) -> EvictRecord:
        """Sec. 3.3's rule after a unit (or, with ``rule``, one of its variants)."""
        if budget < 0 or window < 0:
            raise OracleError("budget and window are non-negative")
        rule = rule or EvictRule()
        if rule.kind == "sink_recent" and budget < rule.n_sink:
            raise OracleError("the budget must cover the sink rows")
        cur = -1 if self.cur is None else self.cur
        plan = plan_by_rule(rule, self.seg, self.unit, budget, window, cur)
        new_slot = compaction_indices(plan.evict_mask)
        keep = ~plan.evict_mask
        if self.keep_history and plan.evict_mask.any():
            gone = np.isin(self.h_pos, self.pos[plan.evict_mask])
            self.h_resident &= ~gone
        self.pos, self.seg, self.unit = self.pos[keep], self.seg[keep], self.unit[keep]
        for l in self.layers:
            self.k[l] = self.k[l][keep]
            self.v[l] = self.v[l][keep]
        self.step_rows = 0
        return EvictRecord(plan=plan, new_slot=new_slot, pos=self.pos.copy(),
                           seg=self.seg.copy(), unit=self.unit.copy())
