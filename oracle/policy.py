"""Online budgeted eviction, step by step (oracle; test infrastructure only).

Sec. 3.3 of the paper, in its order:

1. After each duplex unit, count the resident KV positions R, including the
   system prefix and the text entries, and compare with the budget B.
2. If the cache exceeds B (R > B), take the oldest unit outside the W most
   recent units (the retention window) that still holds acoustic/structural
   rows, and evict those rows (unit marker, audio tokens, native decision,
   ASR delimiters, terminators).  Transcript tokens, model response text and
   the system prefix are kept.
3. Repeat until the cache fits (R <= B) or no eligible unit remains.

Readings (the paper is silent or loose here):
  * evictable classes are ACOUSTIC (marker, audio, decision, terminators) and
    DELIM (the ASR delimiters); TEXT, RESPONSE and PREFIX are never evicted;
  * the W most recent units are cur-W+1 .. cur, with cur the newest unit id,
    so a unit u is eligible iff u <= cur - W;
  * a whole unit's evictable rows go at once (the paper evicts "from the
    oldest unit" and repeats per unit);
  * if no eligible unit remains while R > B the call still succeeds and the
    budget is reported unmet.

Compaction keeps the survivors in their original order: the new index of a
kept row is the number of kept rows before it.

Two variants of the rule (per-row granularity, and the sink + recent window
of the StreamingLLM comparison) follow ``plan_eviction`` below.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np

from synth.streams import SEG_ACOUSTIC, SEG_DELIM

EVICTABLE_SEGS = (SEG_ACOUSTIC, SEG_DELIM)


@dataclass
class EvictionPlan:
    units: List[int]          # evicted unit ids, oldest first
    evict_mask: np.ndarray    # bool [R_pre], True = row evicted
    n_pre: int
    n_post: int
    budget_unmet: bool


def plan_eviction(seg: np.ndarray, unit: np.ndarray, budget: int, window: int,
                  cur: int) -> EvictionPlan:
    """Apply the Sec. 3.3 rule to one stream's resident rows (in cache order)."""
    seg = np.asarray(seg)
    unit = np.asarray(unit)
    evictable = np.isin(seg, EVICTABLE_SEGS)
    removed = np.zeros(seg.shape[0], bool)
    resident = int(seg.shape[0])
    units: List[int] = []
    while resident > budget:
        still = evictable & ~removed
        eligible = unit[still & (unit <= cur - window)]
        if eligible.size == 0:
            break
        oldest = int(eligible.min())
        rows = still & (unit == oldest)
        removed |= rows
        resident -= int(rows.sum())
        units.append(oldest)
    return EvictionPlan(units=units, evict_mask=removed, n_pre=int(seg.shape[0]),
                        n_post=resident, budget_unmet=resident > budget)


def compaction_indices(evict_mask: np.ndarray) -> np.ndarray:
    """new_slot[i] = number of kept rows before i, or -1 if row i is evicted."""
    keep = ~np.asarray(evict_mask, bool)
    before = np.cumsum(keep) - keep
    return np.where(keep, before, -1).astype(np.int32)


# ----------------------------------------------------------------- rule variants
# Two variants of the eviction rule run on the same cache, both evaluated at the
# same points as the paper's rule (after each duplex unit):
#
# * "row": an ablation of Sec. 3.3's granularity.  Eligibility is the paper's
#   (acoustic/structural rows of units outside the W most recent units), but
#   the loop removes one row at a time, the oldest eligible row first, and
#   stops as soon as R <= B; a unit can therefore lose only part of its rows.
# * "sink_recent": the StreamingLLM comparison of Sec. 2 and Table 1 (attention
#   sinks plus a recent window of 2,000 positions).  Whatever their class, every
#   resident row is evicted except the n_sink oldest rows and the B - n_sink
#   newest ones (B = n_sink + recent); the window W plays no part.  The paper
#   does not state the sink count: it is a parameter (4 by default).

RULES = ("unit", "row", "sink_recent")


@dataclass(frozen=True)
class EvictRule:
    kind: str = "unit"
    n_sink: int = 4

    def __post_init__(self):
        if self.kind not in RULES:
            raise ValueError(f"unknown eviction rule {self.kind!r}")
        if self.n_sink < 0:
            raise ValueError("n_sink is non-negative")


def _touched_units(unit: np.ndarray, mask: np.ndarray) -> List[int]:
    """Unit ids that lose at least one row, oldest first."""
    out: List[int] = []
    for u in unit[mask].tolist():
        if not out or out[-1] != u:
            out.append(int(u))
    return out


def plan_eviction_rows(seg: np.ndarray, unit: np.ndarray, budget: int, window: int,
                       cur: int) -> EvictionPlan:
    """Per-row ablation: while R > B, remove the single oldest resident
    acoustic/structural row whose unit is outside the window."""
    seg = np.asarray(seg)
    unit = np.asarray(unit)
    evictable = np.isin(seg, EVICTABLE_SEGS)
    removed = np.zeros(seg.shape[0], bool)
    resident = int(seg.shape[0])
    while resident > budget:
        candidates = np.flatnonzero(evictable & ~removed & (unit <= cur - window))
        if candidates.size == 0:
            break
        removed[candidates[0]] = True      # rows are in position order: the first is the oldest
        resident -= 1
    return EvictionPlan(units=_touched_units(unit, removed), evict_mask=removed,
                        n_pre=int(seg.shape[0]), n_post=resident, budget_unmet=resident > budget)


def plan_eviction_sink_recent(unit: np.ndarray, budget: int, n_sink: int) -> EvictionPlan:
    """StreamingLLM comparison: keep the ``n_sink`` oldest rows and the
    ``budget - n_sink`` newest rows, evict every other row of any class."""
    unit = np.asarray(unit)
    if budget < n_sink:
        raise ValueError("the budget must cover the sink rows")
    R = int(unit.shape[0])
    removed = np.zeros(R, bool)
    if R > budget:
        recent = budget - n_sink
        for i in range(R):
            removed[i] = n_sink <= i < R - recent
    n_post = R - int(removed.sum())
    return EvictionPlan(units=_touched_units(unit, removed), evict_mask=removed, n_pre=R,
                        n_post=n_post, budget_unmet=n_post > budget)


def plan_by_rule(rule: "EvictRule", seg: np.ndarray, unit: np.ndarray, budget: int,
                 window: int, cur: int) -> EvictionPlan:
    if rule.kind == "unit":
        return plan_eviction(seg, unit, budget, window, cur)
    if rule.kind == "row":
        return plan_eviction_rows(seg, unit, budget, window, cur)
    return plan_eviction_sink_recent(unit, budget, rule.n_sink)
