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
