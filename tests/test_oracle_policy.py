"""Pins for the oracle's eviction policy and compaction indices (Sec. 3.3).

* a hand-worked golden fixture (tests/golden/eviction_worked_examples.json);
* an independent brute-force formulation: the smallest prefix of the eligible
  units (oldest first) whose removal brings R within B, else all of them,
  checked on random streams and exhaustively on tiny ones;
* the invariants and closed forms the paper's rule implies;
* mutation checks: plausible mistakes planted in a copy of the policy on the
  CPU must each fail at least one pin.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle.cache import OracleCache
from oracle.policy import EVICTABLE_SEGS, compaction_indices, plan_eviction
from synth.streams import (CONFIGS, SEG_ACOUSTIC, SEG_DELIM, SEG_PREFIX, SEG_RESPONSE, SEG_TEXT)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eviction_worked_examples.json")


def _run_golden(plan_fn):
    """Replay every golden example with ``plan_fn``; return the list of mismatches."""
    bad = []
    with open(GOLDEN) as f:
        data = json.load(f)
    for ex in data["examples"]:
        seg = np.zeros(0, np.uint8)
        unit = np.zeros(0, np.int64)
        cur = -1
        for i, st in enumerate(ex["steps"]):
            seg = np.concatenate([seg, np.asarray(st["seg"], np.uint8)])
            unit = np.concatenate([unit, np.full(len(st["seg"]), st["unit"], np.int64)])
            cur = max(cur, st["unit"])
            plan = plan_fn(seg, unit, st["budget"], ex["window"], cur)
            got = {"n_pre": plan.n_pre, "evicted_units": list(plan.units),
                   "n_post": plan.n_post, "budget_unmet": bool(plan.budget_unmet)}
            for key in got:
                if got[key] != st[key]:
                    bad.append((ex["name"], i, key, got[key], st[key]))
            if "mask" in st:
                if plan.evict_mask.astype(int).tolist() != st["mask"]:
                    bad.append((ex["name"], i, "mask"))
                if compaction_indices(plan.evict_mask).tolist() != st["new_slot"]:
                    bad.append((ex["name"], i, "new_slot"))
            keep = ~plan.evict_mask
            seg, unit = seg[keep], unit[keep]
            if "layout_seg" in st:
                if seg.tolist() != st["layout_seg"] or unit.tolist() != st["layout_unit"]:
                    bad.append((ex["name"], i, "layout"))
    return bad


def test_golden_worked_examples():
    assert _run_golden(plan_eviction) == []


# ---------------------------------------------------------------- brute force
def brute_force(seg, unit, budget, window, cur):
    """Closed form of the repeat-until loop: evict the shortest oldest-first
    prefix of eligible units that brings R within B (or all of them)."""
    seg, unit = np.asarray(seg), np.asarray(unit)
    ev = np.isin(seg, EVICTABLE_SEGS)
    eligible = sorted(set(unit[ev & (unit <= cur - window)].tolist()))
    R = len(seg)
    counts = [int((ev & (unit == u)).sum()) for u in eligible]
    k = 0
    if R > budget:
        k = len(eligible)
        for j in range(1, len(eligible) + 1):
            if R - sum(counts[:j]) <= budget:
                k = j
                break
    chosen = eligible[:k]
    mask = ev & np.isin(unit, chosen)
    return chosen, mask, R - int(mask.sum())


def _random_layout(rng, n_units, prefix, with_response=True):
    seg, unit = [SEG_PREFIX] * prefix, [-1] * prefix
    for u in range(n_units):
        rows = [SEG_ACOUSTIC] * int(rng.integers(0, 4)) + [SEG_DELIM] * int(rng.integers(0, 2)) \
            + [SEG_TEXT] * int(rng.integers(0, 3))
        if with_response and rng.random() < 0.3:
            rows += [SEG_RESPONSE] * int(rng.integers(1, 3))
        rng.shuffle(rows)
        seg += rows
        unit += [u] * len(rows)
    return np.asarray(seg, np.uint8), np.asarray(unit, np.int64)


def test_policy_matches_brute_force_random():
    rng = np.random.default_rng(123)
    for _ in range(3000):
        seg, unit = _random_layout(rng, int(rng.integers(0, 9)), int(rng.integers(0, 3)))
        cur = int(unit.max()) if unit.size and unit.max() >= 0 else -1
        B = int(rng.integers(0, len(seg) + 2))
        W = int(rng.integers(0, 5))
        plan = plan_eviction(seg, unit, B, W, cur)
        chosen, mask, post = brute_force(seg, unit, B, W, cur)
        assert plan.units == chosen
        np.testing.assert_array_equal(plan.evict_mask, mask)
        assert plan.n_post == post
        assert plan.budget_unmet == (post > B)


def test_policy_matches_brute_force_exhaustive_tiny():
    # every assignment of 3 units x 2 rows over {ACOUSTIC, TEXT, DELIM}, every B and W
    classes = [SEG_ACOUSTIC, SEG_TEXT, SEG_DELIM]
    for rows in itertools.product(classes, repeat=6):
        seg = np.asarray(rows, np.uint8)
        unit = np.repeat(np.arange(3), 2)
        for B in range(0, 8):
            for W in range(0, 4):
                plan = plan_eviction(seg, unit, B, W, 2)
                chosen, mask, post = brute_force(seg, unit, B, W, 2)
                assert plan.units == chosen and plan.n_post == post
                np.testing.assert_array_equal(plan.evict_mask, mask)


# ------------------------------------------------------------------ invariants
def _stream_invariants(plan, seg, unit, B, W, cur):
    keep = ~plan.evict_mask
    # I1: transcript / response / prefix rows are never evicted
    assert not np.any(plan.evict_mask & ~np.isin(seg, EVICTABLE_SEGS))
    # I2: every row of the W most recent units stays
    assert not np.any(plan.evict_mask & (unit > cur - W))
    # I3: within budget, or nothing eligible left
    left = np.isin(seg, EVICTABLE_SEGS) & keep & (unit <= cur - W)
    assert plan.n_post <= B or not left.any()
    # I6: whole units, oldest first, and they precede every remaining eligible unit
    for u in plan.units:
        assert not np.any(np.isin(seg, EVICTABLE_SEGS) & (unit == u) & keep)
    if plan.units and left.any():
        assert max(plan.units) < unit[left].min()
    assert plan.units == sorted(plan.units)
    # minimality: before the last evicted unit the cache still exceeded B
    if plan.units:
        last = plan.units[-1]
        n_last = int((plan.evict_mask & (unit == last)).sum())
        assert plan.n_post + n_last > B


def test_invariants_random_streams():
    rng = np.random.default_rng(7)
    for _ in range(300):
        seg, unit = _random_layout(rng, int(rng.integers(1, 30)), int(rng.integers(0, 5)))
        cur = int(unit.max())
        B, W = int(rng.integers(0, 60)), int(rng.integers(0, 6))
        plan = plan_eviction(seg, unit, B, W, cur)
        _stream_invariants(plan, seg, unit, B, W, cur)


def test_compaction_indices_equal_stable_partition():
    rng = np.random.default_rng(5)
    for _ in range(200):
        m = rng.random(int(rng.integers(0, 50))) < 0.4
        ns = compaction_indices(m)
        idx = np.arange(m.size)
        kept = idx[~m]                        # numpy stable boolean selection
        for j, i in enumerate(kept):
            assert ns[i] == j
        assert np.all(ns[m] == -1)


# ---------------------------------------------------------------- closed forms
def _run_stream(units_rows, B, W, prefix=0):
    c = OracleCache(1, 1, 4, layers=[])
    pos = 0
    recs = []
    if prefix:
        c.append([SEG_PREFIX] * prefix, list(range(prefix)), -1)
        pos = prefix
        recs.append(c.evict(B, W))
    for u, rows in enumerate(units_rows):
        c.append(rows, list(range(pos, pos + len(rows))), u)
        pos += len(rows)
        recs.append(c.evict(B, W))
    return c, recs


def _unit_rows(rng):
    t = min(int(rng.poisson(3)), 64)
    return [SEG_ACOUSTIC] * 17 + [SEG_DELIM] + [SEG_TEXT] * t + [SEG_DELIM]


def test_c1_large_budget_evicts_nothing():
    rng = np.random.default_rng(1)
    rows = [_unit_rows(rng) for _ in range(40)]
    total = sum(len(r) for r in rows) + 3
    c, recs = _run_stream(rows, total, 3, prefix=3)
    assert all(r.n_evicted == 0 for r in recs) and c.resident == total


def test_c2_zero_budget_is_the_floor():
    rng = np.random.default_rng(2)
    rows = [_unit_rows(rng) for _ in range(30)]
    W = 4
    c, recs = _run_stream(rows, 0, W, prefix=2)
    for u in range(len(rows)):
        text = sum(r.count(SEG_TEXT) for r in rows[: u + 1])
        recent = sum(len(r) for r in rows[max(0, u - W + 1): u + 1])
        recent_text = sum(r.count(SEG_TEXT) for r in rows[max(0, u - W + 1): u + 1])
        assert recs[u + 1].plan.n_post == 2 + text - recent_text + recent


def test_c3_window_covering_every_unit_evicts_nothing():
    rng = np.random.default_rng(3)
    rows = [_unit_rows(rng) for _ in range(12)]
    _, recs = _run_stream(rows, 0, 12)
    assert all(r.n_evicted == 0 for r in recs)


def test_c4_steady_state_band_like_table3():
    # Table 3: End <= B < Peak, Peak - B about one unit's rows.  Synthetic analogue.
    rng = np.random.default_rng(4)
    rows = [_unit_rows(rng) for _ in range(400)]
    B = 2000
    c, recs = _run_stream(rows, B, 30)
    max_rows = max(len(r) for r in rows)
    assert c.peak <= B + max_rows and c.peak > B
    for r in recs:
        if r.n_evicted and not r.plan.budget_unmet:
            assert B - 19 < r.plan.n_post <= B


# ---------------------------------------------------- mutations must be caught
def _mutant(window_shift=0, trigger_ge=False, newest_first=False, evict_text=False):
    evictable = EVICTABLE_SEGS + ((SEG_TEXT,) if evict_text else ())

    def plan_fn(seg, unit, budget, window, cur):
        ev = np.isin(seg, evictable)
        removed = np.zeros(len(seg), bool)
        R = len(seg)
        units = []
        while (R >= budget) if trigger_ge else (R > budget):
            el = unit[ev & ~removed & (unit <= cur - window + window_shift)]
            if el.size == 0:
                break
            u = int(el.max() if newest_first else el.min())
            rows = ev & ~removed & (unit == u)
            removed |= rows
            R -= int(rows.sum())
            units.append(u)
        from oracle.policy import EvictionPlan
        return EvictionPlan(units, removed, len(seg), R, R > budget)
    return plan_fn


@pytest.mark.parametrize("kw", [dict(window_shift=1), dict(window_shift=-1), dict(trigger_ge=True),
                                dict(newest_first=True), dict(evict_text=True)])
def test_planted_policy_mistakes_fail_the_golden(kw):
    assert _run_golden(_mutant(**kw)) != []


def test_budget_sweep_like_table3():
    # the KV-budget ablation (Table 3) on 15 synthetic ten-minute sessions: with a
    # feasible budget B the final residency sits just under B and the peak just over
    # it (at most one unit above); without eviction both equal the session's rows;
    # the floor keeps only transcript rows plus the recent window
    from synth.streams import make_sessions
    from oracle.replay import replay_metadata
    cfg = CONFIGS[1]
    w = make_sessions(cfg, range(1, 16))
    max_unit = cfg.max_unit_rows
    prev_end = None
    for B in (None, 8000, 6000, 4000, 0):
        ends, peaks = [], []
        for s in w.streams:
            tr = replay_metadata(s, 10 ** 9 if B is None else B, cfg.window, evict=B is not None)
            ends.append(tr.steps[-1].n_post)
            peaks.append(tr.peak)
            if B is None:
                assert ends[-1] == peaks[-1] == s.total_rows()
            elif B > 0:
                assert B - 19 < ends[-1] <= B < peaks[-1] <= B + max_unit
            else:
                text = sum(int(np.sum(st.seg == 3)) for st in s.steps)
                last = sum(st.n for st in s.steps[-cfg.window:])
                last_text = sum(int(np.sum(st.seg == 3)) for st in s.steps[-cfg.window:])
                assert ends[-1] == text - last_text + last
        if prev_end is not None:
            assert np.mean(ends) < prev_end
        prev_end = np.mean(ends)
