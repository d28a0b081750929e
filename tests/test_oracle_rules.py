"""Pins for the oracle's variants of the eviction rule: per-row granularity
(an ablation of Sec. 3.3's whole-unit rule) and the sink + recent window of
the StreamingLLM comparison (Sec. 2, Table 1).

* a hand-worked golden fixture (tests/golden/eviction_rule_variants.json);
* independent formulations: the row rule as "the first min(R - B, |E|)
  eligible rows in cache order" (a closed form of its loop), the sink rule as
  a token-by-token StreamingLLM window (push every row, drop the oldest
  non-sink row whenever the window overflows), compared at every unit end;
* relations between the rules from the same state, invariants and closed
  forms;
* mistakes planted in copies of the oracle functions (on the CPU) must each
  fail a pin.
"""
import collections
import itertools
import json
import os

import numpy as np
import pytest

from oracle.cache import OracleCache
from oracle.policy import (EVICTABLE_SEGS, EvictRule, EvictionPlan, compaction_indices,
                           plan_by_rule, plan_eviction, plan_eviction_rows,
                           plan_eviction_sink_recent)
from oracle.replay import replay_metadata
from synth.streams import (CONFIGS, SEG_ACOUSTIC, SEG_DELIM, SEG_PREFIX, SEG_RESPONSE, SEG_TEXT,
                           make_workload)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eviction_rule_variants.json")


def _run_golden(plan_fn, only=None):
    """Replay every golden example; ``plan_fn(rule, seg, unit, budget, window, cur)``."""
    bad = []
    with open(GOLDEN) as f:
        data = json.load(f)
    for ex in data["examples"]:
        if only and ex["rule"] != only:
            continue
        rule = EvictRule(ex["rule"], ex["n_sink"])
        seg = np.zeros(0, np.uint8)
        unit = np.zeros(0, np.int64)
        cur = -1
        for i, st in enumerate(ex["steps"]):
            seg = np.concatenate([seg, np.asarray(st["seg"], np.uint8)])
            unit = np.concatenate([unit, np.full(len(st["seg"]), st["unit"], np.int64)])
            cur = max(cur, st["unit"])
            plan = plan_fn(rule, seg, unit, st["budget"], ex["window"], cur)
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


def test_golden_rule_variants():
    assert _run_golden(plan_by_rule) == []


# ------------------------------------------------------------ independent forms
def row_closed_form(seg, unit, budget, window, cur):
    """The row rule's loop in closed form: the first min(R - B, |E|) rows of the
    eligible set E in cache order."""
    seg, unit = np.asarray(seg), np.asarray(unit)
    eligible = np.flatnonzero(np.isin(seg, EVICTABLE_SEGS) & (unit <= cur - window))
    k = max(0, min(len(seg) - budget, eligible.size))
    mask = np.zeros(len(seg), bool)
    mask[eligible[:k]] = True
    return mask


def streaming_window(rows, n_sink, budget):
    """Token-by-token StreamingLLM window over a stream's rows (ids in
    arrival order): the first n_sink ids are sinks; whenever more than
    ``budget`` ids are held the oldest non-sink id is dropped."""
    sinks, recent = [], collections.deque()
    for r in rows:
        if len(sinks) < n_sink:
            sinks.append(r)
        else:
            recent.append(r)
        while len(sinks) + len(recent) > budget:
            recent.popleft()
    return sinks + list(recent)


def _random_layout(rng, n_units, prefix):
    seg, unit = [SEG_PREFIX] * prefix, [-1] * prefix
    for u in range(n_units):
        rows = [SEG_ACOUSTIC] * int(rng.integers(0, 4)) + [SEG_DELIM] * int(rng.integers(0, 2)) \
            + [SEG_TEXT] * int(rng.integers(0, 3))
        if rng.random() < 0.3:
            rows += [SEG_RESPONSE] * int(rng.integers(1, 3))
        rng.shuffle(rows)
        seg += rows
        unit += [u] * len(rows)
    return np.asarray(seg, np.uint8), np.asarray(unit, np.int64)


def test_row_rule_matches_closed_form_random():
    rng = np.random.default_rng(7)
    for _ in range(3000):
        seg, unit = _random_layout(rng, int(rng.integers(0, 9)), int(rng.integers(0, 3)))
        cur = int(unit.max()) if unit.size and unit.max() >= 0 else -1
        B, W = int(rng.integers(0, len(seg) + 2)), int(rng.integers(0, 5))
        plan = plan_eviction_rows(seg, unit, B, W, cur)
        want = row_closed_form(seg, unit, B, W, cur)
        np.testing.assert_array_equal(plan.evict_mask, want)
        assert plan.n_post == len(seg) - int(want.sum())
        assert plan.budget_unmet == (plan.n_post > B)


def test_row_rule_matches_closed_form_exhaustive_tiny():
    classes = [SEG_ACOUSTIC, SEG_TEXT, SEG_DELIM]
    unit = np.repeat(np.arange(3), 2)
    for rows in itertools.product(classes, repeat=6):
        seg = np.asarray(rows, np.uint8)
        for B in range(0, 8):
            for W in range(0, 4):
                plan = plan_eviction_rows(seg, unit, B, W, 2)
                np.testing.assert_array_equal(plan.evict_mask, row_closed_form(seg, unit, B, W, 2))


@pytest.mark.parametrize("n_sink,budget", [(0, 1), (0, 7), (1, 1), (2, 5), (4, 40), (4, 4), (3, 60)])
def test_sink_rule_matches_token_by_token_window(n_sink, budget):
    """Evicting after each unit leaves the same rows at every unit end as the
    token-by-token window (dropping the oldest non-sink row is order-free)."""
    spec = make_workload(CONFIGS[0], seed=3, units=40).streams[0]
    ids = np.zeros(0, np.int64)
    unit = np.zeros(0, np.int64)
    arrived = []
    for st in spec.steps:
        new = np.arange(len(arrived), len(arrived) + st.n)
        arrived.extend(new.tolist())
        ids = np.concatenate([ids, new])
        unit = np.concatenate([unit, np.full(st.n, st.unit, np.int64)])
        plan = plan_eviction_sink_recent(unit, budget, n_sink)
        keep = ~plan.evict_mask
        ids, unit = ids[keep], unit[keep]
        assert ids.tolist() == streaming_window(arrived, n_sink, budget)


# ---------------------------------------------------------- relations, invariants
def test_row_rule_is_a_prefix_of_the_unit_rule():
    """From one state: the rows the row rule evicts are among those the unit
    rule evicts, it evicts exactly min(R - B, eligible) rows, and the two
    agree whenever R - B reaches a unit boundary."""
    rng = np.random.default_rng(11)
    for _ in range(2000):
        seg, unit = _random_layout(rng, int(rng.integers(1, 9)), int(rng.integers(0, 3)))
        if not unit.size:
            continue
        cur = int(unit.max())
        B, W = int(rng.integers(0, len(seg) + 2)), int(rng.integers(0, 4))
        row = plan_eviction_rows(seg, unit, B, W, cur)
        whole = plan_eviction(seg, unit, B, W, cur)
        assert not np.any(row.evict_mask & ~whole.evict_mask)
        eligible = int((np.isin(seg, EVICTABLE_SEGS) & (unit <= cur - W)).sum())
        assert int(row.evict_mask.sum()) == max(0, min(len(seg) - B, eligible))
        assert row.budget_unmet == whole.budget_unmet
        if whole.n_post == B:
            np.testing.assert_array_equal(row.evict_mask, whole.evict_mask)


def test_row_rule_invariants_over_streams():
    """No transcript/response/prefix row evicted; the window stays resident;
    R <= B after every check unless nothing eligible is left; exactly B when
    the budget is met and eviction ran."""
    cfg = CONFIGS[0]
    for seed in range(4):
        spec = make_workload(cfg, seed=seed, units=60).streams[0]
        c = OracleCache(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, [])
        for st in spec.steps:
            c.append(st.seg, st.pos, st.unit)
            pre_seg, pre_unit = c.seg.copy(), c.unit.copy()
            rec = c.evict(150, 3, EvictRule("row"))
            m = rec.plan.evict_mask
            assert not np.any(m & ~np.isin(pre_seg, EVICTABLE_SEGS))
            assert not np.any(m & (pre_unit > c.cur - 3))
            if rec.plan.budget_unmet:
                assert not np.any(np.isin(c.seg, EVICTABLE_SEGS) & (c.unit <= c.cur - 3))
            elif m.any():
                assert c.resident == 150


def test_sink_rule_closed_forms():
    rng = np.random.default_rng(5)
    for _ in range(500):
        seg, unit = _random_layout(rng, int(rng.integers(0, 9)), int(rng.integers(0, 3)))
        R = len(seg)
        n_sink = int(rng.integers(0, 5))
        B = n_sink + int(rng.integers(0, R + 2))
        plan = plan_eviction_sink_recent(unit, B, n_sink)
        assert plan.n_post == min(R, B) and not plan.budget_unmet
        if R <= B:
            assert not plan.evict_mask.any()
        else:
            keep = np.flatnonzero(~plan.evict_mask)
            assert keep.tolist() == list(range(n_sink)) + list(range(R - (B - n_sink), R))
    with pytest.raises(ValueError):
        plan_eviction_sink_recent(np.zeros(3, np.int64), 2, 3)


def test_rule_special_cases():
    """B >= R evicts nothing under every rule; with one evictable row per unit
    the row rule is the unit rule; B = 0 empties the eligible set under both."""
    rng = np.random.default_rng(2)
    for _ in range(300):
        seg, unit = _random_layout(rng, int(rng.integers(1, 8)), 1)
        cur = max(int(unit.max()), 0)
        for kind in ("unit", "row"):
            assert not plan_by_rule(EvictRule(kind), seg, unit, len(seg), 1, cur).evict_mask.any()
        a = plan_eviction_rows(seg, unit, 0, 1, cur).evict_mask
        b = plan_eviction(seg, unit, 0, 1, cur).evict_mask
        np.testing.assert_array_equal(a, b)
        # one evictable row per unit: keep the first evictable row of each unit only
        ev = np.isin(seg, EVICTABLE_SEGS)
        first = np.zeros(len(seg), bool)
        for u in np.unique(unit):
            idx = np.flatnonzero(ev & (unit == u))
            if idx.size:
                first[idx[0]] = True
        seg1 = np.where(ev & ~first, SEG_TEXT, seg).astype(np.uint8)
        B = int(rng.integers(0, len(seg) + 1))
        np.testing.assert_array_equal(plan_eviction_rows(seg1, unit, B, 1, cur).evict_mask,
                                      plan_eviction(seg1, unit, B, 1, cur).evict_mask)


@pytest.mark.parametrize("rule", [EvictRule("row"), EvictRule("sink_recent", 4)])
def test_compacted_attention_equals_masked_full_history(rule):
    """Attention over the cache compacted by either variant equals attention
    over the full history with the evicted rows masked (no re-encoding)."""
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=1, units=30).streams[0]
    rng = np.random.default_rng(0)
    c = OracleCache(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, [0], theta=cfg.rope_theta,
                    keep_history=True)
    budget = 120 if rule.kind == "row" else 64
    evicted = 0
    for st in spec.steps:
        k = {0: rng.standard_normal((st.n, cfg.n_kv_heads, cfg.head_dim))}
        v = {0: rng.standard_normal((st.n, cfg.n_kv_heads, cfg.head_dim))}
        c.append(st.seg, st.pos, st.unit, k, v)
        q = rng.standard_normal((st.n, cfg.n_q_heads, cfg.head_dim))
        np.testing.assert_allclose(c.attention(0, q), c.attention_full_history(0, q),
                                   rtol=0, atol=1e-12)
        evicted += c.evict(budget, cfg.window, rule).n_evicted
    assert evicted > 0


def test_replay_settled_matches_layout_under_variants():
    """The rows the variants settle into the retained prefix: survivors older
    than the newest row ever evicted (row rule), the sink rows (sink rule)."""
    from oracle.replay import MetadataReplay
    spec = make_workload(CONFIGS[1], seed=1, units=260).streams[0]
    rp = MetadataReplay(spec, 4096, 30, rule=EvictRule("row"), record_masks=True)
    settled, newest, evicting = 0, -1, 0
    for _ in spec.steps:
        st = spec.steps[rp.i]
        pos_pre = np.concatenate([rp.pos, st.pos])
        s = rp.step()
        settled += s.settled
        if s.evict_mask.any():
            evicting += 1
            newest = max(newest, int(pos_pre[np.flatnonzero(s.evict_mask)[-1]]))
            # a feasible budget is met exactly: the row rule stops at R = B
            assert s.n_post == 4096 or s.budget_unmet
    assert evicting > 50
    assert settled == int((rp.pos < newest).sum())
    tr = replay_metadata(spec, 4 + 2000, 30, rule=EvictRule("sink_recent", 4))
    assert sum(s.settled for s in tr.steps) == 4
    assert tr.pos[:4].tolist() == [0, 1, 2, 3]


# ------------------------------------------------------------------ mutations
def _mut_row_newest_first(seg, unit, budget, window, cur):
    seg, unit = np.asarray(seg), np.asarray(unit)
    removed = np.zeros(len(seg), bool)
    R = len(seg)
    while R > budget:
        cand = np.flatnonzero(np.isin(seg, EVICTABLE_SEGS) & ~removed & (unit <= cur - window))
        if cand.size == 0:
            break
        removed[cand[-1]] = True
        R -= 1
    return EvictionPlan([], removed, len(seg), R, R > budget)


def _mut_row_window_off_by_one(seg, unit, budget, window, cur):
    return plan_eviction_rows(seg, unit, budget, window + 1, cur)


def _mut_row_text_evicted(seg, unit, budget, window, cur):
    seg = np.where(np.asarray(seg) == SEG_TEXT, SEG_ACOUSTIC, seg)
    return plan_eviction_rows(seg, unit, budget, window, cur)


def _mut_row_ge_trigger(seg, unit, budget, window, cur):
    return plan_eviction_rows(seg, unit, budget - 1, window, cur)


def _mut_row_is_unit(seg, unit, budget, window, cur):
    return plan_eviction(seg, unit, budget, window, cur)


def _mut_sink_count(unit, budget, n_sink):
    return plan_eviction_sink_recent(unit, budget, max(0, n_sink - 1)) if n_sink else \
        plan_eviction_sink_recent(unit, budget + 1, 1)


def _mut_sink_recent_count(unit, budget, n_sink):
    return plan_eviction_sink_recent(unit, budget - 1, min(n_sink, budget - 1)) if budget > 0 else \
        plan_eviction_sink_recent(unit, budget, n_sink)


@pytest.mark.parametrize("mut", [_mut_row_newest_first, _mut_row_window_off_by_one,
                                 _mut_row_text_evicted, _mut_row_ge_trigger, _mut_row_is_unit])
def test_planted_row_mistakes_fail_the_golden(mut):
    def fn(rule, seg, unit, budget, window, cur):
        if rule.kind == "row":
            return mut(seg, unit, budget, window, cur)
        return plan_by_rule(rule, seg, unit, budget, window, cur)
    assert _run_golden(fn, only="row") != []


@pytest.mark.parametrize("mut", [_mut_sink_count, _mut_sink_recent_count])
def test_planted_sink_mistakes_fail_the_golden(mut):
    def fn(rule, seg, unit, budget, window, cur):
        if rule.kind == "sink_recent":
            return mut(unit, budget, rule.n_sink)
        return plan_by_rule(rule, seg, unit, budget, window, cur)
    assert _run_golden(fn, only="sink_recent") != []


def test_sink_rule_keeping_transcript_fails_the_golden():
    """A sink rule that protects transcript rows (the paper's classes) is a
    different rule: the golden must tell them apart."""
    def fn(rule, seg, unit, budget, window, cur):
        plan = plan_by_rule(rule, seg, unit, budget, window, cur)
        mask = plan.evict_mask & (np.asarray(seg) != SEG_TEXT)
        return EvictionPlan(plan.units, mask, plan.n_pre, plan.n_pre - int(mask.sum()),
                            plan.budget_unmet)
    assert _run_golden(fn, only="sink_recent") != []
