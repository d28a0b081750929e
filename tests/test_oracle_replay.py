"""Pins of the oracle's metadata replay: the per-step masks and compaction
indices it records, the rows an in-place compaction would shift (``moved``),
and the rows that join the retained prefix (``settled``), each against a
closed form that does not reuse the replay's own arithmetic."""
import numpy as np
import pytest

from oracle.cache import OracleCache
from oracle.replay import MetadataReplay, replay_metadata
from synth.streams import (CONFIGS, SEG_PREFIX, SEG_RESPONSE, SEG_TEXT, make_cadence_workload,
                           make_workload, tiny_stream)


def _streams():
    out = [(make_workload(CONFIGS[0], seed=s).streams[0], 256, 3) for s in range(6)]
    w = make_workload(2, units=240)
    out += [(s, s.budget // 8, 6) for s in w.streams[:4]]
    out.append((tiny_stream([[1, 1, 2, 3, 2]] * 6 + [[4]] * 3 + [[1, 2, 3, 3, 2]] * 5,
                            prefix=3, pos_gap=1), 12, 1))
    return out


def test_recorded_masks_equal_the_cache_policy():
    for spec, B, W in _streams():
        tr = replay_metadata(spec, B, W, record_masks=True)
        c = OracleCache(4, 1, 64, [])
        for st, t in zip(spec.steps, tr.steps):
            c.append(st.seg, st.pos, st.unit)
            rec = c.evict(B, W)
            np.testing.assert_array_equal(t.evict_mask, rec.plan.evict_mask)
            np.testing.assert_array_equal(t.new_slot, rec.new_slot)


def test_moved_is_the_survivors_whose_slot_changes():
    # an in-place stable compaction shifts exactly the survivors whose new slot
    # differs from their old one
    for spec, B, W in _streams():
        for t in replay_metadata(spec, B, W, record_masks=True).steps:
            keep = ~t.evict_mask
            idx = np.arange(t.n_pre)
            assert t.moved == int(np.sum(keep & (t.new_slot != idx)))


def _class_counts(spec):
    """Per unit id: rows of each class over the stream's steps."""
    out = {}
    for st in spec.steps:
        d = out.setdefault(st.unit, np.zeros(5, np.int64))
        d += np.bincount(st.seg, minlength=5)
    return out


def test_settled_is_the_retained_rows_of_the_evicted_units():
    # whole units go oldest first, so a step that evicts units u1 < ... < uk adds
    # to the retained prefix the text and response rows of those units and of
    # every older unit that held no evictable row (the prefix, unit -1, at the
    # first eviction); nothing else ever joins it
    for spec, B, W in _streams():
        counts = _class_counts(spec)
        done = -2
        for t in replay_metadata(spec, B, W).steps:
            if not t.units:
                assert t.settled == 0
                continue
            hi = max(t.units)
            want = sum(int(c[SEG_TEXT] + c[SEG_RESPONSE] + c[SEG_PREFIX])
                       for u, c in counts.items() if done < u <= hi)
            assert t.settled == want, (t.units, t.settled, want)
            done = hi


def test_settled_counts_rows_appended_under_an_evicted_unit_id():
    # window 0: a response row appended (under unit id 0) after unit 0 was
    # evicted joins the prefix at the next eviction (unit 1) with unit 1's text
    # row; unit 2 retains nothing
    spec = tiny_stream([[1, 1, 3], [4], [1, 1, 3], [1, 1]])
    steps = replay_metadata(spec, 2, 0).steps
    assert [t.units for t in steps] == [[0], [], [1], [2]]
    assert [t.settled for t in steps] == [1, 0, 2, 0]


def test_settled_over_a_ten_minute_session_is_the_retained_text():
    spec = make_workload(CONFIGS[1], seed=1).streams[0]
    tr = replay_metadata(spec, 4096, 30)
    last = max(u for t in tr.steps for u in t.units)
    text = sum(int(np.sum(st.seg == SEG_TEXT)) for st in spec.steps if st.unit <= last)
    assert sum(t.settled for t in tr.steps) == text


def test_incremental_replay_equals_the_whole_run():
    spec = make_cadence_workload(CONFIGS[0], seed=2).streams[0]
    whole = replay_metadata(spec, 200, 2)
    rp = MetadataReplay(spec, 200, 2)
    for t in whole.steps:
        s = rp.step()
        assert (s.n_pre, s.n_post, s.units, s.budget_unmet, s.moved, s.settled) == \
               (t.n_pre, t.n_post, t.units, t.budget_unmet, t.moved, t.settled)
    np.testing.assert_array_equal(rp.pos, whole.pos)
