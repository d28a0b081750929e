"""Pins for the side-channel cadence (Sec. 3.1): a duplex unit's prefill chunk
followed by one decode step per side-channel token, with the budget checked
once per unit (Sec. 3.3).  The cadence carries the same rows as the chunk
workload, so the state at every unit end must match it, and causal attention
makes every decode step equal the same row of a chunk attention."""
import numpy as np

from oracle.cache import OracleCache
from oracle.replay import replay_metadata
from synth.streams import (CONFIGS, SEG_ACOUSTIC, make_cadence_workload, make_workload,
                           step_values)


def test_cadence_rows_match_the_chunk_workload():
    for cfg_i in (0, 1, 2):
        cfg = CONFIGS[cfg_i]
        a = make_cadence_workload(cfg, units=80, n_streams=3)
        b = make_workload(cfg, units=80, n_streams=3, decode_steps=0)
        for sa, sb in zip(a.streams, b.streams):
            assert (sa.offset, sa.budget) == (sb.offset, sb.budget)
            for f in ("pos", "seg"):
                np.testing.assert_array_equal(np.concatenate([getattr(s, f) for s in sa.steps]),
                                              np.concatenate([getattr(s, f) for s in sb.steps]))
            # one check per unit, after its closing delimiter
            assert sum(s.evict for s in sa.steps) == len(sb.steps)
            assert all(s.seg[-1] == 2 for s in sa.steps if s.evict)
            # a chunk of the acoustic rows, then single-row decode steps
            for s in sa.steps:
                assert s.decode == (s.n == 1) and (s.decode or np.all(s.seg == SEG_ACOUSTIC))
            keys = [s.key for s in sa.steps]
            assert len(set(keys)) == len(keys)


def test_state_at_unit_ends_matches_the_chunk_workload():
    for cfg_i, budget in ((0, 256), (0, 60), (1, 700), (2, 300)):
        cfg = CONFIGS[cfg_i]
        sa = make_cadence_workload(cfg, units=120, n_streams=1).streams[0]
        sb = make_workload(cfg, units=120, n_streams=1, decode_steps=0).streams[0]
        ta = replay_metadata(sa, budget, cfg.window)
        tb = replay_metadata(sb, budget, cfg.window)
        ends = [i for i, s in enumerate(sa.steps) if s.evict]
        assert len(ends) == len(tb.steps)
        for i, t in zip(ends, tb.steps):
            x = ta.steps[i]
            assert (x.n_pre, x.n_post, x.units, x.budget_unmet) == (t.n_pre, t.n_post, t.units,
                                                                    t.budget_unmet)
        # no eviction inside a unit
        assert all(x.n_pre == x.n_post for i, x in enumerate(ta.steps) if not sa.steps[i].evict)
        assert ta.peak == tb.peak
        np.testing.assert_array_equal(ta.pos, tb.pos)
        np.testing.assert_array_equal(ta.unit, tb.unit)


def test_decode_steps_equal_rows_of_the_chunk_attention():
    # same values: the chunk cache appends a whole unit, the cadence cache the
    # chunk then one row at a time; every cadence output must equal the chunk
    # output of that row (causal by position, nothing evicted inside a unit)
    cfg = CONFIGS[0]
    sb = make_workload(cfg, seed=5, units=30, decode_steps=0).streams[0]
    chunk = OracleCache(4, 1, 64, [0], theta=cfg.rope_theta, scale=cfg.scale)
    cad = OracleCache(4, 1, 64, [0], theta=cfg.rope_theta, scale=cfg.scale)
    worst = 0.0
    for st in sb.steps:
        v = step_values(cfg, 5, 0, st.key, st.n, [0])
        chunk.append(st.seg, st.pos, st.unit, {0: v["k"][0]}, {0: v["v"][0]})
        full = chunk.attention(0, v["q"][0])
        a = int(np.sum(st.seg == SEG_ACOUSTIC))
        cad.append(st.seg[:a], st.pos[:a], st.unit, {0: v["k"][0][:a]}, {0: v["v"][0][:a]})
        out = [cad.attention(0, v["q"][0][:a])]
        for r in range(a, st.n):
            cad.append(st.seg[r:r + 1], st.pos[r:r + 1], st.unit, {0: v["k"][0][r:r + 1]},
                       {0: v["v"][0][r:r + 1]})
            out.append(cad.attention(0, v["q"][0][r:r + 1]))
        worst = max(worst, float(np.abs(np.concatenate(out) - full).max()))
        chunk.evict(cfg.budget, cfg.window)
        cad.evict(cfg.budget, cfg.window)
    assert worst <= 1e-12
