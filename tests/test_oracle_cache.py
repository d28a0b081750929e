"""Pins for the oracle's streaming cache (Sec. 3.3): attention over the
compacted cache equals attention over the full history with the evicted rows
masked; positions are preserved; the state after any step can be rebuilt."""
import numpy as np
import pytest

from oracle.cache import OracleCache, OracleError
from oracle.replay import replay_metadata, resume
from synth.streams import CONFIGS, make_workload, step_values, tiny_stream, SEG_TEXT


def _drive(cache, cfg, seed, spec, budget, window, n_steps, check=None, pos_shift=0):
    outs = []
    for i in range(n_steps):
        st = spec.steps[i]
        vals = step_values(cfg, seed, spec.stream, st.key, st.n, cache.layers)
        k = {l: vals["k"][j] for j, l in enumerate(cache.layers)}
        v = {l: vals["v"][j] for j, l in enumerate(cache.layers)}
        cache.append(st.seg, st.pos + pos_shift, st.unit, k, v)
        o = {l: cache.attention(l, vals["q"][j]) for j, l in enumerate(cache.layers)}
        if check:
            check(cache, vals, o)
        outs.append(o)
        cache.evict(budget, window)
    return outs


def test_compacted_equals_masked_full_history():
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=0).streams[0]
    cache = OracleCache(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, [0],
                        theta=cfg.rope_theta, scale=cfg.scale, keep_history=True)
    worst = [0.0]

    def check(c, vals, o):
        full = c.attention_full_history(0, vals["q"][0])
        worst[0] = max(worst[0], float(np.abs(full - o[0]).max()))
    _drive(cache, cfg, 0, spec, cfg.budget, cfg.window, 60, check)
    assert cache.h_resident.sum() < cache.h_resident.size     # eviction happened
    assert worst[0] <= 1e-12


def test_constant_position_shift_leaves_outputs_unchanged():
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=1, units=25).streams[0]
    a = OracleCache(4, 1, 64, [0], theta=cfg.rope_theta, scale=cfg.scale)
    b = OracleCache(4, 1, 64, [0], theta=cfg.rope_theta, scale=cfg.scale)
    oa = _drive(a, cfg, 1, spec, 200, 3, 25)
    ob = _drive(b, cfg, 1, spec, 200, 3, 25, pos_shift=7_777)
    for x, y in zip(oa, ob):
        np.testing.assert_allclose(x[0], y[0], atol=1e-9)


def test_resume_rebuilds_the_state():
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=2).streams[0]
    full = OracleCache(4, 1, 64, [0], theta=cfg.rope_theta, scale=cfg.scale)
    _drive(full, cfg, 2, spec, cfg.budget, cfg.window, 40)
    res = resume(cfg, 2, spec, cfg.budget, cfg.window, 40, [0])
    np.testing.assert_array_equal(res.pos, full.pos)
    np.testing.assert_array_equal(res.seg, full.seg)
    np.testing.assert_array_equal(res.unit, full.unit)
    np.testing.assert_array_equal(res.k[0], full.k[0])
    np.testing.assert_array_equal(res.v[0], full.v[0])
    # continuing both gives identical outputs
    rest_a = []
    rest_b = []
    for c, out in ((full, rest_a), (res, rest_b)):
        for i in range(40, 50):
            st = spec.steps[i]
            vals = step_values(cfg, 2, 0, st.key, st.n, [0])
            c.append(st.seg, st.pos, st.unit, {0: vals["k"][0]}, {0: vals["v"][0]})
            out.append(c.attention(0, vals["q"][0]))
            c.evict(cfg.budget, cfg.window)
    for x, y in zip(rest_a, rest_b):
        np.testing.assert_array_equal(x, y)


def test_replay_matches_cache_policy():
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=3).streams[0]
    tr = replay_metadata(spec, cfg.budget, cfg.window)
    c = OracleCache(4, 1, 64, [], theta=cfg.rope_theta)
    for i, st in enumerate(spec.steps):
        c.append(st.seg, st.pos, st.unit)
        r = c.evict(cfg.budget, cfg.window)
        assert r.plan.units == tr.steps[i].units and r.plan.n_post == tr.steps[i].n_post
    np.testing.assert_array_equal(c.pos, tr.pos)


def test_resume_without_eviction_at_a_decode_workload_shape():
    # no-eviction replay (linear path) equals the policy replay under a budget it
    # never exceeds; resume from it equals driving the cache step by step
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=4, decode_steps=5).streams[0]
    big = 10 ** 9
    a = replay_metadata(spec, big, cfg.window, evict=False)
    b = replay_metadata(spec, big, cfg.window, evict=True)
    for x, y in zip(a.steps, b.steps):
        assert (x.n_pre, x.n_post, x.units, x.budget_unmet) == (y.n_pre, y.n_post, y.units,
                                                                y.budget_unmet)
    assert a.peak == b.peak == spec.total_rows()
    for name in ("pos", "seg", "unit", "src_step", "src_row"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name))
    n = len(spec.steps)
    full = OracleCache(4, 1, 64, [0], theta=cfg.rope_theta, scale=cfg.scale)
    _drive(full, cfg, 4, spec, big, cfg.window, n)
    res = resume(cfg, 4, spec, big, cfg.window, n, [0])
    np.testing.assert_array_equal(res.k[0], full.k[0])
    np.testing.assert_array_equal(res.v[0], full.v[0])
    np.testing.assert_array_equal(res.unit, full.unit)


def test_load_rows_validates():
    c = OracleCache(1, 1, 4, [0])
    z = {0: np.zeros((2, 1, 4))}
    with pytest.raises(OracleError):
        c.load_rows([1, 1], [3, 3], [0, 0], z, z, 2)      # positions not increasing
    with pytest.raises(OracleError):
        c.load_rows([1, 7], [3, 4], [0, 0], z, z, 2)      # unknown class
    with pytest.raises(OracleError):
        c.load_rows([1, 1], [3, 4], [1, 0], z, z, 2)      # unit ids decrease
    c.load_rows([1, 3], [3, 4], [0, 0], z, z, 2)
    with pytest.raises(OracleError):
        c.load_rows([1, 3], [5, 6], [0, 0], z, z, 2)      # not empty


def test_append_validation():
    c = OracleCache(1, 1, 4, [])
    c.append([1, 1], [3, 4], 0)
    with pytest.raises(OracleError):
        c.append([1], [4], 1)                 # position not increasing
    with pytest.raises(OracleError):
        c.append([9], [5], 1)                 # unknown class
    c.append([1], [5], 2)
    with pytest.raises(OracleError):
        c.append([1], [6], 1)                 # unit id decreasing
    with pytest.raises(OracleError):
        c.attention(0, np.zeros((2, 1, 4)))   # more queries than new rows


def test_prefix_and_decode_rows_with_gaps_in_positions():
    spec = tiny_stream([[1, 1, 2, 3, 2], [4], [1, 1, 2, 2], [4], [1, 3]], prefix=3, pos_gap=5)
    c = OracleCache(2, 1, 8, [0], theta=1e4, keep_history=True)
    rng = np.random.default_rng(0)
    for st in spec.steps:
        c.append(st.seg, st.pos, st.unit, {0: rng.standard_normal((st.n, 1, 8))},
                 {0: rng.standard_normal((st.n, 1, 8))})
        q = rng.standard_normal((st.n, 2, 8))
        np.testing.assert_allclose(c.attention(0, q), c.attention_full_history(0, q), atol=1e-13)
        c.evict(4, 1)
    assert set(c.seg.tolist()) >= {0, 4}


def test_generator_shape_statistics():
    # about 17 acoustic + 2 delimiter + 3 text rows per unit (Sec. 1: ~17 vs ~3 per second)
    w = make_workload(1)
    s = w.streams[0]
    per_unit = s.total_rows() / s.n_units
    assert 21.5 < per_unit < 22.5
    texts = [int((st.seg == SEG_TEXT).sum()) for st in s.steps]
    assert 2.8 < np.mean(texts) < 3.2 and max(texts) <= 64
    tr = replay_metadata(s, 4096, 30)
    first = next(i for i, t in enumerate(tr.steps) if t.units)
    assert 180 <= first <= 192
