"""GPU parity: libA2T on the MI355X against the fp64 CPU oracle, same seeded inputs.

Bars: eviction counts, budget flags, device layout, eviction masks and
compaction indices bit-exact every step; compaction moves every surviving
row's bytes unchanged; attention max abs error <= 1e-4 for fp32 caches and
<= 2e-2 for bf16 caches (fp32 accumulation).
"""
import dataclasses
import os

import numpy as np
import pytest

from synth.streams import CONFIGS, make_workload, tiny_stream
from tests.harness import Lockstep, row_bounds

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


def _bounds(specs, budget, slack=0):
    total = max(row_bounds(s)[0] for s in specs)
    keep = max(row_bounds(s)[1] for s in specs)
    max_step = max(row_bounds(s)[2] for s in specs)
    return dict(unit_rows=total + slack, kept_rows=keep + 1, max_step=max_step)


def _report(ls, name):
    print(f"[{name}] steps={ls.steps_done} evictions={ls.evictions} max_err={ls.max_err:.3e}",
          flush=True)


@pytest.mark.parametrize("seed", range(10))
def test_config0_fp32(gpu, seed):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=seed).streams[0]
    ls = Lockstep(cfg, seed, [spec], layers_checked=[0], n_layers=1, budgets=[cfg.budget],
                  window=cfg.window, tol=F32_TOL, **_bounds([spec], cfg.budget))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"cfg0 seed{seed}")
    assert ls.evictions > 40
    if seed == 4:  # the seed whose stream runs out of eligible units near the end
        assert ls.unmet_steps > 0


@pytest.mark.parametrize("seed", [0, 4])
def test_config0_shape_bf16_mfma(gpu, seed):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=seed).streams[0]
    ls = Lockstep(cfg, seed, [spec], layers_checked=[0], n_layers=1, budgets=[cfg.budget],
                  window=cfg.window, tol=BF16_TOL, dtype="bf16", **_bounds([spec], cfg.budget))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"cfg0-bf16 seed{seed}")
    assert ls.evictions > 40


@pytest.mark.parametrize("hq,hkv,d,splits,fused", [
    (8, 2, 128, None, False),   # two KV heads, group 4
    (24, 3, 64, "5", True),     # KV-head count that does not divide the 8 XCDs, group 8
    (32, 4, 128, "9", False),   # group 8 at head dim 128, forced splits
    (16, 16, 64, None, True),   # multi-head attention (group 1)
])
def test_other_gqa_shapes_bf16(gpu, hq, hkv, d, splits, fused):
    """The MFMA attention at head shapes other than the workloads': workgroup
    (split, KV head) numbering for any KV-head count, query groups of 1 to 8
    heads, head dims 64 and 128, planned and forced key splits, with and
    without the fused append; config 0's stream structure, bf16, against the
    fp64 oracle."""
    cfg = dataclasses.replace(CONFIGS[0], n_q_heads=hq, n_kv_heads=hkv, head_dim=d)
    spec = make_workload(cfg, seed=11).streams[0]
    old = os.environ.get("A2T_SPLITS")
    if splits:
        os.environ["A2T_SPLITS"] = splits
    try:
        ls = Lockstep(cfg, 11, [spec], layers_checked=[0], n_layers=1, budgets=[cfg.budget],
                      window=cfg.window, tol=BF16_TOL, dtype="bf16", fused=fused,
                      **_bounds([spec], cfg.budget))
        try:
            ls.run()
        finally:
            ls.close()
    finally:
        if old is None:
            os.environ.pop("A2T_SPLITS", None)
        else:
            os.environ["A2T_SPLITS"] = old
    _report(ls, f"heads {hq}/{hkv} D{d} splits {splits or 'planned'}{' fused' if fused else ''}")
    assert ls.evictions > 40


def test_all_layers_append_and_partial_queries(gpu):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=5).streams[0]
    for dtype, tol in (("f32", F32_TOL), ("bf16", BF16_TOL)):
        ls = Lockstep(cfg, 5, [spec], layers_checked=[0, 1], n_layers=2, budgets=[cfg.budget],
                      window=cfg.window, tol=tol, dtype=dtype, all_layers_append=True,
                      query_rows=5, **_bounds([spec], cfg.budget))
        try:
            ls.run()
        finally:
            ls.close()
        _report(ls, f"all-layers {dtype}")


def test_config1_shape_first_210_units(gpu):
    cfg = CONFIGS[1]
    spec = make_workload(cfg, units=210).streams[0]
    ls = Lockstep(cfg, cfg.index, [spec], layers_checked=[0, 17, 35], n_layers=36,
                  budgets=[cfg.budget], window=cfg.window, tol=BF16_TOL, check_kv_every=15,
                  **_bounds([spec], cfg.budget))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, "cfg1 210 units")
    assert ls.evictions >= 20


def test_config1_full_600_units(gpu):
    # the benchmark's workload at full size: every step's eviction and layout,
    # attention on the last layer at every unit
    cfg = CONFIGS[1]
    spec = make_workload(cfg).streams[0]
    ls = Lockstep(cfg, cfg.index, [spec], layers_checked=[35], n_layers=36, budgets=[cfg.budget],
                  window=cfg.window, tol=BF16_TOL, check_kv_every=60, unit_rows=4096 + 200,
                  kept_rows=2048, max_step=cfg.max_unit_rows)
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, "cfg1 600 units")
    assert ls.evictions == 414


def test_config3_shape_decode(gpu):
    cfg = CONFIGS[3]
    w = make_workload(cfg, n_streams=3, units=200, decode_steps=24)
    specs = w.streams
    ls = Lockstep(cfg, cfg.index, specs, layers_checked=[0, 35], n_layers=36,
                  budgets=[cfg.budget] * 3, window=cfg.window, tol=BF16_TOL, check_kv_every=40,
                  **_bounds(specs, cfg.budget))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, "cfg3 decode")
    assert ls.evictions > 0


def test_config2_shape_varlen(gpu):
    cfg = CONFIGS[2]
    w = make_workload(cfg, n_streams=6, units=140)
    specs = w.streams
    offsets = [s.offset % 37 for s in specs]
    budgets = [s.budget // 4 for s in specs]      # 512 / 1024: evict within 140 units
    ls = Lockstep(cfg, cfg.index, specs, layers_checked=[0, 35], n_layers=36, budgets=budgets,
                  window=cfg.window, tol=BF16_TOL, check_kv_every=25, **_bounds(specs, 1024))
    try:
        ls.run(offsets=offsets)
    finally:
        ls.close()
    _report(ls, "cfg2 varlen")
    assert ls.evictions > 50


EDGE_UNITS = [
    [1] * 17 + [2] + [3] * 64 + [2],          # the largest unit: 64 transcript tokens
    [1] * 17 + [2, 2],                         # empty transcript segment
    [4], [4], [4],                             # decode rows inside a unit
    [3, 3, 3],                                 # a unit without evictable rows
    [1, 2, 3, 2],
] + [[1] * 17 + [2, 3, 3, 3, 2]] * 14


@pytest.mark.parametrize("dtype,tol", [("f32", F32_TOL), ("bf16", BF16_TOL)])
@pytest.mark.parametrize("budget,window", [(0, 0), (0, 2), (40, 1), (120, 3), (10_000, 2)])
def test_edge_streams(gpu, dtype, tol, budget, window):
    cfg = CONFIGS[0]
    spec = tiny_stream(EDGE_UNITS, prefix=5, pos_gap=3)
    # a tight ring: the ring wraps many times over the stream
    ls = Lockstep(cfg, 11, [spec], layers_checked=[0, 1], n_layers=2, budgets=[budget],
                  window=window, tol=tol, dtype=dtype, unit_rows=budget + 200 if budget < 1000 else 700,
                  kept_rows=400, max_step=84)
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"edge {dtype} B{budget} W{window}")


@pytest.mark.parametrize("fused", [False, True])
def test_maximum_step_rows(gpu, fused):
    """A step of the library's maximum size (max_step_rows = 1024): a 1024-row
    prefix at the config-1 head shape (32/8 heads, head dim 128, bf16) gives 4,096
    query rows per KV head, 32 passes of the MFMA kernel over its keys; then units
    that evict down to the budget around the prefix, which is never evicted."""
    cfg = CONFIGS[1]
    spec = tiny_stream([[1] * 17 + [2, 3, 3, 3, 2]] * 8, prefix=1024)
    ls = Lockstep(cfg, 13, [spec], layers_checked=[0], n_layers=1, budgets=[1100], window=1,
                  tol=BF16_TOL, unit_rows=1024 + 400, kept_rows=1100, max_step=1024, fused=fused)
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"max step rows fused={fused}")
    assert ls.evictions > 0


@pytest.mark.parametrize("fused", [False, True])
def test_edge_streams_config1_heads(gpu, fused):
    """The edge units at the config-1 head shape (32/8 heads, head dim 128, bf16):
    the 84-row unit (64 transcript tokens) gives 336 query rows per KV head, three
    passes of the MFMA kernel over the keys; empty segments, decode rows, a unit
    with nothing evictable, a prefix; budget 40, window 1, a wrapping ring."""
    cfg = CONFIGS[1]
    spec = tiny_stream(EDGE_UNITS, prefix=5, pos_gap=3)
    ls = Lockstep(cfg, 12, [spec], layers_checked=[0], n_layers=1, budgets=[40], window=1,
                  tol=BF16_TOL, unit_rows=240, kept_rows=400, max_step=84, fused=fused)
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"edge cfg1 heads fused={fused}")
    assert ls.evictions > 5


# step sizes that put the step's own rows on every kind of tile boundary: after a
# 5-row prefix the cache reaches exactly 64 and 128 rows, a step of exactly one tile,
# single decode rows, 63/65-row steps and 83-row units spanning up to three tiles
TAIL_UNITS = [
    [1] * 59, [1] * 62 + [2, 2], [4], [1] * 60 + [2, 3, 2],
    [1] * 17 + [2] + [3] * 64 + [2], [1, 2], [1] * 61 + [2], [4], [4], [1] * 64,
    [1] * 17 + [2] + [3] * 64 + [2], [1] * 40 + [2, 3, 3, 2], [1] * 64, [1] * 63, [4],
    [1] * 65, [1] * 17 + [2, 3, 2], [1] * 30 + [2, 2],
]


@pytest.mark.parametrize("budget,window,unit_rows", [(10_000, 2, 1024), (300, 1, 400)])
def test_fused_tail_split_layouts(gpu, budget, window, unit_rows):
    """The fused path with planned key splits at the config-1 head shape, on steps
    whose own rows start on, end on or span tile boundaries: a single-stream
    launch gives the tiles holding the step's rows one-tile splits of their own,
    and every step's attention, layout and stored K/V must still match the
    oracle (without eviction, and with a 300-row budget and a wrapping ring)."""
    cfg = CONFIGS[1]
    spec = tiny_stream(TAIL_UNITS, prefix=5)
    ls = Lockstep(cfg, 13, [spec], layers_checked=[0], n_layers=1, budgets=[budget],
                  window=window, tol=BF16_TOL, unit_rows=unit_rows, kept_rows=400, max_step=84,
                  fused=True)
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"fused tail layouts B{budget}")
    assert ls.steps_done == len(TAIL_UNITS) + 1
    if budget < 10_000:
        assert ls.evictions > 3


def test_short_cache_single_partial_tile(gpu):
    # R < 64 keys: one partial tile, masked tail
    cfg = CONFIGS[0]
    spec = tiny_stream([[1, 1, 3]] * 12)
    for dtype, tol in (("f32", F32_TOL), ("bf16", BF16_TOL)):
        ls = Lockstep(cfg, 3, [spec], layers_checked=[0], n_layers=1, budgets=[20], window=1,
                      tol=tol, dtype=dtype, unit_rows=40, kept_rows=40, max_step=3)
        try:
            ls.run()
        finally:
            ls.close()


@pytest.mark.parametrize("splits", ["1", "2", "3", "64"])
def test_forced_key_splits(gpu, splits):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=7).streams[0]
    old = os.environ.get("A2T_SPLITS")
    os.environ["A2T_SPLITS"] = splits
    try:
        for dtype, tol in (("f32", F32_TOL), ("bf16", BF16_TOL)):
            ls = Lockstep(cfg, 7, [spec], layers_checked=[0], n_layers=1, budgets=[cfg.budget],
                          window=cfg.window, tol=tol, dtype=dtype, **_bounds([spec], cfg.budget))
            try:
                ls.run()
            finally:
                ls.close()
    finally:
        if old is None:
            os.environ.pop("A2T_SPLITS", None)
        else:
            os.environ["A2T_SPLITS"] = old


@pytest.mark.parametrize("splits,nq", [("3", 1), ("22", 1), ("64", 1), ("22", 4), ("7", 4), ("22", 5)])
def test_few_query_rows_with_key_splits(gpu, splits, nq):
    """Few query rows per step (the last n_q = 1, 4 or 5 rows of every unit:
    4 to 20 rows per KV head) over a cache split into 3 to 64 key ranges, at
    the config-1 head shape on one stream of 100 units (~2.2 K rows), against
    the fp64 oracle; with 22 splits and one query row the output is
    bit-identical across two runs (fixed-order merge)."""
    cfg = CONFIGS[1]
    spec = make_workload(cfg, units=100).streams[0]
    old = os.environ.get("A2T_SPLITS")
    os.environ["A2T_SPLITS"] = splits
    outs = []
    try:
        for _ in range(2 if splits == "22" and nq == 1 else 1):
            ls = Lockstep(cfg, 1, [spec], layers_checked=[1], n_layers=2, budgets=[10 ** 6],
                          window=cfg.window, tol=BF16_TOL, query_rows=nq, check_kv_every=50,
                          **_bounds([spec], 10 ** 6))
            try:
                ls.run()
            finally:
                ls.close()
            outs.append(np.concatenate([x.ravel() for x in ls.outputs]))
    finally:
        if old is None:
            os.environ.pop("A2T_SPLITS", None)
        else:
            os.environ["A2T_SPLITS"] = old
    if len(outs) == 2:
        assert np.array_equal(outs[0], outs[1])


def test_runs_are_bit_identical(gpu):
    cfg = CONFIGS[1]
    spec = make_workload(cfg, units=60).streams[0]
    outs = []
    for _ in range(2):
        ls = Lockstep(cfg, 1, [spec], layers_checked=[3], n_layers=4, budgets=[600], window=5,
                      tol=BF16_TOL, check_kv_every=1000, **_bounds([spec], 600))
        try:
            ls.run()
        finally:
            ls.close()
        outs.append(np.concatenate([o.reshape(-1) for o in ls.outputs]))
    assert np.array_equal(outs[0], outs[1])


@pytest.mark.parametrize("dtype,tol", [("f32", F32_TOL), ("bf16", BF16_TOL)])
def test_fused_append_attention_config0(gpu, dtype, tol):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=2).streams[0]
    ls = Lockstep(cfg, 2, [spec], layers_checked=[0, 1], n_layers=2, budgets=[cfg.budget],
                  window=cfg.window, tol=tol, dtype=dtype, fused=True, query_rows=7,
                  **_bounds([spec], cfg.budget))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"fused cfg0 {dtype}")
    assert ls.evictions > 40


@pytest.mark.parametrize("splits", ["1", "5", "32"])
def test_fused_append_attention_config1_shape(gpu, splits):
    cfg = CONFIGS[1]
    spec = make_workload(cfg, units=200).streams[0]
    old = os.environ.get("A2T_SPLITS")
    os.environ["A2T_SPLITS"] = splits
    try:
        ls = Lockstep(cfg, cfg.index, [spec], layers_checked=[0, 35], n_layers=36,
                      budgets=[cfg.budget], window=cfg.window, tol=BF16_TOL, check_kv_every=10,
                      fused=True, **_bounds([spec], cfg.budget))
        try:
            ls.run()
        finally:
            ls.close()
    finally:
        if old is None:
            os.environ.pop("A2T_SPLITS", None)
        else:
            os.environ["A2T_SPLITS"] = old
    _report(ls, f"fused cfg1 splits{splits}")
    assert ls.evictions >= 10


def test_fused_edges_and_varlen(gpu):
    cfg = CONFIGS[0]
    spec = tiny_stream(EDGE_UNITS, prefix=5, pos_gap=3)
    ls = Lockstep(cfg, 11, [spec], layers_checked=[0, 1], n_layers=2, budgets=[40], window=1,
                  tol=BF16_TOL, dtype="bf16", unit_rows=240, kept_rows=400, max_step=84, fused=True)
    try:
        ls.run()
    finally:
        ls.close()
    cfg2 = CONFIGS[2]
    w = make_workload(cfg2, n_streams=5, units=110)
    ls = Lockstep(cfg2, cfg2.index, w.streams, layers_checked=[0, 35], n_layers=36,
                  budgets=[s.budget // 4 for s in w.streams], window=cfg2.window, tol=BF16_TOL,
                  check_kv_every=20, fused=True, **_bounds(w.streams, 1024))
    try:
        ls.run(offsets=[s.offset % 23 for s in w.streams])
    finally:
        ls.close()
    _report(ls, "fused varlen")


def test_errors_on_gpu_leave_cache_usable(gpu):
    import torch
    import paper_2609_31224_amd as a2t
    c = a2t.a2t_cache_create(1, 1, 4, 1, 64, a2t.A2T_F32, 8, 8, 8)
    try:
        k = torch.zeros(6, 1, 64, device="cuda")
        a2t.a2t_append(c, 0, [0], [6], k, k, [1] * 6, list(range(6)), [0])
        with pytest.raises(a2t.A2TError) as e:
            a2t.a2t_append(c, 0, [0], [6], k, k, [1] * 6, list(range(6, 12)), [1])
        assert e.value.status == a2t.A2T_ERR_CAPACITY
        with pytest.raises(ValueError):
            a2t.a2t_append(c, 0, [0], [2], k.to(torch.bfloat16), k.to(torch.bfloat16), [1, 1],
                           [6, 7], [1])
        q = torch.randn(6, 4, 64, device="cuda")
        o = torch.empty_like(q)
        a2t.a2t_chunk_attn(c, 0, [0], [6], q, o)
        a2t.a2t_sync(c)
        assert torch.isfinite(o).all()
        n_ev, unmet = a2t.a2t_evict(c, [0], [0], 0)
        assert int(n_ev[0]) == 6 and not unmet[0]
        assert a2t.a2t_stream_info_get(c, 0)["resident"] == 0
    finally:
        a2t.a2t_cache_destroy(c)


# ---- side-channel cadence (Sec. 3.1): per unit a prefill chunk, then one decode step per
# side-channel token; the budget is checked once per unit
def test_cadence_config0_fp32(gpu):
    from synth.streams import make_cadence_workload
    cfg = CONFIGS[0]
    spec = make_cadence_workload(cfg, seed=3).streams[0]
    ls = Lockstep(cfg, 3, [spec], layers_checked=[0], n_layers=1, budgets=[cfg.budget],
                  window=cfg.window, tol=F32_TOL, **_bounds([spec], cfg.budget))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, "cadence cfg0 fp32")
    assert ls.evictions > 10


@pytest.mark.parametrize("fused", [False, True])
def test_cadence_config1_shape_bf16(gpu, fused):
    from synth.streams import make_cadence_workload
    cfg = CONFIGS[1]
    spec = make_cadence_workload(cfg, units=200).streams[0]
    ls = Lockstep(cfg, cfg.index, [spec], layers_checked=[0, 35], n_layers=36, budgets=[2048],
                  window=cfg.window, tol=BF16_TOL, check_kv_every=97, fused=fused,
                  **_bounds([spec], 2048))
    try:
        ls.run()
    finally:
        ls.close()
    _report(ls, f"cadence cfg1 fused={fused}")
    assert ls.evictions > 50


def test_cadence_varlen_batched(gpu):
    from synth.streams import make_cadence_workload
    cfg = CONFIGS[2]
    w = make_cadence_workload(cfg, n_streams=4, units=90)
    specs = w.streams
    offsets = [s.offset % 23 for s in specs]
    ls = Lockstep(cfg, cfg.index, specs, layers_checked=[35], n_layers=36,
                  budgets=[s.budget // 8 for s in specs], window=cfg.window, tol=BF16_TOL,
                  check_kv_every=53, fused=True, **_bounds(specs, 512))
    try:
        ls.run(offsets=offsets)
    finally:
        ls.close()
    _report(ls, "cadence varlen")
    assert ls.evictions > 20
