"""GPU parity of the eviction-rule variants (a2t_evict_rule): per-row
granularity (an ablation of Sec. 3.3's whole-unit rule) and the sink + recent
window of the StreamingLLM comparison (Sec. 2, Table 1), on the same kernels.

Bars as for the paper's rule: eviction counts, budget flags, device layout,
eviction masks and compaction indices bit-exact at every step; compaction
moves every surviving row's bytes unchanged; attention against the fp64
oracle within 1e-4 (fp32 caches) or 2e-2 (bf16 caches)."""
import dataclasses

import numpy as np
import pytest

from synth.streams import CONFIGS, make_workload, tiny_stream
from tests.harness import Lockstep, row_bounds

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


def _bounds(specs):
    return dict(unit_rows=max(row_bounds(s)[0] for s in specs),
                kept_rows=max(row_bounds(s)[1] for s in specs) + 8,
                max_step=max(row_bounds(s)[2] for s in specs))


def _run(ls, name):
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[{name}] steps={ls.steps_done} evictions={ls.evictions} unmet={ls.unmet_steps} "
          f"max_err={ls.max_err:.3e}", flush=True)
    return ls


@pytest.mark.parametrize("seed", [0, 4])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_row_rule_config0(gpu, seed, dtype):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=seed).streams[0]
    ls = Lockstep(cfg, seed, [spec], layers_checked=[0], n_layers=1, budgets=[cfg.budget],
                  window=cfg.window, tol=F32_TOL if dtype == "f32" else BF16_TOL, dtype=dtype,
                  fused=dtype == "bf16", rule="row", **_bounds([spec]))
    _run(ls, f"row cfg0 seed{seed} {dtype}")
    assert ls.evictions > 40


@pytest.mark.parametrize("n_sink,recent", [(4, 120), (0, 64), (1, 1), (30, 10)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sink_recent_rule_config0(gpu, n_sink, recent, dtype):
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=2).streams[0]
    ls = Lockstep(cfg, 2, [spec], layers_checked=[0], n_layers=1, budgets=[n_sink + recent],
                  window=cfg.window, tol=F32_TOL if dtype == "f32" else BF16_TOL, dtype=dtype,
                  fused=dtype == "bf16", rule="sink_recent", n_sink=n_sink, **_bounds([spec]))
    _run(ls, f"sink {n_sink}+{recent} cfg0 {dtype}")
    assert ls.evictions > 40


def test_rules_on_edge_streams(gpu):
    """Prefix rows, decode (RESPONSE) rows under a unit, W = 0, an unmet
    budget, units that end in retained rows."""
    cfg = CONFIGS[0]
    shapes = [
        ([[1, 1, 2, 3, 2]] * 6 + [[4]] * 3 + [[1, 1, 2, 2]] * 3, 10, 1, 2),
        ([[2, 3, 3, 3, 1, 1]] * 6, 7, 0, 1),
        ([[1, 3]] * 9, 3, 0, 0),
    ]
    for rule, n_sink in (("row", 0), ("sink_recent", 2), ("sink_recent", 0)):
        for units, B, W, prefix in shapes:
            spec = tiny_stream(units, prefix=prefix, pos_gap=2)
            ls = Lockstep(cfg, 9, [spec], layers_checked=[0], n_layers=1,
                          budgets=[max(B, n_sink)], window=W, tol=BF16_TOL, dtype="bf16",
                          rule=rule, n_sink=n_sink, unit_rows=64, kept_rows=64, max_step=16)
            _run(ls, f"{rule}/{n_sink} edge B{B} W{W}")
            assert ls.evictions > 0


@pytest.mark.parametrize("rule,budget,n_sink", [("row", 4096, 0), ("sink_recent", 2004, 4)])
def test_rules_config1_shape(gpu, rule, budget, n_sink):
    """The benchmark's shape (36 layers, 32/8 heads, D 128, bf16, fused append
    + attention with planned key splits) under each variant, layers 0 and 35
    checked at every unit."""
    cfg = CONFIGS[1]
    spec = make_workload(cfg, units=230).streams[0]
    ls = Lockstep(cfg, cfg.index, [spec], layers_checked=[0, 35], n_layers=36, budgets=[budget],
                  window=cfg.window, tol=BF16_TOL, check_kv_every=20, fused=True, rule=rule,
                  n_sink=n_sink, **_bounds([spec]))
    _run(ls, f"{rule} cfg1 230 units")
    assert ls.evictions >= 30


@pytest.mark.parametrize("rule,n_sink", [("row", 0), ("sink_recent", 4)])
def test_rules_varlen_batch(gpu, rule, n_sink):
    """Several streams of different lengths and budgets in one cache, evicted
    in one call per step (one launch), config 0's shape in bf16."""
    cfg = dataclasses.replace(CONFIGS[0], n_q_heads=8, n_kv_heads=2)
    w = make_workload(dataclasses.replace(CONFIGS[2], n_layers=1, n_q_heads=8, n_kv_heads=2,
                                          head_dim=64, units=90, min_units=30),
                      seed=2, n_streams=5)
    specs = w.streams
    budgets = [120 + 40 * i for i in range(len(specs))]
    ls = Lockstep(cfg, 2, specs, layers_checked=[0], n_layers=1, budgets=budgets,
                  window=cfg.window, tol=BF16_TOL, dtype="bf16", fused=True, rule=rule,
                  n_sink=n_sink, **_bounds(specs))
    try:
        ls.run(offsets=[s.offset for s in specs])
    finally:
        ls.close()
    print(f"[{rule} varlen] steps={ls.steps_done} evictions={ls.evictions} "
          f"max_err={ls.max_err:.3e}", flush=True)
    assert ls.evictions > 20
