"""GPU parity on seeded random shapes: head counts and groups, head dims, storage
types, stream counts with varied lengths, start offsets and budgets, unit sizes,
windows, the fused and unfused calls, planned and forced key splits and the
rule variants, every step checked against the fp64 oracle (attention within
1e-4 for fp32 caches and 2e-2 for bf16; eviction counts, flags, layouts, masks,
compaction indices and stored K/V exactly).  The draws are fixed, so a failure
names its case and replays."""
import dataclasses
import os

import numpy as np
import pytest

from synth.streams import CONFIGS, make_workload
from tests.harness import Lockstep, row_bounds

pytestmark = pytest.mark.gpu

HEADS = [(4, 1), (8, 2), (16, 4), (32, 8), (8, 8), (12, 3), (24, 3), (6, 3)]


def draw_case(i):
    """Case i's shape and schedule (numpy's seeded generator)."""
    rng = np.random.default_rng(1000 + i)
    hq, hkv = HEADS[int(rng.integers(len(HEADS)))]
    acoustic = int(rng.integers(2, 41))
    cap = int(rng.choice([4, 16, 64]))
    unit_rows = acoustic + 2 + cap
    n_streams = int(rng.choice([1, 2, 3, 5]))
    b_lo = int(rng.integers(0, 4 * unit_rows))
    b_hi = int(rng.integers(b_lo, 12 * unit_rows + 1))
    cfg = dataclasses.replace(
        CONFIGS[0], index=100 + i, n_q_heads=hq, n_kv_heads=hkv,
        head_dim=int(rng.choice([64, 128])), dtype=str(rng.choice(["f32", "bf16"])),
        n_streams=n_streams, units=int(rng.integers(15, 46)), acoustic_rows=acoustic,
        text_mean=float(rng.uniform(0.3, 6.0)), text_cap=cap, window=int(rng.choice([0, 1, 2, 5])),
        varlen=n_streams > 1, min_units=5, budget_choices=(b_lo, b_hi), budget=b_hi)
    return dict(cfg=cfg, fused=bool(rng.integers(2)),
                splits=[None, None, None, "1", "2", "3", "7"][int(rng.integers(7))],
                rule=[None, None, "row", "sink_recent"][int(rng.integers(4))],
                n_sink=int(rng.integers(0, 6)), n_layers=int(rng.choice([1, 1, 2, 3])))


def _env(name, value):
    """Set (or, for None, clear) an environment variable; returns the old value."""
    old = os.environ.get(name)
    if value is None:
        os.environ.pop(name, None)
    else:
        os.environ[name] = value
    return old


@pytest.mark.parametrize("case", range(48))
def test_random_shape(gpu, case):
    _run_case(draw_case(case), f"random {case}")


@pytest.mark.parametrize("case", range(100, 106))
def test_random_shape_forced_valu(gpu, case):
    """bf16 caches on the VALU kernel (A2T_FORCE_VALU, read at cache creation):
    its fp32 key-split partials and the merge that reads them, unfused calls."""
    c = draw_case(case)
    c["cfg"] = dataclasses.replace(c["cfg"], dtype="bf16")
    c["fused"] = False
    old = _env("A2T_FORCE_VALU", "1")
    try:
        _run_case(c, f"forced VALU {case}")
    finally:
        _env("A2T_FORCE_VALU", old)


@pytest.mark.parametrize("case,dtype,fused", [(300, "bf16", True), (301, "bf16", False),
                                             (302, "f32", False)])
def test_odd_partial_blocks(gpu, case, dtype, fused):
    """Three query heads on three KV heads (one query row per head and row), three
    streams and three forced splits: a stream's split partials then take an odd
    number of floats whenever its step has an odd row count, and the next stream's
    partials must still start 16-byte aligned (MFMA kernel's fp16 partials, VALU
    kernel's fp32 ones)."""
    c = draw_case(case)
    c["cfg"] = dataclasses.replace(c["cfg"], n_q_heads=3, n_kv_heads=3, dtype=dtype, n_streams=3,
                                   varlen=True)
    c.update(fused=fused, splits="3", rule=None)
    _run_case(c, f"odd partials {case} {dtype}")


def _run_case(c, label):
    cfg = c["cfg"]
    specs = make_workload(cfg, seed=cfg.index).streams
    budgets = [s.budget for s in specs]
    if c["rule"] == "sink_recent":
        budgets = [max(b, c["n_sink"]) for b in budgets]
    layers = sorted({0, c["n_layers"] - 1})
    old = _env("A2T_SPLITS", c["splits"] or os.environ.get("A2T_SPLITS"))
    try:
        ls = Lockstep(cfg, cfg.index, specs, layers_checked=layers, n_layers=c["n_layers"],
                      budgets=budgets, window=cfg.window,
                      tol=1e-4 if cfg.dtype == "f32" else 2e-2, dtype=cfg.dtype,
                      unit_rows=max(row_bounds(s)[0] for s in specs) + 8,
                      kept_rows=max(row_bounds(s)[1] for s in specs) + 8,
                      max_step=max(row_bounds(s)[2] for s in specs), fused=c["fused"],
                      rule=c["rule"], n_sink=c["n_sink"] if c["rule"] == "sink_recent" else 0)
        try:
            ls.run(offsets=[int(s.offset) for s in specs])
        finally:
            ls.close()
    finally:
        _env("A2T_SPLITS", old)
    print(f"[{label}] heads {cfg.n_q_heads}/{cfg.n_kv_heads} D{cfg.head_dim} {cfg.dtype} "
          f"streams {len(specs)} units<= {cfg.units} rows/unit<= {cfg.max_unit_rows} "
          f"B {budgets} W {cfg.window} fused={c['fused']} splits={c['splits'] or 'planned'} "
          f"rule={c['rule'] or 'unit'} L={c['n_layers']}: steps {ls.steps_done} evictions "
          f"{ls.evictions} max err {ls.max_err:.2e}", flush=True)
    assert ls.steps_done > 0
