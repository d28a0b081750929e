"""bench.py's host-side pieces, without a GPU: the one-GPU guard, the byte
formulas behind the roofline and path fractions, the lookup of committed
counter summaries, and the oracle legs (cpu_baseline and its variants) on
small slices of config 0, the CPU-sized case."""
import os
import subprocess
import sys

import pytest

import bench
from synth.streams import CONFIGS, make_cadence_workload, make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_stream_step_limits_are_checked_before_any_gpu_work():
    # more steps than the sessions hold, and a warm-up past the session: clear errors
    for flags, msg in ((["--steps", "100000"], "at most 64 fit"), (["--warmup", "400"], "--warmup <")):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *flags, "--no-cpu-baseline"],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode != 0 and msg in r.stderr and r.stdout == ""


def test_byte_formulas():
    cfg = CONFIGS[1]
    row = 2 * cfg.n_kv_heads * cfg.head_dim * 2            # K and V of one row, bf16: 4 KiB
    assert row == 4096
    assert bench.attn_bytes(4100, 22, cfg) == 4100 * row + 2 * 22 * cfg.n_q_heads * cfg.head_dim * 2
    # a step: attention over every layer, the append (staged K/V read, rows written),
    # the rows copied into the kept region (read + write) and 9 B of metadata per row
    per_layer = bench.attn_bytes(4100, 22, cfg) + 2 * 22 * row + 2 * 3 * row
    assert bench.step_bytes(4100, 22, 3, 4078, cfg) == cfg.n_layers * per_layer + 9 * 4078
    cfg0 = CONFIGS[0]                                       # fp32, 1 KV head, D 64: 512 B rows
    assert bench.attn_bytes(10, 1, cfg0) == 10 * 512 + 2 * 1 * 4 * 64 * 4


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    got = bench.measured_traffic("stream", "attn_tile", [205, 225])
    assert got is not None and 17e6 < got < 40e6
    # other timed units, another kernel or another kernel source: no figure
    assert bench.measured_traffic("stream", "attn_tile", [5, 25]) is None
    assert bench.measured_traffic("stream", "evict") is None
    other = tmp_path / "kernels.hip"
    other.write_text("// not the profiled source\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(other))
    assert bench.measured_traffic("stream", "attn_tile", [205, 225]) is None


def test_roofline_fields():
    kern = {"attn_tile": {"launches": 80, "avg_us": 10.0}}
    r = bench.roofline("attn_tile", kern, 17.2e6, "stream", [205, 225])
    assert abs(r["achieved"] - 1720.0) < 1e-9 and abs(r["frac"] - 0.215) < 1e-12
    assert r["traffic"] is not None and abs(r["traffic_gbps"] - r["traffic"] / 10e-6 / 1e9) < 1e-9
    assert abs(r["traffic_over_alg"] - r["traffic"] / 17.2e6) < 1e-12
    r = bench.roofline("attn_tile", kern, 17.2e6, "stream", [5, 25])   # other units: no counters
    assert r["traffic"] is None and r["traffic_gbps"] is None and r["traffic_over_alg"] is None
    assert bench.roofline("attn_tile", {}, 17.2e6, "stream")["achieved"] is None


def _check_baseline(b, unit):
    assert b["kind"] == "oracle" and b["unit"] == unit
    assert b["value"] > 0 and b["cores"] >= 1 and b["sample"]


def test_oracle_leg_single_stream():
    cfg = CONFIGS[0]
    spec = make_workload(cfg, seed=0).streams[0]
    b = bench.cpu_baseline(cfg, spec, 0, 40, 3, 1)
    _check_baseline(b, "unit-steps/s")
    assert b["units"] == [40, 43]


def test_oracle_leg_batched_slice():
    cfg = CONFIGS[0]
    specs = [make_workload(cfg, seed=s).streams[0] for s in (0, 1)]
    b = bench.cpu_baseline_slice(cfg, 0, [(specs[0], 30), (specs[1], 35)], 2, "unit-steps/s")
    _check_baseline(b, "unit-steps/s")


def test_oracle_leg_cadence_steps():
    cfg = CONFIGS[0]
    spec = make_cadence_workload(cfg, seed=0).streams[0]
    # the steps of units 20 and 21 in the side channel's call pattern
    units, cur = [], []
    for st in spec.steps:
        cur.append(st)
        if st.evict:
            units.append(cur)
            cur = []
    k0 = sum(len(u) for u in units[:20])
    n = len(units[20]) + len(units[21])
    b = bench.cpu_baseline_steps(cfg, 0, spec, k0, n, 2, 1)
    _check_baseline(b, "unit-steps/s")
    assert b["steps"] == [k0, k0 + n] and n > 2
