"""Benchmark: the streaming KV unit step of a ten-minute session on one MI355X.

One step = one listening unit of one stream through every layer: per layer
an append (rotary keys into the cache) and causal chunk attention of the
unit's rows over the resident cache, then budgeted eviction and compaction
(36 layers, 32 query / 8 KV heads, head dim 128, bf16, budget 4096 rows,
recent window 30 units).  The session runs from unit 0; the first --warmup
units (the cache fills and eviction starts near unit 186) are untimed, the
next --steps units are timed with HIP events on the cache's stream.

Inputs are synthetic and seeded (synth/): stream structure exactly as the
workload defines it; Q/K/V values cycle through a pool of pre-generated unit
tensors already resident in HBM (values do not change the work done).

Prints one JSON line.  See the design doc for the byte accounting.
"""
from __future__ import annotations

import argparse
import ctypes as C
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from synth.streams import CONFIGS, make_workload, step_values  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "stream unit-steps/s (append+attn+evict) and achieved HBM GB/s vs peak"
POOL = 8


def attn_bytes(R: int, n_q: int, cfg) -> int:
    """Algorithmic HBM bytes of one chunk-attention launch for one stream-layer:
    every resident K and V row read once, Q read once, O written once."""
    elt = 2 if cfg.dtype == "bf16" else 4
    kv = R * 2 * cfg.n_kv_heads * cfg.head_dim * elt
    qo = 2 * n_q * cfg.n_q_heads * cfg.head_dim * elt
    return kv + qo


def step_bytes(R_attn: int, n: int, n_moved: int, R_pre: int, cfg) -> int:
    """Algorithmic HBM bytes of one unit step over all layers: attention reads,
    the append (read the staged K/V, write the rows), the kept rows copied by
    compaction (read + write), and the per-row metadata the eviction scans."""
    elt = 2 if cfg.dtype == "bf16" else 4
    row = 2 * cfg.n_kv_heads * cfg.head_dim * elt
    per_layer = attn_bytes(R_attn, n, cfg) + 2 * n * row + 2 * n_moved * row
    return cfg.n_layers * per_layer + 9 * R_pre


def cpu_baseline(cfg, spec, seed, start_unit, sample_units, sample_layers):
    """Time the float64 oracle on a bounded sample: resumed at a steady-state
    unit, ``sample_units`` unit steps over ``sample_layers`` layers, scaled to
    all layers.  The oracle is test infrastructure; only this leg runs it."""
    from oracle.replay import resume
    layers = list(range(sample_layers))
    cache = resume(cfg, seed, spec, cfg.budget, cfg.window, start_unit, layers)
    vals = [step_values(cfg, seed, 0, spec.steps[u].key, spec.steps[u].n, layers)
            for u in range(start_unit, start_unit + sample_units)]
    t0 = time.perf_counter()
    for j, u in enumerate(range(start_unit, start_unit + sample_units)):
        st = spec.steps[u]
        v = vals[j]
        cache.append(st.seg, st.pos, st.unit, {l: v["k"][i] for i, l in enumerate(layers)},
                     {l: v["v"][i] for i, l in enumerate(layers)})
        for i, l in enumerate(layers):
            cache.attention(l, v["q"][i])
        cache.evict(cfg.budget, cfg.window)
    dt = time.perf_counter() - t0
    per_unit_all_layers = dt / sample_units * (cfg.n_layers / sample_layers)
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    return {"value": 1.0 / per_unit_all_layers, "unit": "unit-steps/s", "cores": int(cores),
            "kind": "oracle",
            "sample": f"{sample_units} steady-state units (from unit {start_unit}) x "
                      f"{sample_layers} of {cfg.n_layers} layers, fp64 numpy, scaled to "
                      f"{cfg.n_layers} layers; {dt:.1f} s of CPU work"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-units", type=int, default=6)
    ap.add_argument("--cpu-sample-layers", type=int, default=4)
    ap.add_argument("--profile-steps", type=int, default=100,
                    help="extra timed units with per-kernel HIP events (roofline)")
    ap.add_argument("--unfused", action="store_true",
                    help="per layer a2t_append then a2t_chunk_attn (default: a2t_append_attn)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(the KV step shards by stream or KV head with no exchange; see DESIGN.md).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_31224_amd as a2t

    base = CONFIGS[1]
    total_units = args.warmup + args.steps + args.profile_steps
    cfg = dataclasses.replace(base, units=max(base.units, total_units))
    spec = make_workload(cfg, seed=args.seed, units=total_units).streams[0]
    L, Hq, Hkv, D = cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    max_n = cfg.max_unit_rows
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    # value pool: POOL unit tensors of the largest unit size, all layers, in HBM
    qp = torch.empty(POOL, L, max_n, Hq, D, dtype=torch.bfloat16, device=dev)
    kp = torch.empty(POOL, L, max_n, Hkv, D, dtype=torch.bfloat16, device=dev)
    vp = torch.empty(POOL, L, max_n, Hkv, D, dtype=torch.bfloat16, device=dev)
    for p in range(POOL):
        vals = step_values(cfg, args.seed, 0, 1_000_000 + p, max_n, range(L))
        qp[p] = torch.from_numpy(vals["q"]).to(torch.bfloat16)
        kp[p] = torch.from_numpy(vals["k"]).to(torch.bfloat16)
        vp[p] = torch.from_numpy(vals["v"]).to(torch.bfloat16)
    out = torch.empty(max_n, Hq, D, dtype=torch.bfloat16, device=dev)

    keep_rows = sum(int(np.isin(st.seg, (0, 3, 4)).sum()) for st in spec.steps)
    unit_rows = max(cfg.budget, cfg.window * max_n) + 2 * max_n
    cache = a2t.a2t_cache_create(L, 1, Hq, Hkv, D, a2t.A2T_BF16, unit_rows, keep_rows + 64, max_n,
                                 rope_theta=cfg.rope_theta, attn_scale=cfg.scale, stream=stream)
    lib = a2t.raw_lib()
    h = cache.ptr
    ids = (C.c_int32 * 1)(0)
    budget = (C.c_int32 * 1)(cfg.budget)
    n_ev = (C.c_int32 * 1)()
    unmet = (C.c_uint8 * 1)()
    info = a2t.a2t_stream_info()

    # per-unit marshalled metadata
    metas = []
    for st in spec.steps:
        n = st.n
        metas.append(((C.c_int32 * 1)(n), (C.c_uint8 * n)(*st.seg.tolist()),
                      (C.c_int32 * n)(*st.pos.tolist()), (C.c_int32 * 1)(st.unit)))
    row_stride_q = max_n * Hq * D * 2
    row_stride_kv = max_n * Hkv * D * 2
    q_base, k_base, v_base = qp.data_ptr(), kp.data_ptr(), vp.data_ptr()
    o_ptr = out.data_ptr()
    R_log = []

    def run_unit(u, record=False):
        nrows, seg, pos, unit = metas[u]
        p = u % POOL
        for layer in range(L):
            off_q = (p * L + layer) * row_stride_q
            off_kv = (p * L + layer) * row_stride_kv
            meta = (seg, pos, unit) if layer == 0 else (None, None, None)
            if args.unfused:
                rc = lib.a2t_append(h, layer, 1, ids, nrows, k_base + off_kv, v_base + off_kv, *meta)
                if rc:
                    raise a2t.A2TError(rc, "a2t_append")
                rc = lib.a2t_chunk_attn(h, layer, 1, ids, nrows, q_base + off_q, o_ptr)
                if rc:
                    raise a2t.A2TError(rc, "a2t_chunk_attn")
            else:
                rc = lib.a2t_append_attn(h, layer, 1, ids, nrows, k_base + off_kv, v_base + off_kv,
                                         *meta, nrows, q_base + off_q, o_ptr)
                if rc:
                    raise a2t.A2TError(rc, "a2t_append_attn")
        if record:
            lib.a2t_stream_info_get(h, 0, C.byref(info))
            R_attn = info.resident
        rc = lib.a2t_evict(h, 1, ids, budget, cfg.window, n_ev, unmet)
        if rc:
            raise a2t.A2TError(rc, "a2t_evict")
        if record:
            lib.a2t_stream_info_get(h, 0, C.byref(info))
            R_log.append((R_attn, nrows[0], int(n_ev[0]), info.moved_total))

    for u in range(args.warmup):
        run_unit(u)
    torch.cuda.synchronize()

    # ---- timed region: K unit steps, an event at every unit boundary
    lib.a2t_stream_info_get(h, 0, C.byref(info))
    moved_before = info.moved_total
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    evs[0].record(stream)
    for j in range(args.steps):
        run_unit(args.warmup + j, record=True)
        evs[j + 1].record(stream)
    t_enqueue = time.perf_counter() - t_wall
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    unit_ms = np.array([evs[j].elapsed_time(evs[j + 1]) for j in range(args.steps)])
    total_ms = float(evs[0].elapsed_time(evs[-1]))
    ms_per_step = total_ms / args.steps

    # algorithmic bytes of the timed steps
    moved_prev = moved_before
    tot_bytes = 0
    attn_alg = []
    for (R_attn, n, ev, moved_total) in R_log:
        moved = moved_total - moved_prev
        moved_prev = moved_total
        tot_bytes += step_bytes(R_attn, n, moved, R_attn, cfg)
        attn_alg.append(attn_bytes(R_attn, n, cfg))
    step_gbps = tot_bytes / (total_ms * 1e-3) / 1e9

    # ---- per-kernel timing pass (same stream, HIP events around each launch)
    kern = {}
    prof_units = range(args.warmup + args.steps, args.warmup + args.steps + args.profile_steps)
    a2t.a2t_profile_enable(cache, "")
    R_log.clear()
    for u in prof_units:
        run_unit(u, record=True)
    torch.cuda.synchronize()
    for name in ("attn_mfma", "attn_merge", "append", "step_meta", "evict"):
        n_launch, ms = a2t.a2t_kernel_time(cache, name)
        kern[name] = {"launches": n_launch, "avg_us": (ms * 1e3 / n_launch) if n_launch else None}
    a2t.a2t_profile_enable(cache, None)
    prof_attn_bytes = np.mean([attn_bytes(R, n, cfg) for (R, n, _, _) in R_log]) if R_log else 0.0
    attn_us = kern["attn_mfma"]["avg_us"]
    achieved = prof_attn_bytes / (attn_us * 1e-6) / 1e9 if attn_us else None

    lib.a2t_stream_info_get(h, 0, C.byref(info))
    peak = info.peak
    rows_no_evict = spec.total_rows()
    a2t.a2t_cache_destroy(cache)

    base_line = None
    if not args.no_cpu_baseline:
        start = min(400, max(200, args.warmup))
        base_spec = make_workload(base, seed=args.seed).streams[0]
        base_line = cpu_baseline(base, base_spec, args.seed, start, args.cpu_sample_units,
                                 args.cpu_sample_layers)

    result = {
        "metric": METRIC,
        "value": 1000.0 / ms_per_step,
        "unit": "unit-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "ten-minute single stream: 36 layers, 32 query / 8 KV heads, head dim 128, "
                        "bf16, units of 17 acoustic + 2 delimiter + Poisson(3) transcript rows, "
                        "budget 4096 rows, recent window 30 units",
            "timed_units": [args.warmup, args.warmup + args.steps],
            "calls": "a2t_append + a2t_chunk_attn per layer" if args.unfused
                     else "a2t_append_attn per layer",
            "seed": args.seed,
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "attn_mfma",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS if achieved else None,
            "traffic": None,
            "avg_launch_us": attn_us,
            "alg_bytes_per_launch": prof_attn_bytes,
        },
        "step_hbm": {"achieved_gbps": step_gbps, "frac": step_gbps / HBM_PEAK_GBPS,
                     "alg_bytes_per_step": tot_bytes / max(1, args.steps)},
        "unit_ms": {"mean": float(unit_ms.mean()), "p50": float(np.percentile(unit_ms, 50)),
                    "p99": float(np.percentile(unit_ms, 99)), "max": float(unit_ms.max()),
                    "over_1s": int((unit_ms > 1000).sum())},
        "kernels_us": kern,
        "peak_rows": peak,
        "rows_without_eviction": rows_no_evict,
        "peak_reduction": 1.0 - peak / rows_no_evict,
        "host_wall_s": t_wall,
        "host_enqueue_ms_per_step": t_enqueue * 1e3 / args.steps,
        "cpu_baseline": base_line,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
