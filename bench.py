"""Benchmark: the streaming KV unit step on one MI355X.

Default workload (the headline line): a ten-minute single stream.  One step =
one listening unit of one stream through every layer: per layer an append
(rotary keys into the cache) and causal chunk attention of the unit's rows
over the resident cache, then budgeted eviction and compaction (36 layers,
32 query / 8 KV heads, head dim 128, bf16, budget 4096 rows, recent window
30 units).  The 600-unit session always starts with 200 untimed units that
bring the cache to steady state (it first exceeds the budget near unit 186);
then --warmup more units run untimed and the next --steps units are timed
with HIP events on the cache's stream (warmup + steps <= 400, so every timed
unit lies inside the session, at steady state with eviction running); the
session then runs on untimed to unit 600, whose peak residency gives the
peak-KV reduction.  The oracle's CPU baseline runs the first timed units.

--workload varlen: 32 streams of 60..600 units with random start steps and
budgets of 2048 or 4096 rows, all active streams of a global step batched in
one call per layer (rate = stream unit-steps/s).

--workload decode: 64 streams filled with 600 listening units each, then
single-row response decode steps, all streams batched (rate = stream
decode-steps/s).

--workload cadence: the ten-minute single stream in the side channel's call
pattern: per unit one prefill chunk of the 17 acoustic/structural rows, then
one decode step per side-channel token (opening delimiter, transcript tokens,
closing delimiter), each step a2t_append_attn on every layer, and the budget
check once per unit (rate = stream unit-steps/s).

--workload sweep: the KV-budget ablation (Table 3) on 15 synthetic ten-minute
sessions batched in one cache: for budgets unbounded, 8000, 6000, 4000 and 0
the full hot path over 600 units; End and Peak resident rows per budget and the
step time (rate = stream unit-steps/s at budget 4000).

--workload hour: 16 hour-long sessions (3,600 units, budget 8192, window 60)
and the same sessions with no eviction (the control): the units before the
timed window are filled by all-layers appends, then the full path is timed
for each group; peak resident rows and KV bytes per stream for both
(rate = stream unit-steps/s of the evicting group).

--workload distill: the adaptation objective (Sec. 3.2) on a batch of 16
short utterances x 12 units (~1,340 prediction rows) over a vocabulary of
151,936 teacher tokens + 2 added tokens, bf16 logits: losses and the gradient
with respect to the student logits per evaluation (rate = evaluations/s).

--workload copy: a plain device-to-device copy of 1 GiB (torch's copy
kernel), the reference point for scaling the HBM byte counters of a profile
and for the bandwidth a streaming kernel can reach on this device.

Inputs are synthetic and seeded (synth/): stream structure exactly as the
workload defines it; Q/K/V values come from a pool of pre-generated tensors
already resident in HBM (values do not change the work done).

Prints one JSON line with the rate, the dominant kernel's roofline (its
average dispatch time from kernel-accurate HIP event timestamps over extra
profiled steps, against the algorithmic bytes per launch) and, for the
default workload, the float64 CPU oracle timed on a bounded sample.
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
ATTN_SAMPLE = 9   # ten-minute stream: attention dispatches timed on every 9th layer
POOL = 8
KEEP_SEGS = (0, 3, 4)     # PREFIX, TEXT, RESPONSE: never evicted

METRICS = {
    "stream": ("stream unit-steps/s (append+attn+evict) and achieved HBM GB/s vs peak",
               "unit-steps/s"),
    "varlen": ("stream unit-steps/s (append+attn+evict), varlen batch of 32 streams",
               "unit-steps/s"),
    "decode": ("stream decode-steps/s (append+decode attn+evict), batch of 64 streams",
               "decode-steps/s"),
    "cadence": ("stream unit-steps/s, side-channel cadence (prefill chunk + one decode step "
                "per transcript token, all layers, eviction per unit)", "unit-steps/s"),
    "sweep": ("stream unit-steps/s at budget 4000, 15 ten-minute sessions batched (budget sweep "
              "unbounded/8K/6K/4K/0 reported alongside)", "unit-steps/s"),
    "hour": ("stream unit-steps/s (append+attn+evict), 16 hour-long sessions with eviction "
             "(no-eviction control reported alongside)", "unit-steps/s"),
    "distill": ("objective evaluations/s (masked CE + T^2 KL + group-balanced means and the "
                "student-logit gradient over a 16-utterance batch)", "evaluations/s"),
    "copy": ("device copy bandwidth (read + write bytes per second)", "GB/s"),
    "graph": ("stream unit-steps/s (append+attn+evict), device-planned steps, one HIP graph "
              "replay per unit", "unit-steps/s"),
}
DEFAULTS = {  # warmup, steps, profile steps
    "stream": (3, 397, 0),
    "varlen": (100, 400, 100),
    "decode": (20, 150, 30),
    "cadence": (200, 100, 30),
    "sweep": (0, 600, 0),
    "distill": (5, 40, 20),
    "hour": (0, 100, 20),
    "copy": (3, 20, 0),
    "graph": (5, 20, 0),
}


def attn_bytes(R: int, n_q: int, cfg) -> int:
    """Algorithmic HBM bytes of one stream-layer of attention: every resident
    K and V row read once, Q read once, O written once."""
    elt = 2 if cfg.dtype == "bf16" else 4
    kv = R * 2 * cfg.n_kv_heads * cfg.head_dim * elt
    qo = 2 * n_q * cfg.n_q_heads * cfg.head_dim * elt
    return kv + qo


def step_bytes(R_attn: int, n: int, n_moved: int, R_pre: int, cfg) -> int:
    """Algorithmic HBM bytes of one stream step over all layers: attention
    reads, the append (read the staged K/V, write the rows), the kept rows
    copied by compaction (read + write), and the per-row metadata the
    eviction scans."""
    elt = 2 if cfg.dtype == "bf16" else 4
    row = 2 * cfg.n_kv_heads * cfg.head_dim * elt
    per_layer = attn_bytes(R_attn, n, cfg) + 2 * n * row + 2 * n_moved * row
    return cfg.n_layers * per_layer + 9 * R_pre


def _threads_used() -> int:
    try:
        from threadpoolctl import threadpool_info
        return int(max([p.get("num_threads", 1) for p in threadpool_info()] + [1]))
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def cpu_baseline(cfg, spec, seed, start_unit, sample_units, sample_layers):
    """Time the float64 oracle on a bounded sample: resumed at ``start_unit`` (the
    first unit the GPU leg times), ``sample_units`` unit steps over the first
    ``sample_layers`` layers, scaled to all layers.  The oracle is test
    infrastructure; only this leg runs it."""
    from oracle.replay import resume
    sample_layers = max(1, min(sample_layers, cfg.n_layers))
    layers = list(range(sample_layers))
    cache = resume(cfg, seed, spec, spec.budget, cfg.window, start_unit, layers)
    vals = [step_values(cfg, seed, spec.stream, spec.steps[u].key, spec.steps[u].n, layers)
            for u in range(start_unit, start_unit + sample_units)]
    t0 = time.perf_counter()
    for j, u in enumerate(range(start_unit, start_unit + sample_units)):
        st = spec.steps[u]
        v = vals[j]
        cache.append(st.seg, st.pos, st.unit, {l: v["k"][i] for i, l in enumerate(layers)},
                     {l: v["v"][i] for i, l in enumerate(layers)})
        for i, l in enumerate(layers):
            cache.attention(l, v["q"][i])
        cache.evict(spec.budget, cfg.window)
    dt = time.perf_counter() - t0
    per_unit_all_layers = dt / sample_units * (cfg.n_layers / sample_layers)
    return {"value": 1.0 / per_unit_all_layers, "unit": "unit-steps/s", "cores": _threads_used(),
            "kind": "oracle", "cpu_model": _cpu_model(), "host_cpus": os.cpu_count(),
            "units": [start_unit, start_unit + sample_units],
            "sample": f"units {start_unit}..{start_unit + sample_units - 1} (the first timed units "
                      f"of the GPU leg) x {sample_layers} of {cfg.n_layers} layers, append + "
                      f"attention + eviction, fp64 numpy, scaled to {cfg.n_layers} layers; "
                      f"{dt:.1f} s of CPU work"}


def cpu_baseline_slice(cfg, seed, picks, n_steps, unit):
    """Time the float64 oracle on a fixed slice of a batched workload: for each
    (stream spec, first step) in ``picks`` the oracle is resumed at that step
    and runs ``n_steps`` steps (append, attention of the step's rows on every
    layer, the eviction check), all layers.  Only the oracle's calls are
    timed (not the regeneration of inputs).  Rate = stream steps per second."""
    from oracle.replay import resume
    layers = list(range(cfg.n_layers))
    caches = [resume(cfg, seed, spec, spec.budget, cfg.window, k0, layers) for spec, k0 in picks]
    dt = 0.0
    for j in range(n_steps):
        for (spec, k0), cache in zip(picks, caches):
            st = spec.steps[k0 + j]
            v = step_values(cfg, seed, spec.stream, st.key, st.n, layers)
            t0 = time.perf_counter()
            cache.append(st.seg, st.pos, st.unit, {l: v["k"][i] for i, l in enumerate(layers)},
                         {l: v["v"][i] for i, l in enumerate(layers)})
            for i, l in enumerate(layers):
                cache.attention(l, v["q"][i], st.n)
            if st.evict:
                cache.evict(spec.budget, cfg.window)
            dt += time.perf_counter() - t0
    return {"value": len(picks) * n_steps / dt, "unit": unit, "cores": _threads_used(),
            "kind": "oracle", "cpu_model": _cpu_model(), "host_cpus": os.cpu_count(),
            "sample": f"{n_steps} steady-state steps x {len(picks)} streams "
                      f"({', '.join(f'stream {sp.stream} from step {k0}' for sp, k0 in picks)}) "
                      f"x all {cfg.n_layers} layers, fp64 numpy; {dt:.1f} s of CPU work"}


def cpu_baseline_steps(cfg, seed, spec, k0, n_steps, n_units, sample_layers):
    """The float64 oracle on steps k0 .. k0 + n_steps - 1 of one stream (``n_units``
    units of a workload whose units take several calls), append + attention on
    the first ``sample_layers`` layers and the eviction check where a step
    carries it, scaled to all layers.  Rate = units per second."""
    from oracle.replay import resume
    sample_layers = max(1, min(sample_layers, cfg.n_layers))
    layers = list(range(sample_layers))
    cache = resume(cfg, seed, spec, spec.budget, cfg.window, k0, layers)
    vals = [step_values(cfg, seed, spec.stream, spec.steps[k].key, spec.steps[k].n, layers)
            for k in range(k0, k0 + n_steps)]
    t0 = time.perf_counter()
    for j, k in enumerate(range(k0, k0 + n_steps)):
        st, v = spec.steps[k], vals[j]
        cache.append(st.seg, st.pos, st.unit, {l: v["k"][i] for i, l in enumerate(layers)},
                     {l: v["v"][i] for i, l in enumerate(layers)})
        for i, l in enumerate(layers):
            cache.attention(l, v["q"][i], st.n)
        if st.evict:
            cache.evict(spec.budget, cfg.window)
    dt = time.perf_counter() - t0
    per_unit_all_layers = dt / n_units * (cfg.n_layers / sample_layers)
    return {"value": 1.0 / per_unit_all_layers, "unit": "unit-steps/s", "cores": _threads_used(),
            "kind": "oracle", "cpu_model": _cpu_model(), "host_cpus": os.cpu_count(),
            "steps": [k0, k0 + n_steps],
            "sample": f"{n_units} units ({n_steps} calls, steps {k0}..{k0 + n_steps - 1}, the first "
                      f"timed units of the GPU leg) x {sample_layers} of {cfg.n_layers} layers, "
                      f"append + attention + eviction, fp64 numpy, scaled to {cfg.n_layers} "
                      f"layers; {dt:.1f} s of CPU work"}


class Runner:
    """Shared plumbing: the library, a cache on torch's current stream, and
    per-kernel dispatch timing."""

    KERNELS = ("attn_tile", "attn_valu", "attn_merge", "append", "step_meta", "evict")

    def __init__(self, cfg, n_streams, unit_rows, kept_rows, max_n):
        import torch
        import paper_2609_31224_amd as a2t
        self.torch, self.a2t, self.cfg = torch, a2t, cfg
        self.dev = torch.device("cuda:0")
        torch.cuda.set_device(self.dev)
        self.stream = torch.cuda.current_stream()
        self.cache = a2t.a2t_cache_create(cfg.n_layers, n_streams, cfg.n_q_heads, cfg.n_kv_heads,
                                          cfg.head_dim, a2t.A2T_BF16, unit_rows, kept_rows, max_n,
                                          rope_theta=cfg.rope_theta, attn_scale=cfg.scale,
                                          stream=self.stream)
        self.lib = a2t.raw_lib()
        self.h = self.cache.ptr
        self.info = a2t.a2t_stream_info()

    def check(self, rc, name):
        if rc:
            raise self.a2t.A2TError(rc, name)

    def stream_info(self, s):
        self.lib.a2t_stream_info_get(self.h, s, C.byref(self.info))
        return self.info

    def pool(self, shape, seed):
        """bf16 N(0,1) values from a seeded device generator (timing inputs)."""
        g = self.torch.Generator(device=self.dev)
        g.manual_seed(seed)
        return self.torch.randn(shape, generator=g, device=self.dev,
                                dtype=self.torch.float32).to(self.torch.bfloat16)

    def timed(self, fn, steps, kernel=None, launches=0):
        """Run fn(j) for j < steps with an event at every step boundary; with
        ``kernel`` also that kernel's dispatches timestamped (the library's
        per-dispatch start/stop events on the cache's stream), whose launch
        count and mean duration over the timed steps go to ``self.kern_timed``."""
        torch = self.torch
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        if kernel:
            # event pairs for every timed dispatch made beforehand
            self.a2t.a2t_profile_reserve(self.cache, launches)
            self.a2t.a2t_profile_enable(self.cache, kernel)
        t_wall = time.perf_counter()
        evs[0].record(self.stream)
        for j in range(steps):
            fn(j)
            evs[j + 1].record(self.stream)
        t_enqueue = time.perf_counter() - t_wall
        torch.cuda.synchronize()
        t_wall = time.perf_counter() - t_wall
        step_ms = np.array([evs[j].elapsed_time(evs[j + 1]) for j in range(steps)])
        total_ms = float(evs[0].elapsed_time(evs[-1]))
        self.kern_timed = {}
        if kernel:
            n_launch, ms = self.a2t.a2t_kernel_time(self.cache, kernel)
            self.a2t.a2t_profile_enable(self.cache, None)
            if n_launch:
                self.kern_timed[kernel] = {"launches": n_launch, "avg_us": ms * 1e3 / n_launch}
        return step_ms, total_ms, t_wall, t_enqueue

    def profiled(self, fn, steps):
        """Run fn(j) with every dispatch timestamped; per-kernel averages."""
        self.a2t.a2t_profile_enable(self.cache, "")
        for j in range(steps):
            fn(j)
        self.torch.cuda.synchronize()
        kern = {}
        for name in self.KERNELS:
            n_launch, ms = self.a2t.a2t_kernel_time(self.cache, name)
            if n_launch:
                kern[name] = {"launches": n_launch, "avg_us": ms * 1e3 / n_launch}
        self.a2t.a2t_profile_enable(self.cache, None)
        return kern

    def close(self):
        self.a2t.a2t_cache_destroy(self.cache)


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "attn_traffic.md")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_31224_amd", "csrc", "kernels.hip")


def measured_traffic(workload, kernel, units=None):
    """HBM bytes per launch of ``kernel`` in ``workload`` from the committed
    rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE, scaled by a plain
    copy's readings), or None when the summary was taken on other kernel
    source than the one built here, or (with ``units``) over other steps than
    the ones timed now."""
    import hashlib
    import re
    try:
        text = open(TRAFFIC_PROFILE).read()
        sha = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    m = re.search(r"<!-- traffic-json (.*) -->", text)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != sha:
        return None
    entry = rec.get(workload, {}).get(kernel, {})
    if units is not None and list(entry.get("units", [])) != list(units):
        return None
    return entry.get("bytes")


def roofline(kernel, kern, alg_bytes, workload, units=None):
    """Roofline of ``kernel`` over the timed steps: algorithmic bytes per launch
    over its mean dispatch duration.  The durations come from a second pass
    over the same steps (fresh cache, same inputs) whose dispatches of the
    kernel carry start/stop events: timestamped dispatches slow the host's
    issue rate, so the pass that gives the rate runs without them."""
    us = kern.get(kernel, {}).get("avg_us")
    achieved = alg_bytes / (us * 1e-6) / 1e9 if us else None
    traffic = measured_traffic(workload, kernel, units)
    return {"bound": "hbm", "kernel": kernel, "achieved": achieved, "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS if achieved else None,
            "traffic": traffic, "avg_launch_us": us,
            "launches_timed": kern.get(kernel, {}).get("launches"),
            "alg_bytes_per_launch": alg_bytes,
            "traffic_over_alg": traffic / alg_bytes if traffic else None,
            # the counters' HBM bytes over the same mean dispatch duration
            "traffic_gbps": traffic / (us * 1e-6) / 1e9 if traffic and us else None,
            "timing": "per-dispatch start/stop events on the cache's stream, in a second pass "
                      "over the timed steps"}


def timing_fields(step_ms, total_ms, steps, t_wall, t_enqueue):
    return {"unit_ms": {"mean": float(step_ms.mean()), "p50": float(np.percentile(step_ms, 50)),
                        "p99": float(np.percentile(step_ms, 99)), "max": float(step_ms.max()),
                        "over_1s": int((step_ms > 1000).sum())},
            "host_wall_s": t_wall, "host_enqueue_ms_per_step": t_enqueue * 1e3 / steps}


# ------------------------------------------------------------ ten-minute stream
SESSION_UNITS = 600   # a ten-minute session of one-second units
MAX_SESSIONS = 64     # sessions of one stream workload run (~0.9 GB of cache each)
FILL_UNITS = 200      # the cache first exceeds the 4096-row budget near unit 186

# The paper's own figures for this workload (context, not the target: whole-model
# times on other hardware, which a kernel-only unit step does not compare with).
PAPER_CONTEXT = {
    "peak_kv_reduction": {
        "value": 0.646, "positions_unbounded": 11350, "positions_at_budget": 4020,
        "budget": "4K", "hardware": "1x H100 80GB, batch 1",
        "workload": "LongSpeech ten-minute sessions, the adapted model with vs without eviction",
        "source": "Sec. 4.5, Table 3"},
    "unit_time_ms_at_4k_budget": {
        "mean": 461, "p99": 675, "share_over_1s": 0.0, "hardware": "1x H100 80GB, batch 1",
        "scope": "whole model per one-second unit, side-channel decoding and eviction included",
        "source": "Table 3"},
    "listening_slack_ms_per_unit": {
        "value": 900, "hardware": "the paper's setup (its only stated GPU: 1x H100 80GB)",
        "source": "Sec. 1"},
}


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_stream(args):
    """The ten-minute session (600 units) of one stream.  Units 0 .. FILL_UNITS-1
    bring the cache to steady state untimed (eviction starts near unit 186), then
    --warmup more units run untimed and the next --steps units are timed; the
    session then runs on, untimed, to unit 600, whose peak residency gives the
    peak-KV reduction.  Every timed unit lies inside the session.  More --steps than
    one session holds after the fill and the warm-up run over several sessions of
    the same stream (independent streams of one cache, each brought to steady
    state before the timed region): session s times units FILL_UNITS + --warmup
    onward after session s - 1 has timed all of its own."""
    cfg = CONFIGS[1]
    first = FILL_UNITS + args.warmup
    span = SESSION_UNITS - first             # timed units one session holds
    if args.warmup < 0 or args.steps < 1 or span < 1:
        raise SystemExit(f"--steps >= 1 and 0 <= --warmup < {SESSION_UNITS - FILL_UNITS}")
    n_sess = -(-args.steps // span)
    if n_sess > MAX_SESSIONS:
        raise SystemExit(f"--steps {args.steps} needs {n_sess} sessions of {span} timed units; "
                         f"at most {MAX_SESSIONS} fit (--steps <= {MAX_SESSIONS * span})")
    last = first + min(args.steps, span)     # session 0's timed units are [first, last)
    spec = make_workload(cfg, seed=args.seed).streams[0]
    assert len(spec.steps) == SESSION_UNITS
    L, Hq, Hkv, D = cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    max_n = cfg.max_unit_rows
    keep_rows = sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in spec.steps)
    unit_rows = max(cfg.budget, cfg.window * max_n) + 2 * max_n
    # value pool: POOL unit tensors of the largest unit size, all layers
    pool_vals = [step_values(cfg, args.seed, 0, 1_000_000 + p, max_n, range(L)) for p in range(POOL)]
    metas = []
    for st in spec.steps:
        n = st.n
        metas.append(((C.c_int32 * 1)(n), (C.c_uint8 * n)(*st.seg.tolist()),
                      (C.c_int32 * n)(*st.pos.tolist()), (C.c_int32 * 1)(st.unit)))

    def session(mode):
        """One pass over the session.  mode None: the rate; "attn": the attention
        dispatches of every ATTN_SAMPLE-th layer of the timed units carry start/stop
        events (timing one layer in nine changes the unit time by ~3 %, all of them
        by ~40 %); "all": every dispatch of the timed units is timestamped (the
        per-kernel averages)."""
        r = Runner(cfg, n_sess, unit_rows, keep_rows + 64, max_n)
        torch, lib, h = r.torch, r.lib, r.h
        qp = torch.empty(POOL, L, max_n, Hq, D, dtype=torch.bfloat16, device=r.dev)
        kp = torch.empty(POOL, L, max_n, Hkv, D, dtype=torch.bfloat16, device=r.dev)
        vp = torch.empty(POOL, L, max_n, Hkv, D, dtype=torch.bfloat16, device=r.dev)
        for p, vals in enumerate(pool_vals):
            qp[p] = torch.from_numpy(vals["q"]).to(torch.bfloat16)
            kp[p] = torch.from_numpy(vals["k"]).to(torch.bfloat16)
            vp[p] = torch.from_numpy(vals["v"]).to(torch.bfloat16)
        out = torch.empty(max_n, Hq, D, dtype=torch.bfloat16, device=r.dev)
        sess_ids = [(C.c_int32 * 1)(s) for s in range(n_sess)]
        budget = (C.c_int32 * 1)(cfg.budget)
        n_ev = (C.c_int32 * 1)()
        unmet = (C.c_uint8 * 1)()
        row_stride_q = max_n * Hq * D * 2
        row_stride_kv = max_n * Hkv * D * 2
        q_base, k_base, v_base = qp.data_ptr(), kp.data_ptr(), vp.data_ptr()
        o_ptr = out.data_ptr()
        R_log = []

        def run_unit(u, sess=0, record=False):
            ids = sess_ids[sess]
            nrows, seg, pos, unit = metas[u]
            p = u % POOL
            for layer in range(L):
                off_q = (p * L + layer) * row_stride_q
                off_kv = (p * L + layer) * row_stride_kv
                meta = (seg, pos, unit) if layer == 0 else (None, None, None)
                timed_layer = mode == "attn" and record and layer % ATTN_SAMPLE == 0
                if timed_layer:
                    r.a2t.a2t_profile_enable(r.cache, "attn_tile")
                if args.unfused:
                    r.check(lib.a2t_append(h, layer, 1, ids, nrows, k_base + off_kv,
                                           v_base + off_kv, *meta), "a2t_append")
                    r.check(lib.a2t_chunk_attn(h, layer, 1, ids, nrows, q_base + off_q, o_ptr),
                            "a2t_chunk_attn")
                else:
                    r.check(lib.a2t_append_attn(h, layer, 1, ids, nrows, k_base + off_kv,
                                                v_base + off_kv, *meta, nrows, q_base + off_q,
                                                o_ptr), "a2t_append_attn")
                if timed_layer:
                    r.a2t.a2t_profile_enable(r.cache, None)
            if record:
                info = r.stream_info(sess)
                R_attn, moved0 = info.resident, info.moved_total
            r.check(lib.a2t_evict(h, 1, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")
            if record:
                R_log.append((R_attn, nrows[0], int(n_ev[0]),
                              r.stream_info(sess).moved_total - moved0))

        def timed_unit(j):
            run_unit(first + j % span, j // span, record=True)

        for sess in range(n_sess):
            for u in range(first):
                run_unit(u, sess)
        res = {}
        if mode == "all":
            res["kern"] = r.profiled(timed_unit, args.steps)
        else:
            if mode == "attn":
                r.a2t.a2t_profile_reserve(r.cache,
                                          args.steps * ((L + ATTN_SAMPLE - 1) // ATTN_SAMPLE))
            res["step_ms"], res["total_ms"], res["t_wall"], res["t_enq"] = r.timed(
                timed_unit, args.steps)
        res["R_log"] = list(R_log)
        res["kern_timed"] = {}
        if mode == "attn":
            n_launch, ms = r.a2t.a2t_kernel_time(r.cache, "attn_tile")
            if n_launch:
                res["kern_timed"]["attn_tile"] = {"launches": n_launch,
                                                  "avg_us": ms * 1e3 / n_launch}
        if mode is None:
            for u in range(last, SESSION_UNITS):
                run_unit(u)
            r.torch.cuda.synchronize()
            res["peak"] = r.stream_info(0).peak
            res["end_rows"] = r.stream_info(0).resident
        r.close()
        return res

    clean = session(None)     # the rate, then the rest of the session for its peak
    timed = session("attn")   # the same units again, attention dispatches timestamped
    prof = session("all")     # and once more with every dispatch timestamped
    R_log = clean["R_log"]
    total_ms = clean["total_ms"]
    ms_per_step = total_ms / args.steps
    # algorithmic bytes of the timed units
    tot_bytes, moved_sum = 0, 0
    for (R_attn, n, _, moved) in R_log:
        tot_bytes += step_bytes(R_attn, n, moved, R_attn, cfg)
        moved_sum += moved
    step_gbps = tot_bytes / (total_ms * 1e-3) / 1e9
    if args.jsonl:
        # one record per timed unit: residency, rows appended / evicted / moved into the
        # kept region, algorithmic bytes and the unit's GPU time
        with open(args.jsonl, "w") as f:
            for j, (R_attn, n, n_ev, moved) in enumerate(R_log):
                f.write(json.dumps({"unit": first + j % span, "session": j // span,
                                    "resident_pre": R_attn, "appended": n,
                                    "evicted": n_ev, "resident_post": R_attn - n_ev,
                                    "moved": moved,
                                    "alg_bytes": step_bytes(R_attn, n, moved, R_attn, cfg),
                                    "ms": float(clean["step_ms"][j])}) + "\n")
    timed_attn_bytes = float(np.mean([attn_bytes(R, n, cfg) for (R, n, _, _) in timed["R_log"]]))
    peak = clean["peak"]
    rows_no_evict = spec.total_rows()
    resident = [R for (R, _, _, _) in R_log]
    evicted = [e for (_, _, e, _) in R_log]

    base_line = None
    if not args.no_cpu_baseline:
        k = max(1, min(args.steps, args.cpu_sample_units))
        base_line = cpu_baseline(cfg, spec, args.seed, first, k, args.cpu_sample_layers)
    # the committed counter summary covers one session's units [205, 225)
    traffic_units = [first, last] if n_sess == 1 else [first, last, n_sess]
    res = {
        "value": 1000.0 / ms_per_step,
        "ms_per_step": ms_per_step,
        "config": {
            "workload": "ten-minute single stream: 36 layers, 32 query / 8 KV heads, head dim 128, "
                        "bf16, units of 17 acoustic + 2 delimiter + Poisson(3) transcript rows, "
                        "budget 4096 rows, recent window 30 units",
            "session_units": SESSION_UNITS,
            "fill_units": FILL_UNITS,
            "timed_units": [first, last],
            "sessions": n_sess,
            "calls": "a2t_append + a2t_chunk_attn per layer" if args.unfused
                     else "a2t_append_attn per layer",
            "seed": args.seed,
        },
        "timed_window": {
            "units": [first, last],
            "sessions": n_sess,
            "resident_rows_before_eviction": [int(min(resident)), int(max(resident))],
            "evicting_units": int(sum(1 for e in evicted if e > 0)),
            "rows_evicted": int(sum(evicted)),
            "rows_moved_to_kept": int(moved_sum),
        },
        "roofline": dict(roofline("attn_tile", timed["kern_timed"], timed_attn_bytes, "stream",
                                  traffic_units),
                         timing=f"per-dispatch start/stop events on the cache's stream, in a second "
                                f"pass over the timed units, on every {ATTN_SAMPLE}th layer"),
        "step_hbm": {"achieved_gbps": step_gbps, "frac": step_gbps / HBM_PEAK_GBPS,
                     "alg_bytes_per_step": tot_bytes / max(1, args.steps)},
        **timing_fields(clean["step_ms"], total_ms, args.steps, clean["t_wall"], clean["t_enq"]),
        "timed_pass_ms_per_step": timed["total_ms"] / args.steps,
        "kernels_us": prof["kern"],
        "kernels_us_steps": [first, last],
        "peak_rows": peak,
        "end_rows": clean["end_rows"],
        "rows_without_eviction": rows_no_evict,
        "peak_reduction": 1.0 - peak / rows_no_evict,
        "peak_reduction_units": SESSION_UNITS,
        "paper_context": PAPER_CONTEXT,
        "cpu_baseline": base_line,
    }
    return res

# ------------------------------------------------------- device-planned graph replay
def run_graph(args):
    """The ten-minute stream through the device-planned calls (a2t_dev_*): the
    device opens each unit from metadata in device memory, plans its key splits
    and the eviction.  Eight HIP graphs (one per slot of the pre-generated
    value pool) each hold a whole unit: a cursor copies the next unit's row
    metadata from a device-resident table into the step's buffers and advances
    itself, then the open, the 36 layers' append + attention and the eviction.
    The host replays one graph per unit.  The same 600-unit session runs
    twice, once replaying the graphs and once issuing the same calls eagerly;
    units FILL_UNITS + --warmup onward are timed for --steps units in each."""
    import torch
    import paper_2609_31224_amd as a2t
    cfg = CONFIGS[1]
    first = FILL_UNITS + args.warmup
    if args.warmup < 0 or args.steps < 1 or first + args.steps > SESSION_UNITS:
        raise SystemExit(f"--warmup + --steps <= {SESSION_UNITS - FILL_UNITS}")
    last = first + args.steps
    spec = make_workload(cfg, seed=args.seed).streams[0]
    L, Hq, Hkv, D, MS = cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.max_unit_rows
    keep_rows = sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in spec.steps)
    unit_rows = max(cfg.budget, cfg.window * MS) + 2 * MS
    n_units = len(spec.steps)
    meta = np.zeros((n_units, 2 + MS), np.int32)   # n_rows, unit id, positions
    segs = np.zeros((n_units, MS), np.uint8)
    for u, st in enumerate(spec.steps):
        meta[u, 0], meta[u, 1] = st.n, st.unit
        meta[u, 2:2 + st.n] = st.pos
        segs[u, :st.n] = st.seg
    side = torch.cuda.Stream()

    def session(replay):
        with torch.cuda.stream(side):
            r = Runner(cfg, 1, unit_rows, keep_rows + 64, MS)
            dev = r.dev
            qp = r.pool((POOL, L, MS, Hq, D), args.seed)
            kp = r.pool((POOL, L, MS, Hkv, D), args.seed + 1)
            vp = r.pool((POOL, L, MS, Hkv, D), args.seed + 2)
            out = torch.empty(L, MS, Hq, D, dtype=torch.bfloat16, device=dev)
            table = torch.from_numpy(meta).to(dev)
            seg_table = torch.from_numpy(segs).to(dev)
            cur = torch.zeros(2 + MS, dtype=torch.int32, device=dev)
            cur_seg = torch.zeros(MS, dtype=torch.uint8, device=dev)
            cursor = torch.zeros(1, dtype=torch.int64, device=dev)
            budget = torch.tensor([cfg.budget], dtype=torch.int32, device=dev)
            c = r.cache

            def unit_calls(p):
                cur.copy_(table.index_select(0, cursor).view(-1))
                cur_seg.copy_(seg_table.index_select(0, cursor).view(-1))
                cursor.add_(1)
                a2t.a2t_dev_open(c, [0], cur[0:1], cur[1:2], cur_seg, cur[2:])
                for layer in range(L):
                    a2t.a2t_dev_append_attn(c, layer, kp[p, layer], vp[p, layer], qp[p, layer],
                                            out[layer])
                a2t.a2t_dev_evict(c, budget, cfg.window)

            a2t.a2t_dev_begin(c)
            graphs = []
            if replay:
                for p in range(POOL):
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=side):
                        unit_calls(p)
                    graphs.append(g)
                cursor.zero_()
            run_unit = (lambda u: graphs[u % POOL].replay()) if replay else \
                (lambda u: unit_calls(u % POOL))
            for u in range(first):
                run_unit(u)
            step_ms, total_ms, t_wall, t_enq = r.timed(lambda j: run_unit(first + j), args.steps)
            for u in range(last, SESSION_UNITS):
                run_unit(u)
            a2t.a2t_dev_end(c)
            info = r.stream_info(0)
            res = {"step_ms": step_ms, "total_ms": total_ms, "t_wall": t_wall, "t_enq": t_enq,
                   "peak": info.peak, "end": info.resident}
            r.close()
            return res

    graph = session(True)
    eager = session(False)
    ms_per_step = graph["total_ms"] / args.steps
    base_line = None
    if not args.no_cpu_baseline:
        k = max(1, min(args.steps, args.cpu_sample_units))
        base_line = cpu_baseline(cfg, spec, args.seed, first, k, args.cpu_sample_layers)
    return {
        "value": 1000.0 / ms_per_step,
        "ms_per_step": ms_per_step,
        "config": {
            "workload": "ten-minute single stream: 36 layers, 32 query / 8 KV heads, head dim 128, "
                        "bf16, units of 17 acoustic + 2 delimiter + Poisson(3) transcript rows, "
                        "budget 4096 rows, recent window 30 units",
            "session_units": SESSION_UNITS, "fill_units": FILL_UNITS, "timed_units": [first, last],
            "calls": "per unit one HIP graph replay: metadata cursor (3 small copy/add kernels), "
                     "a2t_dev_open, a2t_dev_append_attn x 36, a2t_dev_evict",
            "seed": args.seed,
        },
        **timing_fields(graph["step_ms"], graph["total_ms"], args.steps, graph["t_wall"],
                        graph["t_enq"]),
        "eager_device_planned": {"value": 1000.0 * args.steps / eager["total_ms"],
                                 "ms_per_step": eager["total_ms"] / args.steps,
                                 "host_enqueue_ms_per_step": eager["t_enq"] * 1e3 / args.steps},
        "peak_rows": graph["peak"], "end_rows": graph["end"],
        "same_session_end": graph["end"] == eager["end"] and graph["peak"] == eager["peak"],
        "roofline": None,
        "cpu_baseline": base_line,
    }


# ------------------------------------------------------------------- varlen batch
def _varlen_session(args, kernel):
    cfg = CONFIGS[2]
    w = make_workload(cfg, seed=args.seed)
    specs = w.streams
    S, L, Hq, Hkv, D = len(specs), cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = w.global_steps()
    max_n = cfg.max_unit_rows
    keep_rows = max(sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in s.steps) for s in specs)
    unit_rows = max(max(s.budget for s in specs), cfg.window * max_n) + 2 * max_n
    r = Runner(cfg, S, unit_rows, keep_rows + 64, max_n)
    torch, lib, h = r.torch, r.lib, r.h

    # per global step: the active streams and their marshalled metadata
    steps = []
    for t in range(T):
        act = [(i, s.steps[t - s.offset]) for i, s in enumerate(specs)
               if 0 <= t - s.offset < len(s.steps)]
        if not act:
            steps.append(None)
            continue
        n = len(act)
        seg = np.concatenate([st.seg for _, st in act])
        pos = np.concatenate([st.pos for _, st in act])
        steps.append(dict(
            n=n, rows=[st.n for _, st in act], ids=(C.c_int32 * n)(*[i for i, _ in act]),
            nrows=(C.c_int32 * n)(*[st.n for _, st in act]),
            seg=(C.c_uint8 * len(seg))(*seg.tolist()), pos=(C.c_int32 * len(pos))(*pos.tolist()),
            unit=(C.c_int32 * n)(*[st.unit for _, st in act]),
            budget=(C.c_int32 * n)(*[specs[i].budget for i, _ in act]),
            n_ev=(C.c_int32 * n)(), unmet=(C.c_uint8 * n)()))
    max_rows = max(sum(s["rows"]) for s in steps if s)
    P = 2
    qp = r.pool((P, L, max_rows, Hq, D), args.seed)
    kp = r.pool((P, L, max_rows, Hkv, D), args.seed + 1)
    vp = r.pool((P, L, max_rows, Hkv, D), args.seed + 2)
    out = torch.empty(max_rows, Hq, D, dtype=torch.bfloat16, device=r.dev)
    sq, skv = max_rows * Hq * D * 2, max_rows * Hkv * D * 2
    R_log = []

    def run_step(t, record=False):
        st = steps[t]
        if st is None:
            return
        p = t % P
        for layer in range(L):
            oq, okv = (p * L + layer) * sq, (p * L + layer) * skv
            meta = (st["seg"], st["pos"], st["unit"]) if layer == 0 else (None, None, None)
            r.check(lib.a2t_append_attn(h, layer, st["n"], st["ids"], st["nrows"],
                                        kp.data_ptr() + okv, vp.data_ptr() + okv, *meta,
                                        st["nrows"], qp.data_ptr() + oq, out.data_ptr()),
                    "a2t_append_attn")
        if record:
            R_log.append(sum(attn_bytes(r.stream_info(i).resident, n, cfg)
                             for i, n in zip(st["ids"], st["rows"])))
        r.check(lib.a2t_evict(h, st["n"], st["ids"], st["budget"], cfg.window, st["n_ev"],
                              st["unmet"]), "a2t_evict")

    warm = min(args.warmup, T)
    timed_steps = max(0, min(args.steps, T - warm))
    prof_steps = max(0, min(args.profile_steps, T - warm - timed_steps))
    for t in range(warm):
        run_step(t)
    n_calls = sum(1 for t in range(warm, warm + timed_steps) if steps[t])
    step_ms, total_ms, t_wall, t_enq = r.timed(lambda j: run_step(warm + j, record=True),
                                               timed_steps, kernel=kernel,
                                               launches=n_calls * L * 2)
    stream_steps = sum(steps[t]["n"] for t in range(warm, warm + timed_steps) if steps[t])
    # one attention launch per layer covers every active stream of the step
    alg = float(np.mean(R_log)) if R_log else 0.0
    kern_timed = r.kern_timed
    p0 = warm + timed_steps
    kern = r.profiled(lambda j: run_step(p0 + j), prof_steps)
    kern_steps = [p0, p0 + prof_steps]
    unmet_streams = sum(1 for i in range(S) if r.stream_info(i).budget_unmet)
    r.close()
    base_line = None
    if kernel is None and not args.no_cpu_baseline:
        # 10 steps of 4 streams running at the first timed global step (longest histories)
        cand = [s for s in specs if 0 <= warm - s.offset and warm - s.offset + 10 <= len(s.steps)]
        cand.sort(key=lambda s: -(warm - s.offset))
        picks = [(s, warm - s.offset) for s in cand[:4]]
        if picks:
            base_line = cpu_baseline_slice(cfg, args.seed, picks, 10, "unit-steps/s")
    return {
        "value": stream_steps / (total_ms * 1e-3),
        "ms_per_step": total_ms / max(1, timed_steps),
        "config": {
            "workload": "varlen batch: 32 streams of U{60..600} units at random start steps in "
                        "a 600-step schedule, budgets {2048, 4096} rows, recent window 30 units; "
                        "36 layers, 32 query / 8 KV heads, head dim 128, bf16",
            "timed_global_steps": [warm, warm + timed_steps],
            "stream_steps_timed": stream_steps,
            "mean_active_streams": stream_steps / max(1, timed_steps),
            "calls": "a2t_append_attn per layer over all active streams, one a2t_evict per step",
            "seed": args.seed,
        },
        "roofline": roofline("attn_tile", kern_timed, alg, "varlen"),
        **timing_fields(step_ms, total_ms, max(1, timed_steps), t_wall, t_enq),
        "kernels_us": kern,
        "kernels_us_steps": kern_steps,
        "streams_budget_unmet_at_end": unmet_streams,
        "cpu_baseline": base_line,
    }


# ------------------------------------------------------------------- decode batch
def _decode_session(args, kernel):
    cfg = CONFIGS[3]
    w = make_workload(cfg, seed=args.seed)
    specs = w.streams
    S, L, Hq, Hkv, D = len(specs), cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    n_units = specs[0].n_units
    n_dec = len(specs[0].steps) - n_units
    max_n = cfg.max_unit_rows
    keep_rows = max(sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in s.steps) for s in specs)
    unit_rows = max(cfg.budget, cfg.window * max_n) + 2 * max_n + n_dec
    r = Runner(cfg, S, unit_rows, keep_rows + 64, max_n)
    torch, lib, h = r.torch, r.lib, r.h
    ids = (C.c_int32 * S)(*range(S))
    budget = (C.c_int32 * S)(*[cfg.budget] * S)
    n_ev, unmet = (C.c_int32 * S)(), (C.c_uint8 * S)()

    # fill: every listening unit of every stream, all layers in one append call
    fill_rows = max(sum(s.steps[u].n for s in specs) for u in range(n_units))
    kf = r.pool((L, fill_rows, Hkv, D), args.seed + 10)
    vf = r.pool((L, fill_rows, Hkv, D), args.seed + 11)
    for u in range(n_units):
        seg = np.concatenate([s.steps[u].seg for s in specs])
        pos = np.concatenate([s.steps[u].pos for s in specs])
        nrows = (C.c_int32 * S)(*[s.steps[u].n for s in specs])
        unit = (C.c_int32 * S)(*[s.steps[u].unit for s in specs])
        # the all-layers input is packed [L][sum n][Hkv][D]: re-pack for this unit's row count
        tot = int(sum(nrows))
        kk = kf[:, :tot].contiguous() if tot < fill_rows else kf
        vv = vf[:, :tot].contiguous() if tot < fill_rows else vf
        r.check(lib.a2t_append(h, -1, S, ids, nrows, kk.data_ptr(), vv.data_ptr(),
                               (C.c_uint8 * tot)(*seg.tolist()), (C.c_int32 * tot)(*pos.tolist()),
                               unit), "a2t_append")
        r.check(lib.a2t_evict(h, S, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")
    torch.cuda.synchronize()

    # decode steps: one RESPONSE row per stream
    dmeta = []
    for d in range(n_dec):
        st = [s.steps[n_units + d] for s in specs]
        dmeta.append(((C.c_uint8 * S)(*[int(x.seg[0]) for x in st]),
                      (C.c_int32 * S)(*[int(x.pos[0]) for x in st]),
                      (C.c_int32 * S)(*[x.unit for x in st])))
    ones = (C.c_int32 * S)(*[1] * S)
    P = 4
    qp = r.pool((P, L, S, Hq, D), args.seed)
    kp = r.pool((P, L, S, Hkv, D), args.seed + 1)
    vp = r.pool((P, L, S, Hkv, D), args.seed + 2)
    out = torch.empty(S, Hq, D, dtype=torch.bfloat16, device=r.dev)
    sq, skv = S * Hq * D * 2, S * Hkv * D * 2
    fused = args.decode_call == "fused"
    R_log = []

    def run_step(d, record=False):
        seg, pos, unit = dmeta[d]
        p = d % P
        for layer in range(L):
            oq, okv = (p * L + layer) * sq, (p * L + layer) * skv
            meta = (seg, pos, unit) if layer == 0 else (None, None, None)
            if fused:
                r.check(lib.a2t_append_attn(h, layer, S, ids, ones, kp.data_ptr() + okv,
                                            vp.data_ptr() + okv, *meta, ones, qp.data_ptr() + oq,
                                            out.data_ptr()), "a2t_append_attn")
            else:
                r.check(lib.a2t_append(h, layer, S, ids, ones, kp.data_ptr() + okv,
                                       vp.data_ptr() + okv, *meta), "a2t_append")
                r.check(lib.a2t_decode_attn(h, layer, S, ids, qp.data_ptr() + oq, out.data_ptr()),
                        "a2t_decode_attn")
        if record:
            R_log.append(sum(attn_bytes(r.stream_info(i).resident, 1, cfg) for i in range(S)))
        r.check(lib.a2t_evict(h, S, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")

    warm = min(args.warmup, n_dec)
    timed_steps = max(0, min(args.steps, n_dec - warm))
    prof_steps = max(0, min(args.profile_steps, n_dec - warm - timed_steps))
    for d in range(warm):
        run_step(d)
    kname = "attn_valu" if os.environ.get("A2T_FORCE_VALU", "0") not in ("", "0") else "attn_tile"
    step_ms, total_ms, t_wall, t_enq = r.timed(lambda j: run_step(warm + j, record=True),
                                               timed_steps, kernel=kernel and kname,
                                               launches=timed_steps * L)
    alg = float(np.mean(R_log)) if R_log else 0.0
    kern_timed = r.kern_timed
    p0 = warm + timed_steps
    kern = r.profiled(lambda j: run_step(p0 + j), prof_steps)
    kern_steps = [p0, p0 + prof_steps]
    mean_R = float(np.mean([r.stream_info(i).resident for i in range(S)]))
    r.close()
    base_line = None
    if kernel is None and not args.no_cpu_baseline and warm + 10 <= n_dec:
        # 10 decode steps of 4 streams from the first timed decode step
        picks = [(specs[i], n_units + warm) for i in range(min(4, S))]
        base_line = cpu_baseline_slice(cfg, args.seed, picks, 10, "decode-steps/s")
    return {
        "value": S * timed_steps / (total_ms * 1e-3),
        "ms_per_step": total_ms / max(1, timed_steps),
        "config": {
            "workload": "decode batch: 64 streams, each filled with 600 listening units "
                        "(budget 4096 rows, recent window 30 units), then single-row response "
                        "decode steps; 36 layers, 32 query / 8 KV heads, head dim 128, bf16",
            "timed_decode_steps": [warm, warm + timed_steps],
            "calls": ("a2t_append_attn (n_q = 1)" if fused else "a2t_append + a2t_decode_attn")
                     + " per layer over 64 streams, one a2t_evict per step",
            "mean_resident_rows_at_end": mean_R,
            "seed": args.seed,
        },
        "roofline": roofline(kname, kern_timed, alg, "decode"),
        **timing_fields(step_ms, total_ms, max(1, timed_steps), t_wall, t_enq),
        "kernels_us": kern,
        "kernels_us_steps": kern_steps,
        "cpu_baseline": base_line,
    }


# ------------------------------------------------------------------- side-channel cadence
def _cadence_session(args, kernel):
    from synth.streams import make_cadence_workload
    base = CONFIGS[1]
    total_units = args.warmup + args.steps + args.profile_steps
    cfg = dataclasses.replace(base, units=max(base.units, total_units))
    spec = make_cadence_workload(cfg, seed=args.seed, units=total_units).streams[0]
    L, Hq, Hkv, D = cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    max_n = cfg.max_unit_rows
    keep_rows = sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in spec.steps)
    unit_rows = max(cfg.budget, cfg.window * max_n) + 2 * max_n
    r = Runner(cfg, 1, unit_rows, keep_rows + 64, max_n)
    torch, lib, h = r.torch, r.lib, r.h
    qp = r.pool((POOL, L, max_n, Hq, D), args.seed)
    kp = r.pool((POOL, L, max_n, Hkv, D), args.seed + 1)
    vp = r.pool((POOL, L, max_n, Hkv, D), args.seed + 2)
    out = torch.empty(max_n, Hq, D, dtype=torch.bfloat16, device=r.dev)
    ids = (C.c_int32 * 1)(0)
    budget = (C.c_int32 * 1)(cfg.budget)
    n_ev, unmet = (C.c_int32 * 1)(), (C.c_uint8 * 1)()
    # the steps of each unit, marshalled
    units = []
    cur = []
    for st in spec.steps:
        cur.append(((C.c_int32 * 1)(st.n), (C.c_uint8 * st.n)(*st.seg.tolist()),
                    (C.c_int32 * st.n)(*st.pos.tolist()), (C.c_int32 * 1)(st.unit)))
        if st.evict:
            units.append(cur)
            cur = []
    sq, skv = max_n * Hq * D * 2, max_n * Hkv * D * 2
    R_log = []

    def run_unit(u, record=False):
        p = u % POOL
        row = 0
        for (nrows, seg, pos, unit) in units[u]:
            for layer in range(L):
                oq = ((p * L + layer) * max_n + row) * Hq * D * 2
                okv = ((p * L + layer) * max_n + row) * Hkv * D * 2
                meta = (seg, pos, unit) if layer == 0 else (None, None, None)
                r.check(lib.a2t_append_attn(h, layer, 1, ids, nrows, kp.data_ptr() + okv,
                                            vp.data_ptr() + okv, *meta, nrows, qp.data_ptr() + oq,
                                            out.data_ptr()), "a2t_append_attn")
            if record:
                R_log.append((r.stream_info(0).resident, nrows[0]))
            row += nrows[0]
        r.check(lib.a2t_evict(h, 1, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")

    for u in range(args.warmup):
        run_unit(u)
    n_calls = sum(len(units[u]) for u in range(args.warmup, args.warmup + args.steps))
    step_ms, total_ms, t_wall, t_enq = r.timed(lambda j: run_unit(args.warmup + j, record=True),
                                               args.steps, kernel=kernel, launches=n_calls * L)
    launches = len(R_log)
    alg = float(np.mean([attn_bytes(R, n, cfg) for R, n in R_log])) if R_log else 0.0
    kern_timed = r.kern_timed
    p0 = args.warmup + args.steps
    kern = r.profiled(lambda j: run_unit(p0 + j), args.profile_steps)
    kern_steps = [p0, p0 + args.profile_steps]
    steps_per_unit = sum(len(units[u]) for u in range(args.warmup, p0)) / max(1, args.steps)
    r.close()
    base_line = None
    if kernel is None and not args.no_cpu_baseline:
        k0 = sum(len(units[u]) for u in range(args.warmup))
        n_units = max(1, min(args.steps, 4))
        n_steps = sum(len(units[u]) for u in range(args.warmup, args.warmup + n_units))
        base_line = cpu_baseline_steps(cfg, args.seed, spec, k0, n_steps, n_units,
                                       args.cpu_sample_layers)
    return {
        "value": 1000.0 * args.steps / total_ms,
        "ms_per_step": total_ms / args.steps,
        "config": {
            "workload": "ten-minute single stream, side-channel cadence: per unit a prefill chunk of "
                        "17 acoustic/structural rows, then one decode step per side-channel token "
                        "(2 delimiters + Poisson(3) transcript tokens); 36 layers, 32 query / 8 KV "
                        "heads, head dim 128, bf16, budget 4096 rows, recent window 30 units",
            "timed_units": [args.warmup, p0],
            "calls_per_unit": steps_per_unit,
            "calls": "a2t_append_attn per layer and step, one a2t_evict per unit",
            "seed": args.seed,
        },
        "roofline": roofline("attn_tile", kern_timed, alg, "cadence"),
        **timing_fields(step_ms, total_ms, args.steps, t_wall, t_enq),
        "kernels_us": kern,
        "kernels_us_steps": kern_steps,
        "timed_attention_calls": launches,
        "cpu_baseline": base_line,
    }


def two_pass(session, args, kernel):
    """The rate from a pass without timestamped dispatches; the dominant
    kernel's roofline from a second pass over the same steps (fresh cache,
    same inputs) whose dispatches of that kernel are timestamped."""
    clean = session(args, None)
    timed = session(args, kernel)
    clean["roofline"] = timed["roofline"]
    clean["timed_pass_ms_per_step"] = timed["ms_per_step"]
    return clean


def run_varlen(args):
    return two_pass(_varlen_session, args, "attn_tile")


def run_decode(args):
    return two_pass(_decode_session, args, "attn_tile")


def run_cadence(args):
    return two_pass(_cadence_session, args, "attn_tile")


# ------------------------------------------------------------------- hour-long sessions
def run_hour(args):
    """16 hour-long sessions (3,600 units, budget 8192, window 60), then the same
    sessions with no eviction (the control).  Each group: the units before the
    timed window are filled with one all-layers append per unit (plus the
    eviction check for the evicting group), then --steps units run the full path
    (a2t_append_attn on every layer, a2t_evict) timed with HIP events, then
    --profile-steps more units with the attention dispatches timestamped."""
    cfg = CONFIGS[4]
    specs = make_workload(cfg, seed=args.seed).streams
    S, L, Hq, Hkv, D = len(specs), cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = min(len(s.steps) for s in specs)
    steps = min(args.steps, T - 1)
    prof = min(args.profile_steps, T - steps - 1)
    t0 = T - steps - prof
    max_n = cfg.max_unit_rows
    elt_row = 2 * Hkv * D * 2 * L   # K and V bytes of one cached row over all layers
    ids = (C.c_int32 * S)(*range(S))
    budget = (C.c_int32 * S)(*[cfg.budget] * S)
    metas = []
    for t in range(T):
        seg = np.concatenate([s.steps[t].seg for s in specs])
        pos = np.concatenate([s.steps[t].pos for s in specs])
        metas.append(((C.c_int32 * S)(*[s.steps[t].n for s in specs]),
                      (C.c_uint8 * len(seg))(*seg.tolist()), (C.c_int32 * len(pos))(*pos.tolist()),
                      (C.c_int32 * S)(*[s.steps[t].unit for s in specs]), int(len(seg))))
    max_tot = max(m[4] for m in metas)

    def group(evict):
        if evict:
            unit_rows = max(cfg.budget, cfg.window * max_n) + 2 * max_n
            kept = max(sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in s.steps)
                       for s in specs) + 64
        else:
            unit_rows, kept = max(s.total_rows() for s in specs) + 64, 64
        r = Runner(cfg, S, unit_rows, kept, max_n)
        torch, lib, h = r.torch, r.lib, r.h
        n_ev, unmet = (C.c_int32 * S)(), (C.c_uint8 * S)()
        # fill: the all-layers input is packed [L][rows of the unit][Hkv][D]; a view of
        # the front of one flat buffer has that shape for any row count
        kflat = r.pool((L * max_tot * Hkv * D,), args.seed + 10)
        vflat = r.pool((L * max_tot * Hkv * D,), args.seed + 11)
        for t in range(t0):
            nrows, seg, pos, unit, tot = metas[t]
            n_el = L * tot * Hkv * D
            r.check(lib.a2t_append(h, -1, S, ids, nrows, kflat[:n_el].data_ptr(),
                                   vflat[:n_el].data_ptr(), seg, pos, unit), "a2t_append")
            if evict:
                r.check(lib.a2t_evict(h, S, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")
        torch.cuda.synchronize()
        P = 2
        qp = r.pool((P, L, max_tot, Hq, D), args.seed)
        kp = r.pool((P, L, max_tot, Hkv, D), args.seed + 1)
        vp = r.pool((P, L, max_tot, Hkv, D), args.seed + 2)
        out = torch.empty(max_tot, Hq, D, dtype=torch.bfloat16, device=r.dev)
        sq, skv = max_tot * Hq * D * 2, max_tot * Hkv * D * 2
        R_log = []

        def run_unit(t, record=False):
            nrows, seg, pos, unit, _ = metas[t]
            p = t % P
            for layer in range(L):
                oq, okv = (p * L + layer) * sq, (p * L + layer) * skv
                meta = (seg, pos, unit) if layer == 0 else (None, None, None)
                r.check(lib.a2t_append_attn(h, layer, S, ids, nrows, kp.data_ptr() + okv,
                                            vp.data_ptr() + okv, *meta, nrows,
                                            qp.data_ptr() + oq, out.data_ptr()), "a2t_append_attn")
            if record:
                R_log.append(sum(attn_bytes(r.stream_info(i).resident, nrows[i], cfg)
                                 for i in range(S)))
            if evict:
                r.check(lib.a2t_evict(h, S, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")

        step_ms, total_ms, t_wall, t_enq = r.timed(lambda j: run_unit(t0 + j), steps)
        r.timed(lambda j: run_unit(t0 + steps + j, record=True), prof, kernel="attn_tile",
                launches=prof * L)
        kern_timed = r.kern_timed
        peak = max(r.stream_info(i).peak for i in range(S))
        resident = [r.stream_info(i).resident for i in range(S)]
        r.close()
        return {"stream_unit_steps_per_s": S * steps / (total_ms * 1e-3),
                "ms_per_step": total_ms / steps,
                "unit_ms": {"mean": float(step_ms.mean()), "p99": float(np.percentile(step_ms, 99)),
                            "over_1s": int((step_ms > 1000).sum())},
                "peak_rows_per_stream": peak, "peak_kv_bytes_per_stream": peak * elt_row,
                "resident_rows_mean_at_end": float(np.mean(resident)),
                "roofline": roofline("attn_tile", kern_timed,
                                     float(np.mean(R_log)) if R_log else 0.0, "hour")}

    ev = group(True)
    ctl = group(False)
    base_line = None
    if not args.no_cpu_baseline:
        # one of the 16 streams (the oracle runs streams one at a time) on the evicting
        # group's first timed units, 16 of 36 layers, scaled to all layers
        base_line = cpu_baseline(cfg, specs[0], args.seed, t0, min(8, steps), 16)
        base_line["unit"] = "stream unit-steps/s"
    return {
        "value": ev["stream_unit_steps_per_s"],
        "ms_per_step": ev["ms_per_step"],
        "config": {
            "workload": "hour-long sessions: 16 streams x 3600 units, budget 8192 rows, recent "
                        "window 60 units, and the same 16 streams with no eviction (control); "
                        "36 layers, 32 query / 8 KV heads, head dim 128, bf16",
            "timed_units": [t0, t0 + steps],
            "attention_timed_units": [t0 + steps, t0 + steps + prof],
            "calls": "units before the timed window: one all-layers a2t_append (+ a2t_evict); "
                     "timed: a2t_append_attn per layer over the 16 streams, a2t_evict",
            "seed": args.seed,
        },
        "roofline": ev["roofline"],
        "evict": ev,
        "control": ctl,
        "peak_reduction": 1.0 - ev["peak_rows_per_stream"] / ctl["peak_rows_per_stream"],
        "cpu_baseline": base_line,
    }


# ------------------------------------------------------------------- budget sweep
def run_sweep(args):
    from synth.streams import make_sessions
    cfg = CONFIGS[1]
    n_units = min(args.steps, cfg.units)
    specs = make_sessions(cfg, range(args.seed, args.seed + 15), units=n_units).streams
    S, L, Hq, Hkv, D = len(specs), cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    max_n = cfg.max_unit_rows
    total = max(s.total_rows() for s in specs)
    keep_rows = max(sum(int(np.isin(st.seg, KEEP_SEGS).sum()) for st in s.steps) for s in specs)
    metas = []
    for u in range(n_units):
        seg = np.concatenate([s.steps[u].seg for s in specs])
        pos = np.concatenate([s.steps[u].pos for s in specs])
        metas.append(((C.c_int32 * S)(*[s.steps[u].n for s in specs]),
                      (C.c_uint8 * len(seg))(*seg.tolist()), (C.c_int32 * len(pos))(*pos.tolist()),
                      (C.c_int32 * S)(*[s.steps[u].unit for s in specs])))
    rows = []
    value = None
    last = None
    # the paper's rule over Table 3's budgets, then its two variants: per-row
    # granularity at the selected budget, and the StreamingLLM comparison (4
    # sink rows + 2,000 recent positions, Table 1)
    sweep = [(B, None, 0) for B in (None, 8000, 6000, 4000, 0)] + \
        [(4000, "row", 0), (4 + 2000, "sink_recent", 4)]
    rule_ids = {None: 0, "row": 1, "sink_recent": 2}
    for B, rule, n_sink in sweep:
        r = Runner(cfg, S, total + 64, keep_rows + 64, max_n)
        torch, lib, h = r.torch, r.lib, r.h
        if last is None:
            qp = r.pool((2, L, S * max_n, Hq, D), args.seed)
            kp = r.pool((2, L, S * max_n, Hkv, D), args.seed + 1)
            vp = r.pool((2, L, S * max_n, Hkv, D), args.seed + 2)
            out = torch.empty(S * max_n, Hq, D, dtype=torch.bfloat16, device=r.dev)
            last = (qp, kp, vp, out)
        qp, kp, vp, out = last
        ids = (C.c_int32 * S)(*range(S))
        budget = (C.c_int32 * S)(*[B or 0] * S)
        n_ev, unmet = (C.c_int32 * S)(), (C.c_uint8 * S)()
        sq, skv = S * max_n * Hq * D * 2, S * max_n * Hkv * D * 2

        def run_unit(u):
            nrows, seg, pos, unit = metas[u]
            p = u % 2
            for layer in range(L):
                oq, okv = (p * L + layer) * sq, (p * L + layer) * skv
                meta = (seg, pos, unit) if layer == 0 else (None, None, None)
                r.check(lib.a2t_append_attn(h, layer, S, ids, nrows, kp.data_ptr() + okv,
                                            vp.data_ptr() + okv, *meta, nrows, qp.data_ptr() + oq,
                                            out.data_ptr()), "a2t_append_attn")
            if B is not None and rule is None:
                r.check(lib.a2t_evict(h, S, ids, budget, cfg.window, n_ev, unmet), "a2t_evict")
            elif B is not None:
                r.check(lib.a2t_evict_rule(h, S, ids, budget, cfg.window, rule_ids[rule], n_sink,
                                           n_ev, unmet), "a2t_evict_rule")

        step_ms, total_ms, t_wall, t_enq = r.timed(run_unit, n_units)
        ends = [r.stream_info(i).resident for i in range(S)]
        peaks = [r.stream_info(i).peak for i in range(S)]
        r.close()
        if rule == "sink_recent":
            label = f"{n_sink} sinks + {B - n_sink} recent (StreamingLLM)"
        else:
            label = "per-row (ablation)" if rule == "row" else "unit (Sec. 3.3)"
        rows.append({"budget": "unbounded" if B is None else B, "rule": label,
                     "end_rows_mean": float(np.mean(ends)),
                     "peak_rows_mean": float(np.mean(peaks)), "step_ms_mean": float(step_ms.mean()),
                     "step_ms_p99": float(np.percentile(step_ms, 99)),
                     "steps_over_1s": int((step_ms > 1000).sum())})
        if B == 4000 and rule is None:
            value = S * n_units / (total_ms * 1e-3)
            ms_per_step = total_ms / n_units
    return {
        "value": value,
        "ms_per_step": ms_per_step,
        "config": {
            "workload": "budget sweep: 15 synthetic ten-minute sessions (600 units of 17 acoustic + "
                        "2 delimiter + Poisson(3) transcript rows) batched in one cache; budgets "
                        "unbounded/8000/6000/4000/0 rows, recent window 30 units, then per-row "
                        "eviction at 4000 and 4 sinks + 2000 recent rows; 36 layers, 32 "
                        "query / 8 KV heads, head dim 128, bf16",
            "sessions": S, "units": n_units,
            "calls": "a2t_append_attn per layer over all sessions, one a2t_evict (or "
                     "a2t_evict_rule) per unit",
            "seed": args.seed,
        },
        "sweep": rows,
        "roofline": None,
        "cpu_baseline": None,
    }


# ------------------------------------------------------------------- adaptation objective
def run_distill(args):
    import torch
    import paper_2609_31224_amd as a2t
    from synth.distill import make_distill_batch
    vocab, added = 151936, 2
    b = make_distill_batch(seed=args.seed, n_utt=16, units=12, vocab=vocab, added=added,
                           dtype="bf16")
    n = b.n
    ss = (vocab + added + 7) // 8 * 8
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    st = torch.zeros(n, ss, dtype=torch.bfloat16, device=dev)
    st[:, :vocab + added] = torch.from_numpy(b.student).to(dev).to(torch.bfloat16)
    te = torch.from_numpy(b.teacher).to(dev).to(torch.bfloat16).contiguous()
    grad = torch.empty_like(st)
    losses = torch.zeros(5, dtype=torch.float32, device=dev)
    d = a2t.a2t_distill_create(n, vocab, added, a2t.A2T_BF16, stream=stream)
    lib = a2t.raw_lib()
    P8, P32 = C.POINTER(C.c_int8), C.POINTER(C.c_int32)
    kind = np.ascontiguousarray(b.kind, np.int8)
    tgt = np.ascontiguousarray(b.target, np.int32)
    dec = np.ascontiguousarray(b.dec_group, np.int8)
    turn = np.ascontiguousarray(b.turn_group, np.int8)

    def call(with_grad=True):
        rc = lib.a2t_distill_loss(d.ptr, n, st.data_ptr(), ss, te.data_ptr(), vocab,
                                  kind.ctypes.data_as(P8), tgt.ctypes.data_as(P32),
                                  dec.ctypes.data_as(P8), turn.ctypes.data_as(P8), 1.0,
                                  losses.data_ptr(), grad.data_ptr() if with_grad else None)
        if rc:
            raise a2t.A2TError(rc, "a2t_distill_loss")

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for j in range(args.steps):
        call()
        evs[j + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = np.array([evs[j].elapsed_time(evs[j + 1]) for j in range(args.steps)])
    total_ms = float(evs[0].elapsed_time(evs[-1]))
    # the same calls again with the per-row kernel's dispatches timestamped (a
    # second pass: timestamped dispatches slow the issue rate)
    lib.a2t_distill_profile_reserve(d.ptr, args.steps)
    lib.a2t_distill_profile_enable(d.ptr, 1)
    for j in range(args.steps):
        call()
    torch.cuda.synchronize()
    nl, ms = C.c_int64(), C.c_double()
    lib.a2t_distill_kernel_time(d.ptr, C.byref(nl), C.byref(ms))
    lib.a2t_distill_profile_enable(d.ptr, 0)
    kern = {"distill_row": {"launches": nl.value, "avg_us": ms.value * 1e3 / max(1, nl.value)}}
    for name, wg in (("distill_row_loss_only", False),):
        lib.a2t_distill_profile_enable(d.ptr, 1)
        for _ in range(max(1, args.profile_steps)):
            call(wg)
        nl, ms = C.c_int64(), C.c_double()
        lib.a2t_distill_kernel_time(d.ptr, C.byref(nl), C.byref(ms))
        lib.a2t_distill_profile_enable(d.ptr, 0)
        kern[name] = {"launches": nl.value, "avg_us": ms.value * 1e3 / max(1, nl.value)}
    a2t.a2t_distill_destroy(d)
    # a streaming floor for the same bytes: one elementwise pass that reads both
    # logit arrays once and writes one array of the same size (torch's add), the
    # traffic a single-pass evaluation with the gradient would move
    st_v, grad_v = st[:, :vocab], grad[:, :vocab]
    for _ in range(3):
        torch.add(st_v, te, out=grad_v)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        torch.add(st_v, te, out=grad_v)
    ev1.record(stream)
    torch.cuda.synchronize()
    floor_us = ev0.elapsed_time(ev1) * 1e3 / args.steps
    floor_bytes = 3 * n * vocab * 2
    # algorithmic bytes of one evaluation: read both logit rows once, write the gradient once
    alg = n * ((vocab + added) * 2 + vocab * 2 + (vocab + added) * 2)
    alg_loss = n * ((vocab + added) * 2 + vocab * 2)
    us = kern["distill_row"]["avg_us"]
    achieved = alg / (us * 1e-6) / 1e9
    base_line = None
    if not args.no_cpu_baseline:
        from oracle.distill import row_terms, row_gradient
        # chunks of 64 rows (bounded memory) until ~10 s of CPU work or two passes
        done, dt, t0 = 0, 0.0, time.perf_counter()
        while dt < 10.0 and done < 2 * n:
            r0 = done % n
            rows = np.arange(r0, min(n, r0 + 64))
            tg = np.where(b.kind[rows] == 1, b.target[rows], -1)
            row_terms(b.student[rows], b.teacher[rows], tg)
            row_gradient(b.student[rows], b.teacher[rows], tg, np.ones(len(rows)), np.ones(len(rows)))
            done += len(rows)
            dt = time.perf_counter() - t0
        base_line = {"value": done / dt / n, "unit": "evaluations/s", "cores": _threads_used(),
                     "kind": "oracle",
                     "sample": f"{done} row evaluations of the {n}-row batch (per-row terms and "
                               f"gradient, fp64 numpy, 64 rows at a time), scaled to the batch; "
                               f"{dt:.1f} s of CPU work"}
    return {
        "value": 1000.0 * args.steps / total_ms,
        "ms_per_step": total_ms / args.steps,
        "config": {
            "workload": f"adaptation objective: 16 utterances x 12 units = {n} prediction rows "
                        f"(first decisions, side-channel tokens, native non-decision rows), vocabulary "
                        f"{vocab} + {added} added tokens, bf16 logits, T = 1, losses + gradient",
            "rows": n, "seed": args.seed,
        },
        "roofline": {"bound": "hbm", "kernel": "distill_row", "achieved": achieved,
                     "timing": "per-dispatch start/stop events, in a second pass over the same calls",
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": None, "avg_launch_us": us, "alg_bytes_per_launch": alg},
        "loss_only": {"avg_launch_us": kern["distill_row_loss_only"]["avg_us"],
                      "alg_bytes_per_launch": alg_loss,
                      "achieved_gbps": alg_loss / (kern["distill_row_loss_only"]["avg_us"] * 1e-6) / 1e9},
        "kernels_us": kern,
        "single_pass_floor": {"kernel": "torch.add of the two logit arrays into a third",
                              "avg_us": floor_us, "bytes": floor_bytes,
                              "gbps": floor_bytes / (floor_us * 1e-6) / 1e9,
                              "distill_row_over_floor": us / floor_us},
        "unit_ms": {"mean": float(step_ms.mean()), "p50": float(np.percentile(step_ms, 50)),
                    "p99": float(np.percentile(step_ms, 99))},
        "cpu_baseline": base_line,
    }


# ------------------------------------------------------------------- copy reference
def run_copy(args):
    import torch
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    n = 1 << 30
    x = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    y = torch.empty_like(x)
    for _ in range(args.warmup):
        y.copy_(x)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(args.steps):
        y.copy_(x)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / args.steps
    return {"value": 2 * n / (ms * 1e-3) / 1e9, "ms_per_step": ms,
            "config": {"workload": "device copy of 1 GiB (read 1 GiB + write 1 GiB per step)",
                       "bytes_read": n, "bytes_written": n},
            "roofline": {"bound": "hbm", "kernel": "copy", "achieved": 2 * n / (ms * 1e-3) / 1e9,
                         "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": 2 * n / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, "traffic": None},
            "cpu_baseline": None}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", choices=sorted(METRICS), default="stream")
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--profile-steps", type=int, default=None,
                    help="extra steps after the timed ones with every dispatch timestamped "
                         "(the per-kernel averages in kernels_us, over kernels_us_steps)")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--jsonl", default=None,
                    help="ten-minute stream: write one JSON record per timed unit to this file")
    ap.add_argument("--cpu-sample-units", type=int, default=20,
                    help="ten-minute stream: oracle units timed, from the first timed unit")
    ap.add_argument("--cpu-sample-layers", type=int, default=36)
    ap.add_argument("--unfused", action="store_true",
                    help="stream workload: per layer a2t_append then a2t_chunk_attn")
    ap.add_argument("--decode-call", choices=("decode", "fused"), default="decode",
                    help="decode workload: a2t_append + a2t_decode_attn, or a2t_append_attn")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(the KV step shards by stream or by KV head with no exchange).", file=sys.stderr)
        sys.exit(2)
    w, s, p = DEFAULTS[args.workload]
    args.warmup = w if args.warmup is None else args.warmup
    args.steps = s if args.steps is None else args.steps
    args.profile_steps = p if args.profile_steps is None else args.profile_steps
    if args.seed is None:
        args.seed = {"stream": 1, "varlen": 2, "decode": 3, "cadence": 1, "sweep": 1,
                     "distill": 14, "hour": 4, "copy": 0, "graph": 1}[args.workload]

    res = {"stream": run_stream, "varlen": run_varlen, "decode": run_decode,
           "cadence": run_cadence, "sweep": run_sweep, "distill": run_distill,
           "hour": run_hour, "copy": run_copy, "graph": run_graph}[args.workload](args)
    metric, unit = METRICS[args.workload]
    result = {
        "metric": metric,
        "value": res.pop("value"),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8" if args.workload == "copy" else "bf16",
        "data": "synthetic",
    }
    result.update(res)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
