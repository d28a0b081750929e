"""GPU parity of device-planned steps (a2t_dev_*) and their HIP-graph replay.

The same streams run through the device-planned calls (the device opens each
step from metadata in device memory, plans the key splits and Sec. 3.3's
eviction itself) against the fp64 oracle: attention on the checked layers at
every step (<= 2e-2, bf16), and, with the state handed back to the host
(a2t_dev_end), the layout, the eviction mask and compaction indices and the
stored K/V (bit-exact) at every step.  Then one step of the benchmark's shape
is captured in a HIP graph once and replayed for the following units with new
metadata and values in the same device buffers, every replay checked against
the oracle, with eager work and synchronisations between replays."""
import numpy as np
import pytest

from synth.streams import CONFIGS, bf16_round, make_workload, step_values, tiny_stream
from tests.harness import Mismatch, bf16_bits_to_f32, make_cache, row_bounds

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


class DevRun:
    """Streams of one cache driven through the device-planned calls, with the
    oracle alongside.  Values come from the seeded generator on the checked
    layers; other layers reuse the first checked layer's values."""

    def __init__(self, cfg, seed, specs, budgets, window, layers_checked, n_layers, unit_rows,
                 kept_rows, max_step, rule=None, n_sink=0):
        import torch
        import paper_2609_31224_amd as a2t
        from oracle.cache import OracleCache
        from oracle.policy import EvictRule
        self.torch, self.a2t = torch, a2t
        # eviction rule: None = a2t_dev_evict (Sec. 3.3's whole-unit rule), else
        # "unit" / "row" / "sink_recent" through a2t_dev_evict_rule
        self.rule, self.n_sink = rule, n_sink
        self.oracle_rule = EvictRule(rule or "unit", n_sink)
        self.cfg, self.seed, self.specs = cfg, seed, specs
        self.budgets, self.window = budgets, window
        self.layers_checked, self.L = list(layers_checked), n_layers
        self.MS = max_step
        self.cache = make_cache(cfg, len(specs), unit_rows, kept_rows, max_step, n_layers=n_layers,
                                dtype="bf16")
        self.oracles = [OracleCache(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, self.layers_checked,
                                    theta=cfg.rope_theta, scale=cfg.scale) for _ in specs]
        S, MS, Hq, Hkv, D = len(specs), max_step, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
        dev, bf = "cuda", torch.bfloat16
        # fixed device buffers: what a captured step reads and writes
        self.n_rows = torch.zeros(S, dtype=torch.int32, device=dev)
        self.unit = torch.zeros(S, dtype=torch.int32, device=dev)
        self.seg = torch.zeros(S, MS, dtype=torch.uint8, device=dev)
        self.pos = torch.zeros(S, MS, dtype=torch.int32, device=dev)
        self.budget = torch.tensor(budgets, dtype=torch.int32, device=dev)
        self.n_ev = torch.zeros(S, dtype=torch.int32, device=dev)
        self.unmet = torch.zeros(S, dtype=torch.uint8, device=dev)
        self.k = torch.zeros(n_layers, S, MS, Hkv, D, dtype=bf, device=dev)
        self.v = torch.zeros(n_layers, S, MS, Hkv, D, dtype=bf, device=dev)
        self.q = torch.zeros(n_layers, S, MS, Hq, D, dtype=bf, device=dev)
        self.o = torch.zeros(n_layers, S, MS, Hq, D, dtype=bf, device=dev)
        self.max_err = 0.0
        self.evictions = 0

    def close(self):
        self.a2t.a2t_cache_destroy(self.cache)

    def fill(self, t):
        """Write step t of every stream into the fixed buffers; feed the oracle."""
        torch, cfg = self.torch, self.cfg
        self.step_t = t
        S = len(self.specs)
        n_rows = np.zeros(S, np.int32)
        unit = np.zeros(S, np.int32)
        seg = np.zeros((S, self.MS), np.uint8)
        pos = np.zeros((S, self.MS), np.int32)
        self.vals = []
        for i, spec in enumerate(self.specs):
            st = spec.steps[t]
            n_rows[i], unit[i] = st.n, st.unit
            seg[i, :st.n], pos[i, :st.n] = st.seg, st.pos
            vv = step_values(cfg, self.seed, spec.stream, st.key, st.n, self.layers_checked)
            if cfg.dtype != "bf16":
                # a bf16 cache on an fp32 workload: both sides see the bf16-rounded inputs
                vv = {name: bf16_round(a) for name, a in vv.items()}
            self.vals.append(vv)
            k = {l: vv["k"][j] for j, l in enumerate(self.layers_checked)}
            v = {l: vv["v"][j] for j, l in enumerate(self.layers_checked)}
            self.oracles[i].append(st.seg, st.pos, st.unit, k, v)
            for layer in range(self.L):
                j = self.layers_checked.index(layer) if layer in self.layers_checked else 0
                for name, buf in (("k", self.k), ("v", self.v), ("q", self.q)):
                    buf[layer, i, :st.n] = torch.from_numpy(vv[name][j]).to("cuda").to(buf.dtype)
        self.n_rows.copy_(torch.from_numpy(n_rows))
        self.unit.copy_(torch.from_numpy(unit))
        self.seg.copy_(torch.from_numpy(seg))
        self.pos.copy_(torch.from_numpy(pos))

    def issue(self):
        """The step's device-planned calls (what a graph captures)."""
        a2t = self.a2t
        a2t.a2t_dev_open(self.cache, list(range(len(self.specs))), self.n_rows, self.unit, self.seg,
                         self.pos)
        for layer in range(self.L):
            a2t.a2t_dev_append_attn(self.cache, layer, self.k[layer], self.v[layer], self.q[layer],
                                    self.o[layer])
        if self.rule is None:
            a2t.a2t_dev_evict(self.cache, self.budget, self.window, self.n_ev, self.unmet)
        else:
            lib_rule = {"unit": a2t.A2T_RULE_UNIT, "row": a2t.A2T_RULE_ROW,
                        "sink_recent": a2t.A2T_RULE_SINK_RECENT}[self.rule]
            a2t.a2t_dev_evict_rule(self.cache, self.budget, self.window, lib_rule, self.n_sink,
                                   self.n_ev, self.unmet)

    def check(self, full):
        """Attention of step t against the oracle; with ``full`` also the
        eviction, layout and stored K/V (hands the state to the host and back)."""
        torch, a2t = self.torch, self.a2t
        torch.cuda.synchronize()
        t = self.step_t
        for i, spec in enumerate(self.specs):
            st = spec.steps[t]
            for j, layer in enumerate(self.layers_checked):
                og = self.o[layer, i, :st.n].to(torch.float32).cpu().numpy()
                want = self.oracles[i].attention(layer, self.vals[i]["q"][j], st.n)
                err = float(np.abs(og - want).max())
                self.max_err = max(self.max_err, err)
                if not err <= BF16_TOL:
                    raise Mismatch(f"step {t} stream {i} layer {layer}: attention max err {err}")
        n_ev = self.n_ev.cpu().numpy()
        unmet = self.unmet.cpu().numpy()
        recs = [o.evict(b, self.window, self.oracle_rule) for o, b in zip(self.oracles, self.budgets)]
        for i, rec in enumerate(recs):
            if int(n_ev[i]) != rec.n_evicted or bool(unmet[i]) != rec.plan.budget_unmet:
                raise Mismatch(f"step {t} stream {i}: evicted {n_ev[i]}/{rec.n_evicted} "
                               f"unmet {unmet[i]}/{rec.plan.budget_unmet}")
            self.evictions += int(rec.n_evicted > 0)
        if not full:
            return
        a2t.a2t_dev_end(self.cache)
        for i, rec in enumerate(recs):
            p, s, u = a2t.a2t_read_layout(self.cache, i)
            if not (np.array_equal(p, rec.pos) and np.array_equal(s, rec.seg)
                    and np.array_equal(u, rec.unit)):
                raise Mismatch(f"step {t} stream {i}: layout differs")
            if rec.n_evicted:
                n_pre, mask, slot = a2t.a2t_read_last_evict(self.cache, i)
                if n_pre != rec.plan.n_pre or not np.array_equal(mask.astype(bool), rec.plan.evict_mask) \
                        or not np.array_equal(slot, rec.new_slot):
                    raise Mismatch(f"step {t} stream {i}: eviction mask / compaction indices differ")
            layer = self.layers_checked[0]
            k, v = a2t.a2t_read_kv(self.cache, layer, i)
            kf, vf = bf16_bits_to_f32(k), bf16_bits_to_f32(v)
            ko = self.oracles[i].k[layer]
            if kf.shape != ko.shape or not np.all(np.abs(kf - ko) <= np.abs(ko) * 2.0 ** -8 + 1e-6):
                raise Mismatch(f"step {t} stream {i}: stored K differs")
            if not np.array_equal(vf, self.oracles[i].v[layer]):
                raise Mismatch(f"step {t} stream {i}: stored V differs")
        a2t.a2t_dev_begin(self.cache)


def _bounds(specs):
    return dict(unit_rows=max(row_bounds(s)[0] for s in specs),
                kept_rows=max(row_bounds(s)[1] for s in specs) + 8,
                max_step=max(row_bounds(s)[2] for s in specs))


def test_device_planned_config0_shape(gpu):
    """Config 0's stream structure (bf16, 4/1 heads, D 64) with two more
    streams of other seeds and budgets in the same cache: every step checked
    in full."""
    cfg = CONFIGS[0]
    specs = [make_workload(cfg, seed=s).streams[0] for s in (0, 4, 7)]
    run = DevRun(cfg, 0, specs, [cfg.budget, 200, 300], cfg.window, [0], 1, **_bounds(specs))
    import paper_2609_31224_amd as a2t
    try:
        a2t.a2t_dev_begin(run.cache)
        for t in range(len(specs[0].steps)):
            run.fill(t)
            run.issue()
            run.check(full=True)
        a2t.a2t_dev_end(run.cache)
    finally:
        run.close()
    print(f"[device cfg0] evictions={run.evictions} max_err={run.max_err:.3e}", flush=True)
    assert run.evictions > 60


@pytest.mark.parametrize("rule,n_sink,budgets", [("unit", 0, (None, 200, 300)),
                                                   ("row", 0, (None, 200, 300)),
                                                   ("row", 0, (1, 57, 123)),
                                                   ("sink_recent", 4, (None, 200, 64)),
                                                   ("sink_recent", 0, (30, 7, 1)),
                                                   ("sink_recent", 17, (17, 40, 100))])
def test_device_planned_rule_variants_config0(gpu, rule, n_sink, budgets):
    """The variants of the rule planned on the device (a2t_dev_evict_rule):
    config 0's stream structure with two more streams, every step checked in
    full against the oracle's replay of the same rule (layout, mask and
    compaction indices bit-exact, stored K/V, attention).  Budgets include the
    sink count itself (nothing but sinks and recent rows) and tiny budgets that
    evict at almost every step."""
    cfg = CONFIGS[0]
    specs = [make_workload(cfg, seed=s).streams[0] for s in (0, 4, 7)]
    budgets = [cfg.budget if b is None else b for b in budgets]
    run = DevRun(cfg, 0, specs, budgets, cfg.window, [0], 1, rule=rule, n_sink=n_sink,
                 **_bounds(specs))
    import paper_2609_31224_amd as a2t
    try:
        a2t.a2t_dev_begin(run.cache)
        for t in range(len(specs[0].steps)):
            run.fill(t)
            run.issue()
            run.check(full=True)
        a2t.a2t_dev_end(run.cache)
    finally:
        run.close()
    print(f"[device {rule} sinks {n_sink} budgets {budgets}] evictions={run.evictions} "
          f"max_err={run.max_err:.3e}", flush=True)
    assert run.evictions > 40


@pytest.mark.parametrize("case", range(12))
def test_device_planned_random_shapes(gpu, case):
    """Seeded random shapes through the device-planned calls: head counts and
    groups, head dims, up to five streams of one length with their own budgets,
    unit sizes, windows, rules and layer counts, every step checked in full."""
    import dataclasses
    from tests.test_gpu_random_shapes import HEADS
    rng = np.random.default_rng(2000 + case)
    hq, hkv = HEADS[int(rng.integers(len(HEADS)))]
    acoustic, cap = int(rng.integers(2, 41)), int(rng.choice([4, 16, 64]))
    cfg = dataclasses.replace(CONFIGS[0], index=200 + case, n_q_heads=hq, n_kv_heads=hkv,
                              head_dim=int(rng.choice([64, 128])), dtype="bf16",
                              n_streams=int(rng.choice([1, 2, 3, 5])),
                              units=int(rng.integers(15, 41)), acoustic_rows=acoustic,
                              text_mean=float(rng.uniform(0.3, 6.0)), text_cap=cap,
                              window=int(rng.choice([0, 1, 2, 5])))
    rule = [None, "row", "sink_recent"][int(rng.integers(3))]
    n_sink = int(rng.integers(0, 6)) if rule == "sink_recent" else 0
    n_layers = int(rng.choice([1, 2, 3]))
    specs = make_workload(cfg, seed=cfg.index).streams
    unit = acoustic + 2 + cap
    budgets = [max(n_sink, int(rng.integers(0, 10 * unit))) for _ in specs]
    run = DevRun(cfg, cfg.index, specs, budgets, cfg.window, sorted({0, n_layers - 1}), n_layers,
                 rule=rule, n_sink=n_sink, **_bounds(specs))
    import paper_2609_31224_amd as a2t
    try:
        a2t.a2t_dev_begin(run.cache)
        for t in range(len(specs[0].steps)):
            run.fill(t)
            run.issue()
            run.check(full=True)
        a2t.a2t_dev_end(run.cache)
    finally:
        run.close()
    print(f"[device random {case}] heads {hq}/{hkv} D{cfg.head_dim} streams {len(specs)} "
          f"B {budgets} W {cfg.window} rule={rule or 'unit'} sinks {n_sink} L={n_layers}: "
          f"evictions {run.evictions} max err {run.max_err:.2e}", flush=True)


def test_device_planned_odd_partial_blocks(gpu):
    """Three query heads on three KV heads and three streams through the
    device-planned calls: each stream's split partials start 16-byte aligned
    whatever the odd row counts of the streams before it."""
    import dataclasses
    import paper_2609_31224_amd as a2t
    cfg = dataclasses.replace(CONFIGS[0], index=310, n_q_heads=3, n_kv_heads=3, head_dim=64,
                              dtype="bf16", n_streams=3, units=30, acoustic_rows=9,
                              text_mean=2.0, text_cap=16, window=2)
    specs = make_workload(cfg, seed=cfg.index).streams
    budgets = [120, 200, 1000]
    run = DevRun(cfg, cfg.index, specs, budgets, cfg.window, [0], 1, **_bounds(specs))
    try:
        a2t.a2t_dev_begin(run.cache)
        for t in range(len(specs[0].steps)):
            run.fill(t)
            run.issue()
            run.check(full=True)
        a2t.a2t_dev_end(run.cache)
    finally:
        run.close()
    print(f"[device odd partials] evictions {run.evictions} max err {run.max_err:.2e}", flush=True)
    assert run.evictions > 0


def test_device_planned_sink_rule_errors(gpu):
    """A budget below the sink count is refused on the device for that stream
    only (A2T_ERR_INVALID from a2t_dev_end, nothing evicted); the other stream
    evicts as the host-planned rule does."""
    import paper_2609_31224_amd as a2t
    cfg = CONFIGS[0]
    specs = [tiny_stream([[1, 1, 3]] * 6), tiny_stream([[1, 1, 2]] * 6)]
    run = DevRun(cfg, 2, specs, [3, 6], 1, [0], 1, unit_rows=64, kept_rows=16, max_step=8,
                 rule="sink_recent", n_sink=4)
    try:
        a2t.a2t_dev_begin(run.cache)
        for t in range(3):
            run.fill(t)
            run.issue()
        run.torch.cuda.synchronize()
        # step 1 took stream 0 over its budget of 3 < 4 sinks: refused, and the
        # stream sits out step 2; stream 1 went from 9 to 6 rows at step 2
        assert run.n_ev.cpu().tolist() == [0, 3]
        # an open step: an unknown rule or a negative sink count is refused on
        # the host, nothing enqueued, and the step stays open
        run.fill(3)
        a2t.a2t_dev_open(run.cache, [0, 1], run.n_rows, run.unit, run.seg, run.pos)
        a2t.a2t_dev_append_attn(run.cache, 0, run.k[0], run.v[0], run.q[0], run.o[0])
        for rule, sinks in ((7, 0), (a2t.A2T_RULE_SINK_RECENT, -1)):
            with pytest.raises(a2t.A2TError) as e:
                a2t.a2t_dev_evict_rule(run.cache, run.budget, 1, rule, sinks)
            assert e.value.status == a2t.A2T_ERR_INVALID
        a2t.a2t_dev_evict_rule(run.cache, run.budget, 1, a2t.A2T_RULE_SINK_RECENT, 4, run.n_ev,
                               run.unmet)
        run.torch.cuda.synchronize()
        assert run.n_ev.cpu().tolist() == [0, 3]
        with pytest.raises(a2t.A2TError) as e:
            a2t.a2t_dev_end(run.cache)
        assert e.value.status == a2t.A2T_ERR_INVALID
        assert a2t.a2t_stream_info_get(run.cache, 0)["resident"] == 6
        assert a2t.a2t_stream_info_get(run.cache, 1)["resident"] == 6
        p, _, _ = a2t.a2t_read_layout(run.cache, 1)
        # the four sinks, then the budget's two newest rows
        assert p.tolist() == [0, 1, 2, 3, 10, 11]
    finally:
        run.close()


def test_device_planned_edge_streams(gpu):
    """A prefix, response rows under a unit, W = 0 and an unmet budget."""
    cfg = CONFIGS[0]
    units = [[1, 1, 2, 3, 2]] * 5 + [[4]] * 3 + [[1, 1, 2, 2]] * 4 + [[1, 3]] * 4
    spec = tiny_stream(units, prefix=2, pos_gap=2)
    run = DevRun(cfg, 5, [spec], [9], 0, [0], 1, unit_rows=128, kept_rows=64, max_step=16)
    import paper_2609_31224_amd as a2t
    try:
        a2t.a2t_dev_begin(run.cache)
        for t in range(len(spec.steps)):
            run.fill(t)
            run.issue()
            run.check(full=True)
        a2t.a2t_dev_end(run.cache)
    finally:
        run.close()
    assert run.evictions > 3


def test_device_planned_graph_replay_config1_shape(gpu):
    """The benchmark's shape (36 layers, 32/8 heads, D 128, bf16, budget 4096,
    window 30): 200 units eagerly through the device-planned calls, then one
    step captured in a HIP graph and replayed for units 200..239, each replay
    fed new metadata and values in the same buffers (eager copies and a
    synchronisation between replays) and checked against the oracle; the full
    state at the end."""
    import torch
    import paper_2609_31224_amd as a2t
    cfg = CONFIGS[1]
    spec = make_workload(cfg, units=240).streams[0]
    run = DevRun(cfg, cfg.index, [spec], [cfg.budget], cfg.window, [0, 35], cfg.n_layers,
                 **_bounds([spec]))
    stream = torch.cuda.Stream()
    a2t.a2t_set_stream(run.cache, stream.cuda_stream)
    try:
        with torch.cuda.stream(stream):
            a2t.a2t_dev_begin(run.cache)
            for t in range(200):
                run.fill(t)
                run.issue()
                run.check(full=(t % 50 == 49))
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                run.issue()
            replays = 0
            for t in range(200, 240):
                run.fill(t)
                g.replay()
                run.check(full=(t % 10 == 9))
                replays += 1
            a2t.a2t_dev_end(run.cache)
        info = a2t.a2t_stream_info_get(run.cache, 0)
        assert info["resident"] == run.oracles[0].resident
    finally:
        run.close()
    print(f"[device graph cfg1] replays={replays} evictions={run.evictions} "
          f"max_err={run.max_err:.3e}", flush=True)
    assert replays == 40 and run.evictions >= 50


def test_device_planned_error_is_reported(gpu):
    """A step whose positions do not increase is refused on the device: the
    stream keeps its state and a2t_dev_end reports A2T_ERR_POS."""
    import torch
    import paper_2609_31224_amd as a2t
    cfg = CONFIGS[0]
    spec = tiny_stream([[1, 1, 3]] * 3)
    run = DevRun(cfg, 1, [spec], [100], 1, [0], 1, unit_rows=64, kept_rows=16, max_step=8)
    try:
        a2t.a2t_dev_begin(run.cache)
        run.fill(0)
        run.issue()
        run.check(full=False)
        run.pos[0, :3] = torch.tensor([1, 5, 6], dtype=torch.int32)   # 1 <= last position 2
        run.issue()
        torch.cuda.synchronize()
        with pytest.raises(a2t.A2TError) as e:
            a2t.a2t_dev_end(run.cache)
        assert e.value.status == a2t.A2T_ERR_POS
        assert a2t.a2t_stream_info_get(run.cache, 0)["resident"] == 3
        p, _, _ = a2t.a2t_read_layout(run.cache, 0)
        assert p.tolist() == [0, 1, 2]
    finally:
        run.close()
