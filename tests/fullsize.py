"""Full-size batched runs checked on samples (test harness).

A workload runs through libA2T at its full size and in the batched call
pattern of the benchmark: every active stream of a global step goes into one
call per layer, then one a2t_evict.  What the oracle can afford is checked:

* every stream, every step: rows evicted and the budget flag, against the
  oracle's metadata-only policy replay (eviction reads no K/V values); at
  every step that evicts, the device's eviction mask and compaction indices
  (bit-exact) and the rows the library copied into its kept region (against
  the rows that join the oracle's retained prefix);
* every stream at the end: the device layout (pos, seg, unit per slot);
* sampled streams on the checked layers: attention outputs at every
  ``check_every``-th step (or at the global steps in ``check_steps``) and the
  stored K/V at the end, against an oracle cache fed the same seeded values:
  run in lockstep, or (``oracle="rebuild"``, for histories too long to carry
  along) rebuilt from the policy replay and the seeded generator at each
  checked step.

``listen_call``: "fused" (a2t_append_attn per layer), "fill" (one all-layers
a2t_append per listening step, no attention) or "fill_check" (fill, except
fused calls on the checked steps).

Only the sampled streams on the checked layers carry values from the seeded
generator; every other (stream, layer) slice gets fixed seeded pool values.
Streams and layers are independent in the cache (attention of a stream on a
layer reads only that stream's rows of that layer), so this changes no
checked result.
"""
from __future__ import annotations

import time

import numpy as np

from synth.streams import step_values
from tests.harness import Mismatch, bf16_bits_to_f32, make_cache


class SampledBatch:
    def __init__(self, cfg, seed, specs, *, sampled, layers_checked, budgets, window, unit_rows,
                 kept_rows, max_step, tol, check_every=1, check_steps=None, listen_call="fused",
                 decode_call="decode", evict=True, oracle="lockstep", label="", rule=None,
                 n_sink=0):
        import torch
        import paper_2609_31224_amd as a2t
        from oracle.cache import OracleCache
        from oracle.policy import EvictRule
        from oracle.replay import MetadataReplay, replay_metadata
        self.torch, self.a2t = torch, a2t
        # eviction rule: None = a2t_evict (Sec. 3.3), else "row" / "sink_recent"
        # through a2t_evict_rule
        self.rule, self.n_sink = rule, n_sink
        self.oracle_rule = EvictRule(rule or "unit", n_sink)
        self.cfg, self.seed, self.specs = cfg, seed, specs
        self.sampled = list(sampled)
        self.layers_checked = list(layers_checked)
        self.budgets = list(budgets)
        self.window, self.tol, self.check_every = window, tol, check_every
        self.listen_call, self.decode_call, self.evict = listen_call, decode_call, evict
        self.label = label
        self.check_steps = None if check_steps is None else set(check_steps)
        self.rebuild = oracle == "rebuild"
        self.kept_vals = {}
        S, L = len(specs), cfg.n_layers
        self.cache = make_cache(cfg, S, unit_rows, kept_rows, max_step)
        self.oracles = {} if self.rebuild else {
            i: OracleCache(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, self.layers_checked,
                           theta=cfg.rope_theta, scale=cfg.scale) for i in self.sampled}
        self.traces = [replay_metadata(s, b, window, evict=evict, rule=self.oracle_rule)
                       for s, b in zip(specs, self.budgets)]
        # step-by-step replays that also give each step's mask and compaction indices
        self.replays = [MetadataReplay(s, b, window, record_masks=True, rule=self.oracle_rule)
                        for s, b in zip(specs, self.budgets)] if evict else None
        self.moved = [0] * len(specs)
        self.mask_checks = 0
        self.T = max(s.offset + len(s.steps) for s in specs)
        max_rows = max(sum(s.steps[t - s.offset].n for s in specs
                           if 0 <= t - s.offset < len(s.steps)) for t in range(self.T))
        g = torch.Generator(device="cuda")
        g.manual_seed(1_000 + seed)
        bf = torch.bfloat16

        def pool(*shape):
            return torch.randn(shape, generator=g, device="cuda", dtype=torch.float32).to(bf)

        Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
        self.pq, self.pk, self.pv = pool(max_rows, Hq, D), pool(max_rows, Hkv, D), \
            pool(max_rows, Hkv, D)
        self.max_err = 0.0
        self.attn_checks = 0
        self.evictions = 0
        self.unmet_steps = 0
        self.layer_loop_s = 0.0

    def close(self):
        self.a2t.a2t_cache_destroy(self.cache)

    # ------------------------------------------------------------ inputs
    def _fill(self, base, layer, act, offs, vals, name):
        """base[:tot] with the sampled streams' rows replaced on checked layers."""
        torch = self.torch
        if layer not in self.layers_checked or not vals:
            return base
        j = self.layers_checked.index(layer)
        t = base.clone()
        for (i, st), off in zip(act, offs):
            if i in vals:
                t[off:off + st.n] = torch.from_numpy(vals[i][name][j]).to("cuda").to(t.dtype)
        return t

    # ------------------------------------------------------------ one global step
    def step(self, t):
        a2t, torch, cfg = self.a2t, self.torch, self.cfg
        act = [(i, s.steps[t - s.offset]) for i, s in enumerate(self.specs)
               if 0 <= t - s.offset < len(s.steps)]
        if not act:
            return
        ids = [i for i, _ in act]
        n = [st.n for _, st in act]
        offs = list(np.cumsum([0] + n[:-1]))
        tot = int(sum(n))
        seg = np.concatenate([st.seg for _, st in act])
        pos = np.concatenate([st.pos for _, st in act])
        unit = [st.unit for _, st in act]
        decode = all(st.decode for _, st in act)
        vals = {i: step_values(cfg, self.seed, self.specs[i].stream, st.key, st.n,
                               self.layers_checked)
                for i, st in act if i in self.sampled}
        if self.rebuild:
            # keep the sampled streams' K/V (the same values the GPU gets) for rebuilds
            for i, vv in vals.items():
                self.kept_vals.setdefault(i, []).append({"k": vv["k"], "v": vv["v"]})
        check = (t in self.check_steps) if self.check_steps is not None else \
            (t % self.check_every) == 0
        if self.rebuild and check:
            # the sampled streams' state before this step, rebuilt; then this step
            from oracle.replay import resume
            self.oracles = {i: resume(cfg, self.seed, self.specs[i], self.budgets[i], self.window,
                                      t - self.specs[i].offset, self.layers_checked,
                                      evict=self.evict, values=self.kept_vals[i].__getitem__)
                            for i, _ in act if i in self.sampled}
        for i, st in act:
            if i in vals and i in self.oracles:
                k = {l: vals[i]["k"][j] for j, l in enumerate(self.layers_checked)}
                v = {l: vals[i]["v"][j] for j, l in enumerate(self.layers_checked)}
                self.oracles[i].append(st.seg, st.pos, st.unit, k, v)
        pq, pk, pv = self.pq[:tot], self.pk[:tot], self.pv[:tot]
        t0 = time.perf_counter()
        fill = self.listen_call == "fill" or (self.listen_call == "fill_check" and not check)
        if not decode and fill:
            # all layers in one append call, no attention (the decode benchmark's fill)
            L = cfg.n_layers
            kall = pk.unsqueeze(0).expand(L, *pk.shape).contiguous()
            vall = pv.unsqueeze(0).expand(L, *pv.shape).contiguous()
            for l in self.layers_checked:
                kall[l] = self._fill(pk, l, act, offs, vals, "k")
                vall[l] = self._fill(pv, l, act, offs, vals, "v")
            a2t.a2t_append(self.cache, a2t.A2T_ALL_LAYERS, ids, n, kall, vall, seg, pos, unit)
        else:
            for layer in range(cfg.n_layers):
                kk = self._fill(pk, layer, act, offs, vals, "k")
                vv = self._fill(pv, layer, act, offs, vals, "v")
                q = self._fill(pq, layer, act, offs, vals, "q")
                o = torch.empty_like(q)
                meta = (seg, pos, unit) if layer == 0 else (None, None, None)
                if decode and self.decode_call == "decode":
                    a2t.a2t_append(self.cache, layer, ids, n, kk, vv, *meta)
                    a2t.a2t_decode_attn(self.cache, layer, ids, q, o)
                else:
                    a2t.a2t_append_attn(self.cache, layer, ids, n, kk, vv, *meta, n, q, o)
                if check and layer in self.layers_checked:
                    self._check_attention(t, layer, act, offs, vals, o)
        self.layer_loop_s += time.perf_counter() - t0
        rtr = {i: self.replays[i].step() for i, _ in act} if self.replays else {}
        act = [(i, st) for i, st in act if st.evict]  # checked after the steps ending a unit
        ids = [i for i, _ in act]
        if not act:
            return
        if self.evict:
            budgets = [self.budgets[i] for i in ids]
            if self.rule is None:
                n_ev, unmet = a2t.a2t_evict(self.cache, ids, budgets, self.window)
            else:
                n_ev, unmet = a2t.a2t_evict_rule(
                    self.cache, ids, budgets, self.window,
                    {"row": a2t.A2T_RULE_ROW, "sink_recent": a2t.A2T_RULE_SINK_RECENT}[self.rule],
                    self.n_sink)
        else:
            n_ev, unmet = np.zeros(len(ids), np.int32), np.zeros(len(ids), np.uint8)
        for j, (i, st) in enumerate(act):
            tr = self.traces[i].steps[t - self.specs[i].offset]
            want = tr.n_pre - tr.n_post
            if int(n_ev[j]) != want or bool(unmet[j]) != tr.budget_unmet:
                raise Mismatch(f"{self.label} step {t} stream {i}: evicted {n_ev[j]}/{want} "
                               f"unmet {unmet[j]}/{tr.budget_unmet}")
            self.evictions += int(want > 0)
            self.unmet_steps += int(tr.budget_unmet)
            if self.replays:
                self._check_eviction(t, i, rtr[i], want)
            if i in self.oracles and self.evict:
                rec = self.oracles[i].evict(self.budgets[i], self.window, self.oracle_rule)
                assert rec.n_evicted == want
        if self.rebuild:
            self.oracles = {}

    def _check_eviction(self, t, i, rt, want):
        """The device's mask and compaction indices of this step's eviction, and
        the rows moved into the kept region, against the oracle's replay."""
        a2t = self.a2t
        if rt.n_pre - rt.n_post != want:
            raise Mismatch(f"{self.label} step {t} stream {i}: replays disagree")
        moved = a2t.a2t_stream_info_get(self.cache, i)["moved_total"]
        if moved - self.moved[i] != rt.settled:
            raise Mismatch(f"{self.label} step {t} stream {i}: moved {moved - self.moved[i]} rows "
                           f"into the kept region, oracle {rt.settled}")
        self.moved[i] = moved
        if want == 0:
            return
        n_pre, mask, slot = a2t.a2t_read_last_evict(self.cache, i)
        if n_pre != rt.n_pre or not np.array_equal(mask.astype(bool), rt.evict_mask) \
                or not np.array_equal(slot, rt.new_slot):
            raise Mismatch(f"{self.label} step {t} stream {i}: eviction mask / compaction "
                           f"indices differ from the oracle")
        self.mask_checks += 1

    def _check_attention(self, t, layer, act, offs, vals, o):
        og = None
        j = self.layers_checked.index(layer)
        for (i, st), off in zip(act, offs):
            if i not in vals or i not in self.oracles:
                continue
            if og is None:
                og = o.to(self.torch.float32).cpu().numpy()
            want = self.oracles[i].attention(layer, vals[i]["q"][j], st.n)
            err = float(np.abs(og[off:off + st.n] - want).max())
            self.max_err = max(self.max_err, err)
            self.attn_checks += 1
            if not err <= self.tol:
                raise Mismatch(f"{self.label} step {t} stream {i} layer {layer}: attention max "
                               f"err {err}")

    # ------------------------------------------------------------ whole run
    def run(self, progress_every=100):
        t_start = time.perf_counter()
        for t in range(self.T):
            self.step(t)
            if progress_every and (t + 1) % progress_every == 0:
                print(f"[{self.label}] global step {t + 1}/{self.T}, "
                      f"{time.perf_counter() - t_start:.1f} s", flush=True)
        self.final_checks()
        return self

    def final_checks(self):
        a2t = self.a2t
        for i, tr in enumerate(self.traces):
            p, s, u = a2t.a2t_read_layout(self.cache, i)
            if not (np.array_equal(p, tr.pos) and np.array_equal(s, tr.seg)
                    and np.array_equal(u, tr.unit)):
                raise Mismatch(f"{self.label} stream {i}: final layout differs")
            peak = a2t.a2t_stream_info_get(self.cache, i)["peak"]
            if peak != tr.peak:
                raise Mismatch(f"{self.label} stream {i}: peak {peak} vs {tr.peak}")
        if self.rebuild:
            from oracle.replay import resume
            self.oracles = {i: resume(self.cfg, self.seed, self.specs[i], self.budgets[i],
                                      self.window, len(self.specs[i].steps), self.layers_checked,
                                      evict=self.evict, values=self.kept_vals[i].__getitem__)
                            for i in self.sampled}
        for i, o in self.oracles.items():
            for layer in self.layers_checked:
                k, v = a2t.a2t_read_kv(self.cache, layer, i)
                kf, vf = bf16_bits_to_f32(k), bf16_bits_to_f32(v)
                if kf.shape != o.k[layer].shape:
                    raise Mismatch(f"{self.label} stream {i} layer {layer}: K shape "
                                   f"{kf.shape} vs {o.k[layer].shape}")
                # stored keys: bf16 rounding of the fp64-rotated key (one rounding)
                if not np.all(np.abs(kf - o.k[layer]) <= np.abs(o.k[layer]) * 2.0 ** -8 + 1e-6):
                    raise Mismatch(f"{self.label} stream {i} layer {layer}: stored K differs")
                if not np.array_equal(vf, o.v[layer]):
                    raise Mismatch(f"{self.label} stream {i} layer {layer}: stored V differs")
