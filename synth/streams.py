"""Seeded stream generator shaped like the paper's duplex sessions.

Shape of a session (Sec. 1 and Sec. 3.1 of the paper): audio arrives in
one-second units; each unit holds about 17 acoustic/structural positions and
its transcript segment about 3 text positions, opened and closed by the two
ASR delimiter tokens, with at most 64 transcript tokens per segment.

Per unit this generator emits, in order: 17 ACOUSTIC rows, one DELIM row,
t TEXT rows, one DELIM row, with t = min(Poisson(3), 64).  Positions are
consecutive integers from 0 within a stream, so they are strictly increasing;
unit ids count units from 0.  A decode (speaking) step appends a single
RESPONSE row carrying the id of the last listened unit.

Randomness (numpy PCG64):
  * structure: one ``default_rng(seed)``; for the varlen workload it first
    draws every stream's length, start offset and budget, then, stream by
    stream, the per-unit transcript lengths;
  * values: a child ``default_rng([seed, stream, step_key, layer])`` per
    (stream, step, layer) draws Q ``[n][Hq][D]``, K ``[n][Hkv][D]`` and
    V ``[n][Hkv][D]`` from N(0, 1) in float32, in that order, so any slice
    can be regenerated alone.  ``step_key`` is the unit index for listening
    units and ``n_units + d`` for the d-th decode step.  For bf16 workloads
    each value is rounded to bfloat16 with round-to-nearest-even.

Nothing here implements the method: no rotary embedding, attention or
eviction arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

SEG_PREFIX = 0
SEG_ACOUSTIC = 1
SEG_DELIM = 2
SEG_TEXT = 3
SEG_RESPONSE = 4
SEG_NAMES = {SEG_PREFIX: "PREFIX", SEG_ACOUSTIC: "ACOUSTIC", SEG_DELIM: "DELIM",
             SEG_TEXT: "TEXT", SEG_RESPONSE: "RESPONSE"}


@dataclass(frozen=True)
class WorkloadConfig:
    index: int
    name: str
    n_layers: int
    n_streams: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str                 # "f32" or "bf16": storage type of Q, K, V, O
    units: int                 # units per stream (upper bound when varlen)
    budget: int                # resident-row budget B
    window: int                # recent acoustic window W, in units
    decode_steps: int = 0      # speaking-phase single-row steps after the units
    rope_theta: float = 1.0e6
    acoustic_rows: int = 17
    text_mean: float = 3.0
    text_cap: int = 64
    varlen: bool = False       # stream lengths / offsets / budgets drawn per stream
    min_units: int = 0
    budget_choices: tuple = ()
    control: bool = False      # also run a no-eviction control of every stream

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.head_dim))

    @property
    def max_unit_rows(self) -> int:
        return self.acoustic_rows + 2 + self.text_cap

    @property
    def row_bytes(self) -> int:
        """Bytes of one cached row (K and V, all KV heads) in one layer."""
        elt = 4 if self.dtype == "f32" else 2
        return 2 * self.n_kv_heads * self.head_dim * elt


CONFIGS: Dict[int, WorkloadConfig] = {
    0: WorkloadConfig(0, "tiny: 1 layer, 1 stream, 4/1 heads, D64, fp32, 60 units, B256, W3",
                      n_layers=1, n_streams=1, n_q_heads=4, n_kv_heads=1, head_dim=64,
                      dtype="f32", units=60, budget=256, window=3),
    1: WorkloadConfig(1, "ten-minute single stream: 36 layers, 32/8 heads, D128, bf16, "
                         "600 units, B4096, W30",
                      n_layers=36, n_streams=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                      dtype="bf16", units=600, budget=4096, window=30),
    2: WorkloadConfig(2, "batched listening: 32 streams of 60-600 units, random start, "
                         "B in {2048,4096}, W30",
                      n_layers=36, n_streams=32, n_q_heads=32, n_kv_heads=8, head_dim=128,
                      dtype="bf16", units=600, budget=4096, window=30, varlen=True,
                      min_units=60, budget_choices=(2048, 4096)),
    3: WorkloadConfig(3, "speaking-phase decode: 64 streams, 600-unit fill, 200 decode steps, "
                         "B4096, W30",
                      n_layers=36, n_streams=64, n_q_heads=32, n_kv_heads=8, head_dim=128,
                      dtype="bf16", units=600, budget=4096, window=30, decode_steps=200),
    4: WorkloadConfig(4, "hour-long sessions: 16 streams x 3600 units, B8192, W60, "
                         "with a no-eviction control",
                      n_layers=36, n_streams=16, n_q_heads=32, n_kv_heads=8, head_dim=128,
                      dtype="bf16", units=3600, budget=8192, window=60, control=True),
}


@dataclass
class UnitSpec:
    """One step of one stream: a listening unit (or its prefill chunk) or a
    single decode row.  ``evict``: the eviction check runs after this step
    (after every step of a listening workload; in the side-channel cadence
    once per duplex unit, after its closing delimiter)."""
    unit: int                 # unit id carried by every row of the step
    key: int                  # value-generator step key
    seg: np.ndarray           # uint8 [n]
    pos: np.ndarray           # int32 [n]
    decode: bool = False
    evict: bool = True

    @property
    def n(self) -> int:
        return int(self.seg.shape[0])


@dataclass
class StreamSpec:
    stream: int
    budget: int
    offset: int               # global step at which the stream's first unit runs
    steps: List[UnitSpec] = field(default_factory=list)

    @property
    def n_units(self) -> int:
        return sum(1 for s in self.steps if not s.decode)

    def total_rows(self) -> int:
        return sum(s.n for s in self.steps)


@dataclass
class Workload:
    config: WorkloadConfig
    seed: int
    streams: List[StreamSpec]

    def global_steps(self) -> int:
        return max(s.offset + len(s.steps) for s in self.streams)

    def active(self, t: int):
        """(stream, step spec) pairs that run at global step t."""
        out = []
        for s in self.streams:
            k = t - s.offset
            if 0 <= k < len(s.steps):
                out.append((s, s.steps[k]))
        return out


def _unit_rows(acoustic: int, t: int) -> np.ndarray:
    return np.concatenate([
        np.full(acoustic, SEG_ACOUSTIC, np.uint8),
        np.array([SEG_DELIM], np.uint8),
        np.full(t, SEG_TEXT, np.uint8),
        np.array([SEG_DELIM], np.uint8),
    ])


def make_workload(cfg: WorkloadConfig | int, seed: Optional[int] = None,
                  units: Optional[int] = None, n_streams: Optional[int] = None,
                  decode_steps: Optional[int] = None) -> Workload:
    """Draw the structure of every stream of a workload.

    ``seed`` defaults to the workload index.  ``units``/``n_streams``/
    ``decode_steps`` truncate the workload (same draws, fewer of them are
    used) for cheaper test slices; the draws for the included streams and
    units are identical to the full workload's.
    """
    if isinstance(cfg, int):
        cfg = CONFIGS[cfg]
    if seed is None:
        seed = cfg.index
    rng = np.random.default_rng(seed)
    S = cfg.n_streams
    if cfg.varlen:
        lengths = rng.integers(cfg.min_units, cfg.units + 1, size=S)
        offsets = np.array([rng.integers(0, cfg.units - int(L) + 1) for L in lengths])
        budgets = rng.choice(np.array(cfg.budget_choices), size=S)
    else:
        lengths = np.full(S, cfg.units)
        offsets = np.zeros(S, np.int64)
        budgets = np.full(S, cfg.budget)
    texts = [np.minimum(rng.poisson(cfg.text_mean, size=int(L)), cfg.text_cap) for L in lengths]

    n_keep = S if n_streams is None else min(n_streams, S)
    n_dec = cfg.decode_steps if decode_steps is None else decode_steps
    streams = []
    for s in range(n_keep):
        L = int(lengths[s]) if units is None else min(int(lengths[s]), units)
        pos = 0
        steps = []
        for u in range(L):
            seg = _unit_rows(cfg.acoustic_rows, int(texts[s][u]))
            p = np.arange(pos, pos + seg.shape[0], dtype=np.int32)
            pos += seg.shape[0]
            steps.append(UnitSpec(unit=u, key=u, seg=seg, pos=p))
        for d in range(n_dec):
            steps.append(UnitSpec(unit=L - 1, key=int(lengths[s]) + d,
                                  seg=np.array([SEG_RESPONSE], np.uint8),
                                  pos=np.array([pos], np.int32), decode=True))
            pos += 1
        streams.append(StreamSpec(stream=s, budget=int(budgets[s]), offset=int(offsets[s]),
                                  steps=steps))
    return Workload(config=cfg, seed=seed, streams=streams)


def make_sessions(cfg: WorkloadConfig | int, seeds: Sequence[int],
                  units: Optional[int] = None) -> Workload:
    """Independent single-stream sessions, one per seed (stream i is the first
    stream of ``make_workload(cfg, seed=seeds[i])``), batched as one workload:
    the budget sweep of the ablation runs several sessions per budget."""
    if isinstance(cfg, int):
        cfg = CONFIGS[cfg]
    streams = []
    for i, sd in enumerate(seeds):
        st = make_workload(cfg, seed=sd, units=units, n_streams=1).streams[0]
        streams.append(StreamSpec(stream=i, budget=st.budget, offset=0, steps=st.steps))
    return Workload(config=cfg, seed=int(seeds[0]) if len(seeds) else 0, streams=streams)


CADENCE_KEY_STRIDE = 80   # value keys of unit u's steps: u * 80 + 0 .. 66


def make_cadence_workload(cfg: WorkloadConfig | int, seed: Optional[int] = None,
                          units: Optional[int] = None,
                          n_streams: Optional[int] = None) -> Workload:
    """The same sessions as ``make_workload`` (same draws, same rows and
    positions), delivered in the side channel's call pattern (Sec. 3.1): per
    duplex unit one prefill chunk of its acoustic/structural rows, then one
    decode step per side-channel token -- the opening delimiter, the t
    transcript tokens and the closing delimiter (a forced close at the 64-token
    cap is the same row).  Every row keeps its unit id; the eviction check runs
    once per unit, after the closing delimiter."""
    base = make_workload(cfg, seed=seed, units=units, n_streams=n_streams, decode_steps=0)
    streams = []
    for s in base.streams:
        steps = []
        for st in s.steps:
            a = int(np.sum(st.seg == SEG_ACOUSTIC))
            k0 = st.unit * CADENCE_KEY_STRIDE
            steps.append(UnitSpec(unit=st.unit, key=k0, seg=st.seg[:a].copy(),
                                  pos=st.pos[:a].copy(), evict=False))
            for r in range(a, st.n):
                steps.append(UnitSpec(unit=st.unit, key=k0 + 1 + (r - a), seg=st.seg[r:r + 1].copy(),
                                      pos=st.pos[r:r + 1].copy(), decode=True,
                                      evict=(r == st.n - 1)))
        streams.append(StreamSpec(stream=s.stream, budget=s.budget, offset=s.offset, steps=steps))
    return Workload(config=base.config, seed=base.seed, streams=streams)


def tiny_stream(units: Sequence[Sequence[int]], prefix: int = 0, start_pos: int = 0,
                pos_gap: int = 0) -> StreamSpec:
    """A hand-shaped stream for tests.

    ``units`` lists, per unit, the segment class of each row.  ``prefix``
    PREFIX rows (unit id -1) come first.  ``pos_gap`` inserts that many
    unused positions between steps (positions only need to increase).
    """
    steps = []
    pos = start_pos
    if prefix:
        seg = np.full(prefix, SEG_PREFIX, np.uint8)
        steps.append(UnitSpec(unit=-1, key=10_000_000, seg=seg,
                              pos=np.arange(pos, pos + prefix, dtype=np.int32)))
        pos += prefix + pos_gap
    u = 0
    for rows in units:
        seg = np.asarray(rows, np.uint8)
        decode = bool(seg.shape[0] == 1 and seg[0] == SEG_RESPONSE)
        unit = u - 1 if decode else u
        steps.append(UnitSpec(unit=unit, key=len(steps), seg=seg,
                              pos=np.arange(pos, pos + seg.shape[0], dtype=np.int32),
                              decode=decode))
        pos += seg.shape[0] + pos_gap
        if not decode:
            u += 1
    return StreamSpec(stream=0, budget=0, offset=0, steps=steps)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).reshape(np.shape(x))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bfloat16-exact."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (u >> 16).astype(np.uint16)


def step_values(cfg: WorkloadConfig, seed: int, stream: int, key: int, n: int,
                layers: Sequence[int]) -> Dict[str, np.ndarray]:
    """Q, K, V of one step for the given layers, float32 ``[len(layers)][n][H][D]``.

    Values are bf16-exact for bf16 workloads.
    """
    Hq, Hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    q = np.empty((len(layers), n, Hq, D), np.float32)
    k = np.empty((len(layers), n, Hkv, D), np.float32)
    v = np.empty((len(layers), n, Hkv, D), np.float32)
    for i, layer in enumerate(layers):
        g = np.random.default_rng([seed, stream, key, layer])
        q[i] = g.standard_normal((n, Hq, D), dtype=np.float32)
        k[i] = g.standard_normal((n, Hkv, D), dtype=np.float32)
        v[i] = g.standard_normal((n, Hkv, D), dtype=np.float32)
    if cfg.dtype == "bf16":
        q, k, v = bf16_round(q), bf16_round(k), bf16_round(v)
    return {"q": q, "k": k, "v": v}
