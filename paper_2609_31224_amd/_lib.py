"""ctypes binding of libA2T (include/a2t.h): the same calls, argument marshalling only.

Every step of the KV path runs in the library's HIP kernels.  If libA2T.so is
not built this module raises ImportError; there is no fallback.

Device buffers are torch tensors on the GPU (contiguous, the cache dtype:
torch.float32 or torch.bfloat16) or raw integer device addresses.  Host arrays
are anything numpy can turn into a contiguous array of the right type.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libA2T.so")

A2T_OK = 0
A2T_ERR_INVALID = -1
A2T_ERR_POS = -2
A2T_ERR_CAPACITY = -3
A2T_ERR_STATE = -4
A2T_ERR_OOM = -5
A2T_ERR_HIP = -6
A2T_ERR_NODEV = -7
A2T_F32 = 0
A2T_BF16 = 1
A2T_ALL_LAYERS = -1
A2T_FLAG_HOST_ONLY = 1
A2T_FLAG_NO_WORKSPACE = 2
A2T_RULE_UNIT, A2T_RULE_ROW, A2T_RULE_SINK_RECENT = 0, 1, 2
SEG_PREFIX, SEG_ACOUSTIC, SEG_DELIM, SEG_TEXT, SEG_RESPONSE = 0, 1, 2, 3, 4

EXPORTED = (
    "a2t_cache_create", "a2t_cache_destroy", "a2t_set_stream", "a2t_append",
    "a2t_chunk_attn", "a2t_append_attn", "a2t_append_attn_noalloc", "a2t_decode_attn",
    "a2t_evict", "a2t_evict_rule", "a2t_dev_begin", "a2t_dev_end", "a2t_dev_open",
    "a2t_dev_append_attn", "a2t_dev_evict", "a2t_dev_evict_rule",
    "a2t_stream_info_get", "a2t_resident",
    "a2t_read_layout", "a2t_read_last_evict", "a2t_read_kv", "a2t_sync",
    "a2t_profile_enable", "a2t_kernel_time", "a2t_profile_reserve", "a2t_status_str",
    "a2t_abi_version", "a2t_distill_create", "a2t_distill_destroy", "a2t_distill_loss",
    "a2t_distill_profile_enable", "a2t_distill_profile_reserve", "a2t_distill_kernel_time",
)
A2T_ROW_NONE, A2T_ROW_ASR, A2T_ROW_NATIVE = 0, 1, 2


class a2t_config(C.Structure):
    _fields_ = [
        ("n_layers", C.c_int32), ("n_streams", C.c_int32), ("n_q_heads", C.c_int32),
        ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("dtype", C.c_int32),
        ("unit_rows", C.c_int32), ("kept_rows", C.c_int32), ("max_step_rows", C.c_int32),
        ("flags", C.c_uint32), ("rope_theta", C.c_double), ("attn_scale", C.c_double),
        ("device", C.c_int32), ("reserved", C.c_int32), ("k_pool", C.c_void_p),
        ("v_pool", C.c_void_p),
    ]


class a2t_stream_info(C.Structure):
    _fields_ = [
        ("resident", C.c_int32), ("peak", C.c_int32), ("kept", C.c_int32), ("ring", C.c_int32),
        ("ring_head", C.c_int32), ("cur_unit", C.c_int32), ("last_evicted_unit", C.c_int32),
        ("step_rows", C.c_int32), ("last_pos", C.c_int64), ("evicted_total", C.c_int64),
        ("moved_total", C.c_int64), ("budget_unmet", C.c_int32), ("last_evict_pre", C.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2609_31224_amd/build.py`")
    # torch ships its own HIP runtime and loads it under the unversioned name.
    # Loading torch first lets libA2T's libamdhip64.so.7 dependency resolve,
    # by SONAME, to that same runtime: one HIP/HSA runtime per process, so
    # torch's device pointers and streams are valid in libA2T.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = C.CDLL(LIB_PATH)
    P, I32, VP = C.POINTER, C.c_int32, C.c_void_p
    sig = {
        "a2t_cache_create": (C.c_int, [P(a2t_config), VP, P(VP)]),
        "a2t_cache_destroy": (C.c_int, [VP]),
        "a2t_set_stream": (C.c_int, [VP, VP]),
        "a2t_append": (C.c_int, [VP, I32, I32, P(I32), P(I32), VP, VP, P(C.c_uint8), P(I32), P(I32)]),
        "a2t_chunk_attn": (C.c_int, [VP, I32, I32, P(I32), P(I32), VP, VP]),
        "a2t_append_attn": (C.c_int, [VP, I32, I32, P(I32), P(I32), VP, VP, P(C.c_uint8), P(I32),
                                      P(I32), P(I32), VP, VP]),
        "a2t_append_attn_noalloc": (C.c_int, [VP, I32, I32, P(I32), P(I32), VP, VP, P(C.c_uint8),
                                              P(I32), P(I32), P(I32), VP, VP]),
        "a2t_decode_attn": (C.c_int, [VP, I32, I32, P(I32), VP, VP]),
        "a2t_evict": (C.c_int, [VP, I32, P(I32), P(I32), I32, P(I32), P(C.c_uint8)]),
        "a2t_evict_rule": (C.c_int, [VP, I32, P(I32), P(I32), I32, I32, I32, P(I32),
                                     P(C.c_uint8)]),
        "a2t_dev_begin": (C.c_int, [VP]),
        "a2t_dev_end": (C.c_int, [VP]),
        "a2t_dev_open": (C.c_int, [VP, I32, P(I32), VP, VP, VP, VP]),
        "a2t_dev_append_attn": (C.c_int, [VP, I32, VP, VP, VP, VP]),
        "a2t_dev_evict": (C.c_int, [VP, VP, I32, VP, VP]),
        "a2t_dev_evict_rule": (C.c_int, [VP, VP, I32, I32, I32, VP, VP]),
        "a2t_stream_info_get": (C.c_int, [VP, I32, P(a2t_stream_info)]),
        "a2t_resident": (C.c_int, [VP, I32, P(C.c_int32), P(C.c_int32)]),
        "a2t_read_layout": (C.c_int, [VP, I32, P(I32), P(C.c_uint8), P(I32)]),
        "a2t_read_last_evict": (C.c_int, [VP, I32, P(I32), P(C.c_uint8), P(I32)]),
        "a2t_read_kv": (C.c_int, [VP, I32, I32, VP, VP]),
        "a2t_sync": (C.c_int, [VP]),
        "a2t_profile_enable": (C.c_int, [VP, C.c_char_p]),
        "a2t_kernel_time": (C.c_int, [VP, C.c_char_p, P(C.c_int64), P(C.c_double)]),
        "a2t_profile_reserve": (C.c_int, [VP, I32]),
        "a2t_status_str": (C.c_char_p, [C.c_int]),
        "a2t_abi_version": (C.c_int, []),
        "a2t_distill_create": (C.c_int, [I32, I32, I32, I32, I32, VP, P(VP)]),
        "a2t_distill_destroy": (C.c_int, [VP]),
        "a2t_distill_loss": (C.c_int, [VP, I32, VP, C.c_int64, VP, C.c_int64, P(C.c_int8), P(I32),
                                       P(C.c_int8), P(C.c_int8), C.c_float, VP, VP]),
        "a2t_distill_profile_enable": (C.c_int, [VP, I32]),
        "a2t_distill_profile_reserve": (C.c_int, [VP, I32]),
        "a2t_distill_kernel_time": (C.c_int, [VP, P(C.c_int64), P(C.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()


class A2TError(RuntimeError):
    def __init__(self, status: int, call: str):
        self.status = status
        super().__init__(f"{call}: {a2t_status_str(status)} ({status})")


def _check(rc: int, call: str) -> None:
    if rc != A2T_OK:
        raise A2TError(rc, call)


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x), dtype=np.int32)


def _u8(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x), dtype=np.uint8)


def _p(arr: Optional[np.ndarray], ctype):
    if arr is None:
        return None
    return arr.ctypes.data_as(C.POINTER(ctype))


def _dev(x, what: str, dtype=None) -> Optional[int]:
    """Device address of a torch tensor (validated) or a raw integer address."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    import torch
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"{what}: expected a GPU torch tensor or a device address")
    if not x.is_cuda:
        raise ValueError(f"{what}: tensor must live on the GPU")
    if not x.is_contiguous():
        raise ValueError(f"{what}: tensor must be contiguous")
    if dtype is not None and x.dtype != dtype:
        raise ValueError(f"{what}: dtype {x.dtype}, cache uses {dtype}")
    return x.data_ptr()


@dataclass
class Cache:
    """Handle returned by a2t_cache_create (plus what marshalling needs)."""
    ptr: C.c_void_p
    config: a2t_config

    @property
    def torch_dtype(self):
        import torch
        return torch.float32 if self.config.dtype == A2T_F32 else torch.bfloat16


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def a2t_abi_version() -> int:
    return _lib.a2t_abi_version()


def a2t_status_str(status: int) -> str:
    return _lib.a2t_status_str(status).decode()


def a2t_cache_create(n_layers: int, n_streams: int, n_q_heads: int, n_kv_heads: int,
                     head_dim: int, dtype: int, unit_rows: int, kept_rows: int,
                     max_step_rows: int, flags: int = 0, rope_theta: float = 0.0,
                     attn_scale: float = 0.0, device: int = 0, stream=None,
                     k_pool=None, v_pool=None) -> Cache:
    """``k_pool``/``v_pool``: optional caller-owned device pools (torch tensors or
    addresses) of L*S*Hkv*(unit_rows+kept_rows)*D elements each; the caller keeps
    them alive until a2t_cache_destroy."""
    cfg = a2t_config(n_layers, n_streams, n_q_heads, n_kv_heads, head_dim, dtype, unit_rows,
                     kept_rows, max_step_rows, flags, rope_theta, attn_scale, device, 0,
                     _dev(k_pool, "k_pool"), _dev(v_pool, "v_pool"))
    out = C.c_void_p()
    _check(_lib.a2t_cache_create(C.byref(cfg), _stream_handle(stream), C.byref(out)),
           "a2t_cache_create")
    return Cache(out, cfg)


def a2t_cache_destroy(c: Cache) -> None:
    if c.ptr:
        _check(_lib.a2t_cache_destroy(c.ptr), "a2t_cache_destroy")
        c.ptr = C.c_void_p()


def a2t_set_stream(c: Cache, stream) -> None:
    _check(_lib.a2t_set_stream(c.ptr, _stream_handle(stream)), "a2t_set_stream")


def a2t_append(c: Cache, layer: int, stream_ids: Sequence[int], n_rows: Sequence[int], k, v,
               seg=None, pos=None, unit_id=None) -> None:
    ids, nr = _i32(stream_ids), _i32(n_rows)
    if ids.shape != nr.shape:
        raise ValueError("stream_ids and n_rows differ in length")
    sg = None if seg is None else _u8(seg)
    ps = None if pos is None else _i32(pos)
    un = None if unit_id is None else _i32(unit_id)
    dt = c.torch_dtype if not isinstance(k, (int, type(None))) else None
    rc = _lib.a2t_append(c.ptr, layer, len(ids), _p(ids, C.c_int32), _p(nr, C.c_int32),
                         _dev(k, "k", dt), _dev(v, "v", dt), _p(sg, C.c_uint8),
                         _p(ps, C.c_int32), _p(un, C.c_int32))
    _check(rc, "a2t_append")


def a2t_chunk_attn(c: Cache, layer: int, stream_ids: Sequence[int], n_q: Sequence[int], q, o) -> None:
    ids, nq = _i32(stream_ids), _i32(n_q)
    if ids.shape != nq.shape:
        raise ValueError("stream_ids and n_q differ in length")
    dt = c.torch_dtype if not isinstance(q, int) else None
    rc = _lib.a2t_chunk_attn(c.ptr, layer, len(ids), _p(ids, C.c_int32), _p(nq, C.c_int32),
                             _dev(q, "q", dt), _dev(o, "o", dt))
    _check(rc, "a2t_chunk_attn")


def _append_attn(fn, name, c, layer, stream_ids, n_rows, k, v, seg, pos, unit_id, n_q, q, o):
    ids, nr, nq = _i32(stream_ids), _i32(n_rows), _i32(n_q)
    if not (ids.shape == nr.shape == nq.shape):
        raise ValueError("stream_ids, n_rows and n_q differ in length")
    sg = None if seg is None else _u8(seg)
    ps = None if pos is None else _i32(pos)
    un = None if unit_id is None else _i32(unit_id)
    dt = c.torch_dtype if not isinstance(k, (int, type(None))) else None
    rc = fn(c.ptr, layer, len(ids), _p(ids, C.c_int32), _p(nr, C.c_int32), _dev(k, "k", dt),
            _dev(v, "v", dt), _p(sg, C.c_uint8), _p(ps, C.c_int32), _p(un, C.c_int32),
            _p(nq, C.c_int32), _dev(q, "q", dt), _dev(o, "o", dt))
    _check(rc, name)


def a2t_append_attn(c: Cache, layer: int, stream_ids: Sequence[int], n_rows: Sequence[int], k, v,
                    seg, pos, unit_id, n_q: Sequence[int], q, o) -> None:
    _append_attn(_lib.a2t_append_attn, "a2t_append_attn", c, layer, stream_ids, n_rows, k, v, seg,
                 pos, unit_id, n_q, q, o)


def a2t_append_attn_noalloc(c: Cache, layer: int, stream_ids: Sequence[int],
                            n_rows: Sequence[int], k, v, seg, pos, unit_id, n_q: Sequence[int],
                            q, o) -> None:
    _append_attn(_lib.a2t_append_attn_noalloc, "a2t_append_attn_noalloc", c, layer, stream_ids,
                 n_rows, k, v, seg, pos, unit_id, n_q, q, o)


def a2t_decode_attn(c: Cache, layer: int, stream_ids: Sequence[int], q, o) -> None:
    ids = _i32(stream_ids)
    dt = c.torch_dtype if not isinstance(q, int) else None
    rc = _lib.a2t_decode_attn(c.ptr, layer, len(ids), _p(ids, C.c_int32), _dev(q, "q", dt),
                              _dev(o, "o", dt))
    _check(rc, "a2t_decode_attn")


def a2t_evict(c: Cache, stream_ids: Sequence[int], budget, window: int) -> Tuple[np.ndarray, np.ndarray]:
    ids = _i32(stream_ids)
    b = _i32(np.broadcast_to(np.asarray(budget), ids.shape))
    n_ev = np.zeros(ids.shape, np.int32)
    unmet = np.zeros(ids.shape, np.uint8)
    rc = _lib.a2t_evict(c.ptr, len(ids), _p(ids, C.c_int32), _p(b, C.c_int32), window,
                        _p(n_ev, C.c_int32), _p(unmet, C.c_uint8))
    _check(rc, "a2t_evict")
    return n_ev, unmet.astype(bool)


def a2t_evict_rule(c: Cache, stream_ids: Sequence[int], budget, window: int, rule: int,
                   n_sink: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    ids = _i32(stream_ids)
    b = _i32(np.broadcast_to(np.asarray(budget), ids.shape))
    n_ev = np.zeros(ids.shape, np.int32)
    unmet = np.zeros(ids.shape, np.uint8)
    rc = _lib.a2t_evict_rule(c.ptr, len(ids), _p(ids, C.c_int32), _p(b, C.c_int32), window, rule,
                             n_sink, _p(n_ev, C.c_int32), _p(unmet, C.c_uint8))
    _check(rc, "a2t_evict_rule")
    return n_ev, unmet.astype(bool)


def a2t_dev_begin(c: Cache) -> None:
    _check(_lib.a2t_dev_begin(c.ptr), "a2t_dev_begin")


def a2t_dev_end(c: Cache) -> None:
    _check(_lib.a2t_dev_end(c.ptr), "a2t_dev_end")


def a2t_dev_open(c: Cache, stream_ids: Sequence[int], n_rows, unit_id, seg, pos) -> None:
    """n_rows, unit_id: device int32 [n]; seg: device uint8 [n][max_step_rows];
    pos: device int32 [n][max_step_rows] (torch tensors or addresses)."""
    ids = _i32(stream_ids)
    rc = _lib.a2t_dev_open(c.ptr, len(ids), _p(ids, C.c_int32), _dev(n_rows, "n_rows"),
                           _dev(unit_id, "unit_id"), _dev(seg, "seg"), _dev(pos, "pos"))
    _check(rc, "a2t_dev_open")


def a2t_dev_append_attn(c: Cache, layer: int, k, v, q, o) -> None:
    dt = c.torch_dtype if not isinstance(k, int) else None
    rc = _lib.a2t_dev_append_attn(c.ptr, layer, _dev(k, "k", dt), _dev(v, "v", dt),
                                  _dev(q, "q", dt), _dev(o, "o", dt))
    _check(rc, "a2t_dev_append_attn")


def a2t_dev_evict(c: Cache, budget, window: int, n_evicted=None, budget_unmet=None) -> None:
    """budget: device int32 [n]; n_evicted (int32), budget_unmet (uint8): optional
    device [n] outputs."""
    rc = _lib.a2t_dev_evict(c.ptr, _dev(budget, "budget"), window, _dev(n_evicted, "n_evicted"),
                            _dev(budget_unmet, "budget_unmet"))
    _check(rc, "a2t_dev_evict")


def a2t_dev_evict_rule(c: Cache, budget, window: int, rule: int, n_sink: int = 0, n_evicted=None,
                       budget_unmet=None) -> None:
    """a2t_dev_evict with an a2t_rule (A2T_RULE_*) and, for the sink rule, the sink count."""
    rc = _lib.a2t_dev_evict_rule(c.ptr, _dev(budget, "budget"), window, rule, n_sink,
                                 _dev(n_evicted, "n_evicted"), _dev(budget_unmet, "budget_unmet"))
    _check(rc, "a2t_dev_evict_rule")


def a2t_stream_info_get(c: Cache, stream: int) -> dict:
    info = a2t_stream_info()
    _check(_lib.a2t_stream_info_get(c.ptr, stream, C.byref(info)), "a2t_stream_info_get")
    return {name: getattr(info, name) for name, _ in a2t_stream_info._fields_}


def a2t_resident(c: Cache, stream: int) -> tuple:
    """(resident rows R, peak R) of one stream."""
    n, peak = C.c_int32(), C.c_int32()
    _check(_lib.a2t_resident(c.ptr, stream, C.byref(n), C.byref(peak)), "a2t_resident")
    return n.value, peak.value


def a2t_read_layout(c: Cache, stream: int):
    n = a2t_stream_info_get(c, stream)["resident"]
    pos = np.zeros(n, np.int32)
    seg = np.zeros(n, np.uint8)
    unit = np.zeros(n, np.int32)
    _check(_lib.a2t_read_layout(c.ptr, stream, _p(pos, C.c_int32), _p(seg, C.c_uint8),
                                _p(unit, C.c_int32)), "a2t_read_layout")
    return pos, seg, unit


def a2t_read_last_evict(c: Cache, stream: int):
    n_pre = C.c_int32()
    _check(_lib.a2t_read_last_evict(c.ptr, stream, C.byref(n_pre), None, None),
           "a2t_read_last_evict")
    mask = np.zeros(n_pre.value, np.uint8)
    slot = np.zeros(n_pre.value, np.int32)
    _check(_lib.a2t_read_last_evict(c.ptr, stream, C.byref(n_pre), _p(mask, C.c_uint8),
                                    _p(slot, C.c_int32)), "a2t_read_last_evict")
    return n_pre.value, mask, slot


def a2t_read_kv(c: Cache, layer: int, stream: int):
    """Resident K (rotated) and V of one layer in cache order.  float32 arrays
    for fp32 caches; for bf16 caches the raw 16-bit patterns (uint16)."""
    n = a2t_stream_info_get(c, stream)["resident"]
    shape = (n, c.config.n_kv_heads, c.config.head_dim)
    dt = np.float32 if c.config.dtype == A2T_F32 else np.uint16
    k = np.zeros(shape, dt)
    v = np.zeros(shape, dt)
    _check(_lib.a2t_read_kv(c.ptr, layer, stream, k.ctypes.data, v.ctypes.data), "a2t_read_kv")
    return k, v


def a2t_sync(c: Cache) -> None:
    _check(_lib.a2t_sync(c.ptr), "a2t_sync")


def a2t_profile_enable(c: Cache, kernel_filter: Optional[str]) -> None:
    arg = None if kernel_filter is None else kernel_filter.encode()
    _check(_lib.a2t_profile_enable(c.ptr, arg), "a2t_profile_enable")


def a2t_kernel_time(c: Cache, kernel: str) -> Tuple[int, float]:
    n = C.c_int64()
    ms = C.c_double()
    _check(_lib.a2t_kernel_time(c.ptr, kernel.encode(), C.byref(n), C.byref(ms)), "a2t_kernel_time")
    return n.value, ms.value


def a2t_profile_reserve(c: Cache, n_launches: int) -> None:
    _check(_lib.a2t_profile_reserve(c.ptr, n_launches), "a2t_profile_reserve")


def raw_lib():
    """The ctypes library with argument types set, for callers that marshal
    their arguments once and call the C entry points directly."""
    return _lib


# ---- adaptation objective (Sec. 3.2)
@dataclass
class Distill:
    """Handle returned by a2t_distill_create."""
    ptr: C.c_void_p
    max_rows: int
    vocab: int
    n_added: int
    dtype: int


def a2t_distill_create(max_rows: int, vocab: int, n_added: int, dtype: int, device: int = 0,
                       stream=None) -> Distill:
    out = C.c_void_p()
    _check(_lib.a2t_distill_create(max_rows, vocab, n_added, dtype, device, _stream_handle(stream),
                                   C.byref(out)), "a2t_distill_create")
    return Distill(out, max_rows, vocab, n_added, dtype)


def a2t_distill_destroy(d: Distill) -> None:
    _check(_lib.a2t_distill_destroy(d.ptr), "a2t_distill_destroy")


def a2t_distill_loss(d: Distill, student, teacher, kind, target, dec_group, turn_group,
                     temperature: float, losses, grad=None) -> None:
    """student / teacher / grad: GPU tensors [n_rows][stride] (rows of the
    extended / teacher vocabulary, strides multiples of 8); kind, target,
    dec_group, turn_group: host arrays [n_rows]; losses: GPU float32 [5]."""
    import torch
    dt = torch.float32 if d.dtype == A2T_F32 else torch.bfloat16
    n = int(student.shape[0])
    kd = np.ascontiguousarray(np.asarray(kind), dtype=np.int8)
    tg = _i32(target)
    dg = np.ascontiguousarray(np.asarray(dec_group), dtype=np.int8)
    tu = np.ascontiguousarray(np.asarray(turn_group), dtype=np.int8)
    if not (kd.shape == tg.shape == dg.shape == tu.shape == (n,)):
        raise ValueError("row metadata must have one entry per row")
    rc = _lib.a2t_distill_loss(d.ptr, n, _dev(student, "student", dt), int(student.stride(0)),
                               _dev(teacher, "teacher", dt), int(teacher.stride(0)),
                               _p(kd, C.c_int8), _p(tg, C.c_int32), _p(dg, C.c_int8),
                               _p(tu, C.c_int8), float(temperature),
                               _dev(losses, "losses", torch.float32), _dev(grad, "grad", dt))
    _check(rc, "a2t_distill_loss")
