"""ctypes binding of libtorpor (include/torpor.h, include/torpor_plan.h).

Argument marshalling only: every step of swap-in and execution runs in the library's
HIP code. The functions keep the C names; failures raise ``TorporError`` carrying the
status code and ``tp_last_error()``. ``Runtime`` is a convenience wrapper that lets
torch allocate the arena and workspace once and passes torch streams through.

The library is loaded from this package directory; if it is missing, importing
``lib()`` raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtorpor.so")
HOST_LIB_PATH = os.path.join(_HERE, "libtorpor_host.so")
PROBE_LIB_PATH = os.path.join(_HERE, "libtorpor_probe.so")

TP_OK, TP_E_INVAL, TP_E_NOENT, TP_E_NOSPC, TP_E_HIP, TP_E_STATE = 0, -1, -2, -3, -4, -5
TP_F32, TP_BF16 = 0, 1
TP_ARCH_MLP, TP_ARCH_RESNET50, TP_ARCH_BERT = 0, 1, 2
TP_ACT = {"none": 0, "relu": 1, "gelu": 2}
TP_COPY_MEMCPY, TP_COPY_GATHER, TP_COPY_PAGEABLE, TP_COPY_ZERO = 0, 1, 2, 3
TP_FLAG_POISON, TP_FLAG_THROTTLE, TP_FLAG_NO_GRAPH, TP_FLAG_SERIAL, TP_FLAG_PER_TENSOR, TP_FLAG_TRACE = 1, 2, 4, 8, 16, 32
TP_FLAG_CALLER_STREAM = 64
TP_FLAG_NO_TOUCH, TP_FLAG_TOUCH_ALWAYS = 128, 256
TP_PLAN_GREEDY, TP_PLAN_COST = 0, 1
TP_EVICT_LRU, TP_EVICT_HEAVINESS, TP_EVICT_LRU_WINDOW = 0, 1, 2
TP_CLASS_AUTO, TP_CLASS_LIGHT, TP_CLASS_HEAVY = 0, 1, 2
TP_ALLOC_FIRST_FIT, TP_ALLOC_PARTITION, TP_ALLOC_PARTITION_CONSOLIDATE = 0, 1, 2
TP_QUEUE_FIFO, TP_QUEUE_SLO = 0, 1
ROLES = {
    "w": 0, "b": 1,
    "tok_emb": 10, "pos_emb": 11, "type_emb": 12, "emb_ln_g": 13, "emb_ln_b": 14,
    "qkv_w": 20, "qkv_b": 21, "o_w": 22, "o_b": 23, "ln1_g": 24, "ln1_b": 25,
    "ffn1_w": 26, "ffn1_b": 27, "ffn2_w": 28, "ffn2_b": 29, "ln2_g": 30, "ln2_b": 31,
}
# transfer group size G (whole layers per chunk, closed once a chunk holds >= G bytes)
DEFAULT_CHUNK = 8 << 20
# cold requests of models up to this size read their weights over the host link directly
# (the swap runs behind them): below it the copy engine's fixed start-up and hand-off
# latency costs more than direct reads
DEFAULT_DIRECT = 2 << 20
ARCHS = {"mlp": TP_ARCH_MLP, "resnet50": TP_ARCH_RESNET50, "bert": TP_ARCH_BERT}
DTYPES = {"f32": TP_F32, "bf16": TP_BF16}


class tp_tensor_desc(C.Structure):
    _fields_ = [("layer", C.c_uint32), ("role", C.c_uint32), ("offset", C.c_uint64), ("bytes", C.c_uint64),
                ("shape", C.c_int64 * 4)]


class tp_model_desc(C.Structure):
    _fields_ = [("arch", C.c_int32), ("dtype", C.c_int32), ("dims", C.c_int32 * 8), ("n_tensors", C.c_uint32),
                ("tensors", C.POINTER(tp_tensor_desc))]


class tp_config(C.Structure):
    _fields_ = [("arena_dev", C.c_void_p), ("arena_bytes", C.c_uint64), ("work_dev", C.c_void_p),
                ("work_bytes", C.c_uint64), ("copy_stream", C.c_void_p), ("chunk_min_bytes", C.c_uint64),
                ("copy_method", C.c_int32), ("gather_wgs", C.c_int32), ("flags", C.c_int32),
                ("throttle_us", C.c_int32), ("copy_streams", C.c_int32), ("direct_max_bytes", C.c_uint64),
                ("plan", C.c_int32), ("plan_batch", C.c_int32), ("link_gbs", C.c_float), ("chunk_us", C.c_float),
                ("evict_policy", C.c_int32), ("heavy_ratio", C.c_float), ("alloc", C.c_int32),
                ("partition_bytes", C.c_uint64)]


class tp_arena_stats_t(C.Structure):
    _fields_ = [("capacity", C.c_uint64), ("used", C.c_uint64), ("largest_free", C.c_uint64),
                ("resident", C.c_uint32), ("registered", C.c_uint32), ("hits", C.c_uint64),
                ("misses", C.c_uint64), ("evictions", C.c_uint64), ("frag_evictions", C.c_uint64),
                ("bytes_swapped", C.c_uint64), ("admit_calls", C.c_uint64), ("admit_ns_total", C.c_uint64),
                ("admit_ns_max", C.c_uint64), ("partitions", C.c_uint32), ("partitions_free", C.c_uint32),
                ("evacuations", C.c_uint64), ("bytes_moved", C.c_uint64), ("graph_captures", C.c_uint64),
                ("graph_repoints", C.c_uint64), ("graph_rebases", C.c_uint64), ("cache_touches", C.c_uint64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class tp_model_info_t(C.Structure):
    _fields_ = [("host_bytes", C.c_uint64), ("param_bytes", C.c_uint64), ("n_chunks", C.c_uint32),
                ("resident", C.c_int32), ("extent_offset", C.c_uint64), ("last_use_clock", C.c_uint64),
                ("heavy", C.c_int32), ("cold_est_us", C.c_float), ("warm_est_us", C.c_float)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class tp_request(C.Structure):
    _fields_ = [("model_id", C.c_int32), ("batch", C.c_int32), ("input_dev", C.c_void_p),
                ("output_dev", C.c_void_p), ("arrival_ns", C.c_uint64)]


class tp_request_result(C.Structure):
    _fields_ = [("issue_ns", C.c_uint64), ("done_ns", C.c_uint64), ("hit", C.c_int32), ("status", C.c_int32),
                ("admit_ns", C.c_uint64)]


class tp_sched_config(C.Structure):
    _fields_ = [("policy", C.c_int32), ("max_inflight", C.c_int32), ("slo_pct", C.c_double), ("alpha", C.c_double),
                ("scalar", C.c_double), ("threshold", C.c_double), ("period_ns", C.c_uint64)]


class tp_sched_stats(C.Structure):
    _fields_ = [("alpha", C.c_double), ("periods", C.c_uint32), ("alpha_changes", C.c_uint32),
                ("compliant", C.c_uint32), ("functions", C.c_uint32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class TorporError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


_P = C.c_void_p
_SIGS = {
    "tp_create": [C.POINTER(tp_config), C.POINTER(_P)],
    "tp_destroy": [_P],
    "tp_register_model": [_P, C.POINTER(tp_model_desc), _P, C.c_uint64, C.POINTER(C.c_int32)],
    "tp_unregister_model": [_P, C.c_int32],
    "tp_infer": [_P, C.c_int32, _P, C.c_int32, _P, _P],
    "tp_infer_noalloc": [_P, C.c_int32, _P, C.c_int32, _P, _P],
    "tp_swap_in": [_P, C.c_int32, _P],
    "tp_evict": [_P, C.c_int32],
    "tp_debug_fail_copy": [_P, C.c_int32],
    "tp_is_resident": [_P, C.c_int32, C.POINTER(C.c_int32)],
    "tp_arena_stats": [_P, C.POINTER(tp_arena_stats_t)],
    "tp_model_info": [_P, C.c_int32, C.POINTER(tp_model_info_t)],
    "tp_set_model_class": [_P, C.c_int32, C.c_int32],
    "tp_model_chunks": [_P, C.c_int32, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64), C.POINTER(C.c_uint32),
                        C.c_uint32, C.POINTER(C.c_uint32)],
    "tp_workspace_bytes": [C.POINTER(tp_model_desc), C.c_int32, C.POINTER(C.c_uint64)],
    "tp_last_timeline": [_P, C.POINTER(C.c_float), C.POINTER(C.c_float), C.POINTER(C.c_float), C.c_uint32,
                         C.POINTER(C.c_uint32), C.POINTER(C.c_float)],
    "tp_model_host_image": [_P, C.c_int32, C.POINTER(_P), C.POINTER(C.c_uint64)],
    "tp_run_trace": [_P, C.POINTER(tp_request), C.c_uint32, _P, C.POINTER(tp_request_result)],
    "tp_run_trace_sched": [_P, C.POINTER(tp_request), C.c_uint32, _P, C.POINTER(tp_sched_config),
                           C.POINTER(C.c_uint64), C.POINTER(tp_request_result), C.POINTER(tp_sched_stats)],
    "tph_rrc": [C.c_uint64, C.c_uint64, C.c_double, C.POINTER(C.c_double)],
    "tph_sched_pick": [C.c_uint32, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64), C.c_double, C.c_double, C.c_uint32,
                       C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_uint8)],
    "tph_alpha_update": [C.c_double, C.c_double, C.c_double, C.c_double, C.c_double, C.POINTER(C.c_double)],
    "tph_validate": [C.POINTER(tp_model_desc), C.c_uint64],
    "tph_touch_span": [C.POINTER(tp_model_desc), C.c_uint64, C.POINTER(C.c_int32), C.POINTER(C.c_uint64),
                       C.POINTER(C.c_uint64)],
    "tph_plan": [C.POINTER(tp_model_desc), C.c_uint64, C.c_uint64, C.c_int32, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                 C.POINTER(C.c_uint32), C.c_uint32, C.POINTER(C.c_uint32)],
    "tph_plan_cost_model": [C.POINTER(tp_model_desc), C.c_uint64, C.c_int32, C.c_float, C.c_float,
                            C.POINTER(C.c_uint64), C.POINTER(C.c_uint64), C.POINTER(C.c_uint32), C.c_uint32,
                            C.POINTER(C.c_uint32), C.POINTER(C.c_double)],
    "tph_plan_cost": [C.POINTER(C.c_uint64), C.POINTER(C.c_double), C.c_uint32, C.c_uint64, C.c_double, C.c_double,
                      C.c_double, C.POINTER(C.c_uint32), C.c_uint32, C.POINTER(C.c_uint32), C.POINTER(C.c_double)],
    "tph_layer_costs": [C.POINTER(tp_model_desc), C.c_uint64, C.c_int32, C.POINTER(C.c_double), C.c_uint32,
                        C.POINTER(C.c_uint32)],
    "tph_arena_create": [C.c_uint64, C.c_uint64, C.POINTER(_P)],
    "tph_arena_destroy": [_P],
    "tph_arena_register": [_P, C.c_int32, C.c_uint64],
    "tph_arena_unregister": [_P, C.c_int32],
    "tph_arena_request": [_P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_uint64), C.POINTER(C.c_int32),
                          C.c_uint32, C.POINTER(C.c_uint32)],
    "tph_arena_evict": [_P, C.c_int32],
    "tph_arena_set_policy": [_P, C.c_int32],
    "tph_arena_set_heavy": [_P, C.c_int32, C.c_int32],
    "tph_arena_set_partitioned": [_P, C.c_uint64, C.c_int32],
    "tph_arena_steps": [_P, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_uint64),
                        C.POINTER(C.c_uint64), C.c_uint32, C.POINTER(C.c_uint32)],
    "tph_arena_stats": [_P, C.POINTER(tp_arena_stats_t)],
}
HOST_ONLY = [n for n in _SIGS if n.startswith("tph_")]

_lib = None
_host = None


def _bind(lib, names):
    for n in names:
        f = getattr(lib, n)
        f.argtypes = _SIGS[n]
        f.restype = C.c_int32
    lib.tp_last_error.argtypes = []
    lib.tp_last_error.restype = C.c_char_p
    return lib


def lib():
    """The HIP library. torch is imported first so both share torch's HIP runtime."""
    global _lib
    if _lib is None:
        import torch  # noqa: F401  (loads the HIP runtime the library binds to)
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2306_03622_amd.build")
        _lib = _bind(C.CDLL(LIB_PATH), list(_SIGS))
    return _lib


def host_lib():
    """The host-only planning library (same tph_* calls, built without HIP)."""
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB_PATH):
            raise ImportError(f"{HOST_LIB_PATH} is not built; run python -m paper_2306_03622_amd.build")
        _host = _bind(C.CDLL(HOST_LIB_PATH), HOST_ONLY)
    return _host


def _check(L, status):
    if status != TP_OK:
        raise TorporError(status, L.tp_last_error().decode())


def _ptr(x):
    """Device or host address of a torch tensor, an int or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "cuda_stream"):
        return x.cuda_stream
    raise TypeError(type(x))


# ------------------------------------------------------------------ descriptors

class ModelDesc:
    """Owns a tp_model_desc and its tensor table.

    tensors: iterable of (layer, role name, offset, nbytes, shape).
    """

    def __init__(self, arch: str, dtype: str, dims, tensors):
        self.tensors = list(tensors)
        self._arr = (tp_tensor_desc * len(self.tensors))()
        for i, (layer, role, off, nb, shape) in enumerate(self.tensors):
            t = self._arr[i]
            t.layer, t.role, t.offset, t.bytes = layer, ROLES[role], off, nb
            for k, s in enumerate(tuple(shape)[:4]):
                t.shape[k] = s
        self.desc = tp_model_desc()
        self.desc.arch = ARCHS[arch]
        self.desc.dtype = DTYPES[dtype]
        for k, v in enumerate(list(dims)[:8]):
            self.desc.dims[k] = int(v)
        self.desc.n_tensors = len(self.tensors)
        self.desc.tensors = self._arr

    @classmethod
    def of(cls, model):
        """From any object with arch, dtype, dims and tensors(layer, role, offset, nbytes, shape)."""
        d = model.dims
        if model.arch == "mlp":
            dims = [d["layers"], d["width"], TP_ACT[d["act"]]]
        elif model.arch == "resnet50":
            dims = [d["classes"], d["image"]]
        else:
            dims = [d["layers"], d["d"], d["heads"], d["ffn"], d["seq"], d["vocab"], d["maxpos"]]
        return cls(model.arch, model.dtype, dims,
                   [(t.layer, t.role, t.offset, t.nbytes, t.shape) for t in model.tensors])


# ------------------------------------------------------------------ C calls

def tp_create(arena_dev, arena_bytes, work_dev, work_bytes, copy_stream=None, chunk_min_bytes=DEFAULT_CHUNK,
              copy_method=TP_COPY_MEMCPY, gather_wgs=0, flags=0, throttle_us=0, copy_streams=0, direct_max_bytes=0,
              plan=TP_PLAN_GREEDY, plan_batch=0, link_gbs=0.0, chunk_us=0.0, evict_policy=TP_EVICT_LRU,
              heavy_ratio=0.0, alloc=TP_ALLOC_FIRST_FIT, partition_bytes=0):
    L = lib()
    cfg = tp_config(_ptr(arena_dev), arena_bytes, _ptr(work_dev), work_bytes, _ptr(copy_stream), chunk_min_bytes,
                    copy_method, gather_wgs, flags, throttle_us, copy_streams, direct_max_bytes, plan, plan_batch,
                    link_gbs, chunk_us, evict_policy, heavy_ratio, alloc, partition_bytes)
    ctx = _P()
    _check(L, L.tp_create(C.byref(cfg), C.byref(ctx)))
    return ctx


def tp_destroy(ctx):
    _check(lib(), lib().tp_destroy(ctx))


def tp_register_model(ctx, desc: ModelDesc, host_weights: np.ndarray) -> int:
    buf = np.ascontiguousarray(host_weights).view(np.uint8)
    mid = C.c_int32()
    _check(lib(), lib().tp_register_model(ctx, C.byref(desc.desc), buf.ctypes.data, buf.nbytes, C.byref(mid)))
    return mid.value


def tp_unregister_model(ctx, model_id):
    _check(lib(), lib().tp_unregister_model(ctx, model_id))


def tp_infer(ctx, model_id, input_dev, batch, output_dev, stream=None):
    _check(lib(), lib().tp_infer(ctx, model_id, _ptr(input_dev), batch, _ptr(output_dev), _ptr(stream)))


def tp_infer_noalloc(ctx, model_id, input_dev, batch, output_dev, stream=None):
    _check(lib(), lib().tp_infer_noalloc(ctx, model_id, _ptr(input_dev), batch, _ptr(output_dev), _ptr(stream)))


def tp_swap_in(ctx, model_id, stream=None):
    _check(lib(), lib().tp_swap_in(ctx, model_id, _ptr(stream)))


def tp_evict(ctx, model_id):
    _check(lib(), lib().tp_evict(ctx, model_id))


def tp_debug_fail_copy(ctx, nth: int):
    _check(lib(), lib().tp_debug_fail_copy(ctx, nth))


def tp_is_resident(ctx, model_id) -> bool:
    r = C.c_int32()
    _check(lib(), lib().tp_is_resident(ctx, model_id, C.byref(r)))
    return bool(r.value)


def tp_arena_stats(ctx) -> dict:
    s = tp_arena_stats_t()
    _check(lib(), lib().tp_arena_stats(ctx, C.byref(s)))
    return s.as_dict()


def tp_model_info(ctx, model_id) -> dict:
    s = tp_model_info_t()
    _check(lib(), lib().tp_model_info(ctx, model_id, C.byref(s)))
    return s.as_dict()


def tp_set_model_class(ctx, model_id, model_class):
    _check(lib(), lib().tp_set_model_class(ctx, model_id, model_class))


def tp_model_chunks(ctx, model_id):
    L = lib()
    n = C.c_uint32()
    _check(L, L.tp_model_chunks(ctx, model_id, None, None, None, 0, C.byref(n)))
    b, e, f = (C.c_uint64 * n.value)(), (C.c_uint64 * n.value)(), (C.c_uint32 * n.value)()
    _check(L, L.tp_model_chunks(ctx, model_id, b, e, f, n.value, C.byref(n)))
    return [{"begin": b[i], "end": e[i], "first_layer": f[i]} for i in range(n.value)]


def tp_last_timeline(ctx):
    """Per-chunk copy begin/end and wait-passed times (ms) of the last traced cold request."""
    L = lib()
    n, total = C.c_uint32(), C.c_float()
    _check(L, L.tp_last_timeline(ctx, None, None, None, 0, C.byref(n), C.byref(total)))
    cb, ce, xb = (C.c_float * n.value)(), (C.c_float * n.value)(), (C.c_float * n.value)()
    _check(L, L.tp_last_timeline(ctx, cb, ce, xb, n.value, C.byref(n), C.byref(total)))
    return {"total_ms": total.value, "copy_begin_ms": list(cb), "copy_end_ms": list(ce), "exec_begin_ms": list(xb)}


def tp_model_host_image(ctx, model_id) -> np.ndarray:
    """Read-only uint8 view of the library's pinned host image of a model."""
    p, n = _P(), C.c_uint64()
    _check(lib(), lib().tp_model_host_image(ctx, model_id, C.byref(p), C.byref(n)))
    arr = np.ctypeslib.as_array(C.cast(p, C.POINTER(C.c_uint8)), shape=(n.value,))
    arr.flags.writeable = False
    return arr


def tp_workspace_bytes(desc: ModelDesc, batch: int) -> int:
    out = C.c_uint64()
    _check(lib(), lib().tp_workspace_bytes(C.byref(desc.desc), batch, C.byref(out)))
    return out.value


def tp_run_trace(ctx, requests, stream=None):
    """requests: iterable of (model_id, batch, input_dev, output_dev, arrival_ns).

    Returns a list of dicts (issue_ns, done_ns, hit, status, admit_ns). Raises if any request failed
    (after the whole trace ran)."""
    reqs = list(requests)
    arr = (tp_request * len(reqs))()
    for i, (mid, b, x, y, t) in enumerate(reqs):
        arr[i] = tp_request(mid, b, _ptr(x), _ptr(y), int(t))
    res = (tp_request_result * len(reqs))()
    st = lib().tp_run_trace(ctx, arr, len(reqs), _ptr(stream), res)
    out = [{"issue_ns": r.issue_ns, "done_ns": r.done_ns, "hit": bool(r.hit), "status": r.status,
            "admit_ns": r.admit_ns} for r in res]
    _check(lib(), st)
    return out


def tp_run_trace_sched(ctx, requests, deadlines_ns, policy=TP_QUEUE_SLO, max_inflight=2, slo_pct=0.98, alpha=0.5,
                       scalar=2.0, threshold=0.04, period_ns=1_000_000_000, stream=None):
    """Like tp_run_trace with a host-side request queue (FIFO or SLO-aware). Returns
    (results as tp_run_trace gives them, stats dict)."""
    reqs = list(requests)
    arr = (tp_request * len(reqs))()
    for i, (mid, b, x, y, t) in enumerate(reqs):
        arr[i] = tp_request(mid, b, _ptr(x), _ptr(y), int(t))
    dl = (C.c_uint64 * len(reqs))(*[int(v) for v in deadlines_ns])
    cfg = tp_sched_config(policy, max_inflight, slo_pct, alpha, scalar, threshold, period_ns)
    res = (tp_request_result * len(reqs))()
    st = tp_sched_stats()
    status = lib().tp_run_trace_sched(ctx, arr, len(reqs), _ptr(stream), C.byref(cfg), dl, res, C.byref(st))
    out = [{"issue_ns": r.issue_ns, "done_ns": r.done_ns, "hit": bool(r.hit), "status": r.status,
            "admit_ns": r.admit_ns} for r in res]
    _check(lib(), status)
    return out, st.as_dict()


# host-only planning calls; `L` picks the library (the HIP one by default)

def tph_validate(desc: ModelDesc, host_bytes: int, L=None):
    L = L or lib()
    _check(L, L.tph_validate(C.byref(desc.desc), host_bytes))


def tph_touch_span(desc: ModelDesc, host_bytes: int, L=None):
    """(lo, hi) of the extent a warm request of this model pre-reads into the caches, or None."""
    L = L or lib()
    applies, lo, hi = C.c_int32(), C.c_uint64(), C.c_uint64()
    _check(L, L.tph_touch_span(C.byref(desc.desc), host_bytes, C.byref(applies), C.byref(lo), C.byref(hi)))
    return (lo.value, hi.value) if applies.value else None


def tph_plan(desc: ModelDesc, host_bytes: int, chunk_min_bytes: int, flags: int = 0, L=None):
    L = L or lib()
    n = C.c_uint32()
    _check(L, L.tph_plan(C.byref(desc.desc), host_bytes, chunk_min_bytes, flags, None, None, None, 0, C.byref(n)))
    b, e, f = (C.c_uint64 * n.value)(), (C.c_uint64 * n.value)(), (C.c_uint32 * n.value)()
    _check(L, L.tph_plan(C.byref(desc.desc), host_bytes, chunk_min_bytes, flags, b, e, f, n.value, C.byref(n)))
    return [{"begin": b[i], "end": e[i], "first_layer": f[i]} for i in range(n.value)]


def tph_plan_cost_model(desc: ModelDesc, host_bytes: int, plan_batch: int = 1, link_gbs: float = 0.0,
                        chunk_us: float = 0.0, L=None):
    """The TP_PLAN_COST chunk plan of a model: (chunks as tph_plan returns them, modelled us)."""
    L = L or lib()
    n, est = C.c_uint32(), C.c_double()
    _check(L, L.tph_plan_cost_model(C.byref(desc.desc), host_bytes, plan_batch, link_gbs, chunk_us, None, None, None, 0,
                                    C.byref(n), None))
    b, e, f = (C.c_uint64 * n.value)(), (C.c_uint64 * n.value)(), (C.c_uint32 * n.value)()
    _check(L, L.tph_plan_cost_model(C.byref(desc.desc), host_bytes, plan_batch, link_gbs, chunk_us, b, e, f, n.value,
                                    C.byref(n), C.byref(est)))
    return [{"begin": b[i], "end": e[i], "first_layer": f[i]} for i in range(n.value)], est.value


def tph_plan_cost(unit_begin, unit_us, total_bytes: int, link_bytes_per_us: float, chunk_us: float, wait_us: float,
                  L=None):
    """Cost-model grouping over explicit units: (first unit of each chunk, modelled us)."""
    L = L or lib()
    nu = len(unit_begin)
    ub = (C.c_uint64 * nu)(*[int(v) for v in unit_begin])
    us = (C.c_double * nu)(*[float(v) for v in unit_us])
    first = (C.c_uint32 * nu)()
    n, est = C.c_uint32(), C.c_double()
    _check(L, L.tph_plan_cost(ub, us, nu, total_bytes, link_bytes_per_us, chunk_us, wait_us, first, nu, C.byref(n),
                              C.byref(est)))
    return [first[i] for i in range(n.value)], est.value


def tph_layer_costs(desc: ModelDesc, host_bytes: int, batch: int, L=None):
    L = L or lib()
    n = C.c_uint32()
    _check(L, L.tph_layer_costs(C.byref(desc.desc), host_bytes, batch, None, 0, C.byref(n)))
    out = (C.c_double * n.value)()
    _check(L, L.tph_layer_costs(C.byref(desc.desc), host_bytes, batch, out, n.value, C.byref(n)))
    return list(out)


def tph_rrc(n: int, m: int, p: float, L=None) -> float:
    L = L or lib()
    out = C.c_double()
    _check(L, L.tph_rrc(n, m, p, C.byref(out)))
    return out.value


def tph_sched_pick(n, m, p: float, alpha: float, pending_func, L=None):
    """(index into pending_func of the request to run next or -1, high-priority flags)."""
    L = L or lib()
    nf, npend = len(n), len(pending_func)
    na, ma = (C.c_uint64 * max(nf, 1))(*n), (C.c_uint64 * max(nf, 1))(*m)
    pa = (C.c_int32 * max(npend, 1))(*pending_func)
    pick, high = C.c_int32(), (C.c_uint8 * max(nf, 1))()
    _check(L, L.tph_sched_pick(nf, na, ma, p, alpha, npend, pa, C.byref(pick), high))
    return pick.value, [bool(high[i]) for i in range(nf)]


def tph_alpha_update(alpha, last_ratio, new_ratio, scalar=2.0, threshold=0.04, L=None) -> float:
    L = L or lib()
    out = C.c_double()
    _check(L, L.tph_alpha_update(alpha, last_ratio, new_ratio, scalar, threshold, C.byref(out)))
    return out.value


_probe = None


def probe_lib():
    """libtorpor_probe.so (include/torpor_probe.h): the machine's measured peaks."""
    global _probe
    if _probe is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise ImportError(f"{PROBE_LIB_PATH} is not built; run python -m paper_2306_03622_amd.build")
        L = C.CDLL(PROBE_LIB_PATH)
        L.tpp_mfma_bf16.argtypes = [C.c_int, C.c_int, C.c_int, C.POINTER(C.c_double), C.POINTER(C.c_double)]
        L.tpp_hbm_read.argtypes = [C.c_uint64, C.c_int, C.c_int, C.POINTER(C.c_double)]
        L.tpp_gather_h2d.argtypes = [C.c_uint64, C.c_int, C.c_int, C.POINTER(C.c_double)]
        for f in (L.tpp_mfma_bf16, L.tpp_hbm_read, L.tpp_gather_h2d):
            f.restype = C.c_int
        _probe = L
    return _probe


def _probe_check(rc, what):
    if rc != 0:
        raise RuntimeError(f"{what}: HIP error {rc}")


def probe_mfma_bf16(wgs=1024, iters=2048, reps=5):
    """(TFLOP/s, shader clock GHz) of back-to-back bf16 16x16x32 MFMAs on every CU."""
    t, c = C.c_double(), C.c_double()
    _probe_check(probe_lib().tpp_mfma_bf16(wgs, iters, reps, C.byref(t), C.byref(c)), "tpp_mfma_bf16")
    return t.value, c.value


def probe_hbm_read(nbytes=4 << 30, wgs=2048, reps=5):
    """GB/s of a streaming read of nbytes of device memory."""
    g = C.c_double()
    _probe_check(probe_lib().tpp_hbm_read(nbytes, wgs, reps, C.byref(g)), "tpp_hbm_read")
    return g.value


def probe_gather_h2d(nbytes=1 << 30, wgs=1024, reps=5):
    """GB/s of a kernel copying pinned host memory to the device."""
    g = C.c_double()
    _probe_check(probe_lib().tpp_gather_h2d(nbytes, wgs, reps, C.byref(g)), "tpp_gather_h2d")
    return g.value


class HostArena:
    """tph_arena_*: the arena bookkeeping without a device."""

    def __init__(self, capacity: int, align: int = 256, L=None, policy: int = TP_EVICT_LRU, partition: int = 0,
                 consolidate: bool = False):
        self.L = L or lib()
        self.h = _P()
        _check(self.L, self.L.tph_arena_create(capacity, align, C.byref(self.h)))
        if policy != TP_EVICT_LRU:
            _check(self.L, self.L.tph_arena_set_policy(self.h, policy))
        self.consolidate = consolidate
        if partition:
            self.set_partitioned(partition, consolidate)

    def set_partitioned(self, partition: int, consolidate: bool = False):
        _check(self.L, self.L.tph_arena_set_partitioned(self.h, partition, int(consolidate)))
        self.consolidate = consolidate and partition > 0

    def steps(self):
        """The last request's victims and consolidation moves in the order made:
        [("evict", model)] and [("move", model, old offset, new offset)] entries."""
        n = C.c_uint32()
        _check(self.L, self.L.tph_arena_steps(self.h, None, None, None, None, 0, C.byref(n)))
        ids, mv = (C.c_int32 * n.value)(), (C.c_int32 * n.value)()
        fr, to = (C.c_uint64 * n.value)(), (C.c_uint64 * n.value)()
        _check(self.L, self.L.tph_arena_steps(self.h, ids, mv, fr, to, n.value, C.byref(n)))
        return [("move", ids[i], fr[i], to[i]) if mv[i] else ("evict", ids[i]) for i in range(n.value)]

    def __del__(self):
        if getattr(self, "h", None):
            self.L.tph_arena_destroy(self.h)
            self.h = None

    def register(self, mid, nbytes, heavy: bool = False):
        _check(self.L, self.L.tph_arena_register(self.h, mid, nbytes))
        if heavy:
            _check(self.L, self.L.tph_arena_set_heavy(self.h, mid, 1))

    def set_heavy(self, mid, heavy: bool):
        _check(self.L, self.L.tph_arena_set_heavy(self.h, mid, int(heavy)))

    def unregister(self, mid):
        _check(self.L, self.L.tph_arena_unregister(self.h, mid))

    def request(self, mid):
        hit, off, n = C.c_int32(), C.c_uint64(), C.c_uint32()
        vict = (C.c_int32 * 1024)()
        _check(self.L, self.L.tph_arena_request(self.h, mid, C.byref(hit), C.byref(off), vict, 1024, C.byref(n)))
        out = {"hit": bool(hit.value), "offset": off.value, "evicted": [vict[i] for i in range(n.value)]}
        if self.consolidate:
            out["steps"] = self.steps()
        return out

    def evict(self, mid):
        _check(self.L, self.L.tph_arena_evict(self.h, mid))

    def stats(self):
        s = tp_arena_stats_t()
        _check(self.L, self.L.tph_arena_stats(self.h, C.byref(s)))
        return s.as_dict()


# ------------------------------------------------------------------ convenience

class Runtime:
    """A context whose arena and workspace are torch allocations made once."""

    def __init__(self, arena_bytes: int, work_bytes: int, device: int = 0, chunk_min_bytes: int = DEFAULT_CHUNK,
                 copy_method: int = TP_COPY_MEMCPY, gather_wgs: int = 0, flags: int = 0, throttle_us: int = 0,
                 copy_stream=None, copy_streams: int = 0, direct_max_bytes: int = DEFAULT_DIRECT,
                 plan: int = TP_PLAN_GREEDY, plan_batch: int = 0, link_gbs: float = 0.0, chunk_us: float = 0.0,
                 evict_policy: int = TP_EVICT_LRU, heavy_ratio: float = 0.0, alloc: int = TP_ALLOC_FIRST_FIT,
                 partition_bytes: int = 0):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("libtorpor needs a HIP device")
        self.torch = torch
        self.device = torch.device("cuda", device)
        torch.cuda.set_device(self.device)
        self.arena = torch.empty(arena_bytes, dtype=torch.uint8, device=self.device)
        self.work = torch.empty(max(work_bytes, 256), dtype=torch.uint8, device=self.device)
        self.copy_stream = copy_stream
        self.ctx = tp_create(self.arena, arena_bytes, self.work, self.work.numel(), copy_stream, chunk_min_bytes,
                             copy_method, gather_wgs, flags, throttle_us, copy_streams, direct_max_bytes, plan,
                             plan_batch, link_gbs, chunk_us, evict_policy, heavy_ratio, alloc, partition_bytes)
        self.descs = {}

    def close(self):
        if self.ctx is not None:
            tp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def register(self, desc: ModelDesc, host_weights: np.ndarray) -> int:
        mid = tp_register_model(self.ctx, desc, host_weights)
        self.descs[mid] = desc
        return mid

    def unregister(self, mid):
        tp_unregister_model(self.ctx, mid)
        self.descs.pop(mid, None)

    def infer(self, mid, x, out, stream=None):
        """x, out: torch device tensors; stream: a torch stream (default: current)."""
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        tp_infer(self.ctx, mid, x, int(x.shape[0]), out, s)

    def infer_noalloc(self, mid, x, out, stream=None):
        """tp_infer on the library's static workspace (allocates nothing)."""
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        tp_infer_noalloc(self.ctx, mid, x, int(x.shape[0]), out, s)

    def swap_in(self, mid, stream=None):
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        tp_swap_in(self.ctx, mid, s)

    def evict(self, mid):
        tp_evict(self.ctx, mid)

    def fail_copy(self, nth: int):
        """Test hook: the nth copy enqueued from now on fails (0 disarms)."""
        tp_debug_fail_copy(self.ctx, nth)

    def resident(self, mid) -> bool:
        return tp_is_resident(self.ctx, mid)

    def stats(self) -> dict:
        return tp_arena_stats(self.ctx)

    def info(self, mid) -> dict:
        return tp_model_info(self.ctx, mid)

    def set_class(self, mid, model_class: int):
        tp_set_model_class(self.ctx, mid, model_class)

    def timeline(self):
        return tp_last_timeline(self.ctx)

    def chunks(self, mid):
        return tp_model_chunks(self.ctx, mid)

    def host_image(self, mid) -> np.ndarray:
        return tp_model_host_image(self.ctx, mid)

    def run_trace(self, requests, stream=None):
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        return tp_run_trace(self.ctx, requests, s)

    def run_trace_sched(self, requests, deadlines_ns, stream=None, **kw):
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        return tp_run_trace_sched(self.ctx, requests, deadlines_ns, stream=s, **kw)

    def extent(self, mid):
        """The model's arena bytes (a view of the arena), when resident."""
        i = self.info(mid)
        return self.arena[i["extent_offset"]:i["extent_offset"] + i["host_bytes"]]
