"""ctypes binding of libcrosspool.so (include/crosspool.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels. PyTorch is used for device buffers and streams. The functions
keep the C names; ``Pool`` is a small convenience wrapper over them.

Importing this module loads the library and fails loudly if it has not been
built (``python -m paper_2606_24506_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcrosspool.so")

CP_OK, CP_EINVAL, CP_ENOMEM, CP_ENOSPC, CP_EHIP, CP_ESTATE = 0, -1, -2, -3, -4, -5
CP_KIND_MLA, CP_KIND_GQA = 0, 1
CP_PATH_AUTO, CP_PATH_VALU, CP_PATH_MFMA = 0, 1, 2
CP_SCHED_BALANCED, CP_SCHED_QUEUE, CP_SCHED_GRID = 0, 1, 2
CP_BACKING_BUFFER, CP_BACKING_VIRTUAL = 0, 1
_NAMES = {0: "CP_OK", -1: "CP_EINVAL", -2: "CP_ENOMEM", -3: "CP_ENOSPC", -4: "CP_EHIP", -5: "CP_ESTATE"}


class CrossPoolError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class cp_pool_desc(C.Structure):
    _fields_ = [
        ("page_tokens", C.c_int32),
        ("device", C.c_int32),
        ("pool_bytes", C.c_uint64),
        ("chunk_bytes", C.c_uint64),
        ("placement_seed", C.c_uint64),
        ("device_mem", C.c_void_p),
        ("max_requests", C.c_int32),
        ("backing", C.c_int32),
        ("max_workspace_bytes", C.c_uint64),
        ("device_pages", C.c_int32),
    ]


class cp_pool_stats_t(C.Structure):
    _fields_ = [
        ("chunks_total", C.c_uint64),
        ("chunks_used", C.c_uint64),
        ("pages_used", C.c_uint64),
        ("pages_reserved", C.c_uint64),
        ("requests_open", C.c_int32),
        ("models", C.c_int32),
        ("span_bytes", C.c_uint64),
        ("backing", C.c_int32),
        ("max_models", C.c_int32),
    ]


class cp_model_desc(C.Structure):
    _fields_ = [
        ("kind", C.c_int32),
        ("n_q_heads", C.c_int32),
        ("n_kv_heads", C.c_int32),
        ("head_dim", C.c_int32),
        ("latent_dim", C.c_int32),
        ("rope_dim", C.c_int32),
        ("softmax_scale", C.c_float),
        ("dtype", C.c_int32),
        ("n_layers", C.c_int32),
    ]


class cp_model_info_t(C.Structure):
    _fields_ = [
        ("d_k", C.c_int32),
        ("d_v", C.c_int32),
        ("kappa", C.c_int32),
        ("page_bytes", C.c_int32),
        ("pages_per_chunk", C.c_int32),
        ("row_elems", C.c_int32),
        ("n_layers", C.c_int32),
    ]


class cp_decode_opts(C.Structure):
    _fields_ = [
        ("num_splits", C.c_int32),
        ("schedule", C.c_int32),
        ("path", C.c_int32),
        ("reserved0", C.c_int32),
        ("ev_begin", C.c_void_p),
        ("ev_end", C.c_void_p),
    ]


class cp_plan_model(C.Structure):
    _fields_ = [("kappa_bytes", C.c_double), ("arrival_rate", C.c_double), ("n_samples", C.c_int64),
                ("prompt_tokens", C.POINTER(C.c_int64)), ("output_tokens", C.POINTER(C.c_int64)),
                ("service_time_s", C.POINTER(C.c_double))]


class cp_plan_opts(C.Structure):
    _fields_ = [("horizon_s", C.c_double), ("n_obs", C.c_int64), ("quantile", C.c_double), ("seed", C.c_uint64),
                ("chunk_bytes", C.c_uint64)]


class cp_plan_result(C.Structure):
    _fields_ = [("quantile_bytes", C.c_double), ("mean_bytes", C.c_double), ("max_bytes", C.c_double),
                ("pool_bytes", C.c_uint64), ("n_arrivals", C.c_int64)]


def _load() -> C.CDLL:
    # PyTorch ships its own HIP runtime (soname libamdhip64.so.7, like the
    # system one). Loading torch first makes the library bind to that same
    # runtime instance, so torch's streams and allocations are valid here.
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover - plain C users do not need torch
        pass
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2606_24506_amd.build`")
    lib = C.CDLL(_LIB_PATH)
    P, I32, I64, VP = C.c_void_p, C.c_int32, C.c_int64, C.c_void_p
    sig = {
        "cp_last_error": ([], C.c_char_p),
        "cp_version": ([], I32),
        "cp_pool_create": ([C.POINTER(cp_pool_desc), C.POINTER(P)], I32),
        "cp_pool_destroy": ([P], I32),
        "cp_pool_stats": ([P, C.POINTER(cp_pool_stats_t)], I32),
        "cp_model_register": ([P, C.POINTER(cp_model_desc), C.POINTER(I32)], I32),
        "cp_model_info": ([P, I32, C.POINTER(cp_model_info_t)], I32),
        "cp_request_open": ([P, I32, I64, C.POINTER(I32)], I32),
        "cp_request_close": ([P, I32], I32),
        "cp_request_len": ([P, I32, C.POINTER(I64)], I32),
        "cp_request_cursor": ([P, I32, C.POINTER(I32), C.POINTER(I32)], I32),
        "cp_request_pages": ([P, I32, I64, I64, C.POINTER(C.c_uint32)], I32),
        "cp_kv_append": ([P, I32, VP, VP, VP, VP], I32),
        "cp_attn_decode": ([P, I32, VP, VP, VP, VP, VP], I32),
        "cp_attn_decode_ex": ([P, I32, VP, VP, VP, VP, VP, C.POINTER(cp_decode_opts)], I32),
        "cp_attn_decode_noalloc": ([P, I32, VP, VP, VP, VP, VP, C.POINTER(cp_decode_opts)], I32),
        "cp_attn_decode_step": ([P, I32, VP, VP, VP, VP, VP, VP, VP, C.POINTER(cp_decode_opts)],
                                I32),
        "cp_attn_decode_layers": ([P, I32, VP, VP, VP, VP, VP, VP, VP,
                                   C.POINTER(cp_decode_opts)], I32),
        "cp_request_layer_state": ([P, I32, C.POINTER(I32), C.POINTER(I64)], I32),
        "cp_kv_gather": ([P, I32, I64, I64, VP, VP], I32),
        "cp_plan_pool": ([C.POINTER(cp_plan_model), I32, C.POINTER(cp_plan_opts), C.POINTER(cp_plan_result)], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()


def _check(rc: int):
    if rc != CP_OK:
        raise CrossPoolError(rc, LIB.cp_last_error().decode(errors="replace"))


def i32_array(xs: Sequence[int]):
    """A host int32 array argument built once, for callers that repeat a
    call with the same request ids (it is passed as it is)."""
    return (C.c_int32 * len(xs))(*[int(x) for x in xs])


def _i32_array(xs: Sequence[int]):
    """A host int32 array argument: an array from i32_array passes as it is,
    a contiguous numpy int32 array passes its address (no copy), anything
    else is copied into a ctypes array."""
    if isinstance(xs, C.Array):
        return xs
    if isinstance(xs, np.ndarray) and xs.dtype == np.int32 and xs.flags.c_contiguous:
        return xs.__array_interface__["data"][0]
    return (C.c_int32 * len(xs))(*[int(x) for x in xs])


def _ptr(t) -> Optional[int]:
    """Device pointer of a tensor (or None / raw int)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


_OPTS = {}


def _event(e):
    if e is None:
        return None
    return e.cuda_event if hasattr(e, "cuda_event") else int(e)


def _opts(num_splits: int, schedule: int, path: int, ev_begin, ev_end):
    """Pointer to a cp_decode_opts; the event-free ones are built once per
    (num_splits, schedule, path) and reused."""
    if ev_begin is None and ev_end is None:
        key = (num_splits, schedule, path)
        o = _OPTS.get(key)
        if o is None:
            o = _OPTS[key] = C.pointer(cp_decode_opts(num_splits, schedule, path, 0, None, None))
        return o
    return C.pointer(cp_decode_opts(num_splits, schedule, path, 0, _event(ev_begin), _event(ev_end)))


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch

        if not torch.cuda.is_available():
            return None
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------ C names ----

def cp_version() -> int:
    return int(LIB.cp_version())


def cp_pool_create(page_tokens: int = 64, pool_bytes: int = 0, chunk_bytes: int = 0, placement_seed: int = 0,
                   device: int = 0, device_mem=None, max_requests: int = 0, backing: int = 0,
                   max_workspace_bytes: int = 0, device_pages: int = 0) -> int:
    d = cp_pool_desc(page_tokens, device, pool_bytes, chunk_bytes, placement_seed, _ptr(device_mem), max_requests,
                     backing, max_workspace_bytes, device_pages)
    out = C.c_void_p()
    _check(LIB.cp_pool_create(C.byref(d), C.byref(out)))
    return out.value


def cp_pool_destroy(pool: int) -> None:
    _check(LIB.cp_pool_destroy(pool))


def cp_pool_stats(pool: int) -> dict:
    s = cp_pool_stats_t()
    _check(LIB.cp_pool_stats(pool, C.byref(s)))
    return {f: getattr(s, f) for f, _ in s._fields_}


def cp_model_register(pool: int, kind: int, n_q_heads: int, n_kv_heads: int, head_dim: int = 0,
                      latent_dim: int = 0, rope_dim: int = 0, softmax_scale: float = 0.0, n_layers: int = 1) -> int:
    m = cp_model_desc(kind, n_q_heads, n_kv_heads, head_dim, latent_dim, rope_dim, softmax_scale, 0, n_layers)
    mid = C.c_int32()
    _check(LIB.cp_model_register(pool, C.byref(m), C.byref(mid)))
    return mid.value


def cp_model_info(pool: int, model_id: int) -> dict:
    s = cp_model_info_t()
    _check(LIB.cp_model_info(pool, model_id, C.byref(s)))
    return {f: getattr(s, f) for f, _ in s._fields_}


def cp_request_open(pool: int, model_id: int, reserve_tokens: int) -> int:
    rid = C.c_int32()
    _check(LIB.cp_request_open(pool, model_id, reserve_tokens, C.byref(rid)))
    return rid.value


def cp_request_close(pool: int, req_id: int) -> None:
    _check(LIB.cp_request_close(pool, req_id))


def cp_request_len(pool: int, req_id: int) -> int:
    n = C.c_int64()
    _check(LIB.cp_request_len(pool, req_id, C.byref(n)))
    return n.value


def cp_request_cursor(pool: int, req_id: int):
    """(layer, in_flight) of the request's layer cursor."""
    layer, inflight = C.c_int32(), C.c_int32()
    _check(LIB.cp_request_cursor(pool, req_id, C.byref(layer), C.byref(inflight)))
    return layer.value, inflight.value


def cp_request_pages(pool: int, req_id: int, first: int, count: int, layers: int = 1) -> np.ndarray:
    """Page-table entries, [count] for one layer or [layers][count]."""
    out = np.zeros((layers, count), dtype=np.uint32)
    _check(LIB.cp_request_pages(pool, req_id, first, count, out.ctypes.data_as(C.POINTER(C.c_uint32))))
    return out[0] if layers == 1 else out


def cp_kv_append(pool: int, req_ids: Sequence[int], n_new: Sequence[int], rows, stream=None) -> None:
    n = len(req_ids)
    if len(n_new) != n:
        raise ValueError("req_ids and n_new differ in length")
    _check(LIB.cp_kv_append(pool, n, _i32_array(req_ids), _i32_array(n_new), _ptr(rows), _stream(stream)))


def cp_attn_decode(pool: int, req_ids: Sequence[int], q, out, lse, stream=None) -> None:
    _check(LIB.cp_attn_decode(pool, len(req_ids), _i32_array(req_ids), _ptr(q), _ptr(out), _ptr(lse), _stream(stream)))


def cp_attn_decode_ex(pool: int, req_ids: Sequence[int], q, out, lse, stream=None, *, num_splits: int = 0,
                      schedule: int = CP_SCHED_BALANCED, path: int = CP_PATH_AUTO, ev_begin=None,
                      ev_end=None) -> None:
    o = _opts(num_splits, schedule, path, ev_begin, ev_end)
    _check(LIB.cp_attn_decode_ex(pool, len(req_ids), _i32_array(req_ids), _ptr(q), _ptr(out), _ptr(lse),
                                 _stream(stream), o))


def cp_attn_decode_noalloc(pool: int, req_ids: Sequence[int], q, out, lse, stream=None, *, num_splits: int = 0,
                           schedule: int = CP_SCHED_BALANCED, path: int = CP_PATH_AUTO, ev_begin=None,
                           ev_end=None) -> None:
    o = _opts(num_splits, schedule, path, ev_begin, ev_end)
    _check(LIB.cp_attn_decode_noalloc(pool, len(req_ids), _i32_array(req_ids), _ptr(q), _ptr(out), _ptr(lse),
                                      _stream(stream), o))


def cp_attn_decode_step(pool: int, req_ids: Sequence[int], n_new: Sequence[int], rows, q, out, lse, stream=None, *,
                        num_splits: int = 0, schedule: int = CP_SCHED_BALANCED, path: int = CP_PATH_AUTO,
                        ev_begin=None, ev_end=None) -> None:
    n = len(req_ids)
    if len(n_new) != n:
        raise ValueError("req_ids and n_new differ in length")
    o = _opts(num_splits, schedule, path, ev_begin, ev_end)
    _check(LIB.cp_attn_decode_step(pool, n, _i32_array(req_ids), _i32_array(n_new), _ptr(rows), _ptr(q), _ptr(out),
                                   _ptr(lse), _stream(stream), o))


def cp_attn_decode_layers(pool: int, req_ids: Sequence[int], n_new: Sequence[int], rows, q, out, lse, stream=None, *,
                          num_splits: int = 0, schedule: int = CP_SCHED_BALANCED, path: int = CP_PATH_AUTO,
                          ev_begin=None, ev_end=None) -> None:
    o = _opts(num_splits, schedule, path, ev_begin, ev_end)
    n = len(req_ids)
    _check(LIB.cp_attn_decode_layers(pool, n, _i32_array(req_ids), _i32_array(n_new), _ptr(rows), _ptr(q), _ptr(out),
                                     _ptr(lse), _stream(stream), o))


def cp_request_layer_state(pool: int, req_id: int):
    layer, tokens = C.c_int32(), C.c_int64()
    _check(LIB.cp_request_layer_state(pool, req_id, C.byref(layer), C.byref(tokens)))
    return layer.value, tokens.value


def cp_kv_gather(pool: int, req_id: int, start: int, n_tok: int, dst, stream=None) -> None:
    _check(LIB.cp_kv_gather(pool, req_id, start, n_tok, _ptr(dst), _stream(stream)))


def cp_plan_pool(models, horizon_s: float, n_obs: int, quantile: float, seed: int, chunk_bytes: int = 2 << 20) -> dict:
    """models: sequence of dicts with kappa_bytes, arrival_rate and equal-length
    prompt_tokens / output_tokens / service_time_s sequences (trace records)."""
    keep = []
    arr = (cp_plan_model * len(models))()
    for i, m in enumerate(models):
        op = (C.c_int64 * len(m["prompt_tokens"]))(*[int(x) for x in m["prompt_tokens"]])
        od = (C.c_int64 * len(m["output_tokens"]))(*[int(x) for x in m["output_tokens"]])
        tr = (C.c_double * len(m["service_time_s"]))(*[float(x) for x in m["service_time_s"]])
        if not (len(op) == len(od) == len(tr)):
            raise ValueError("trace columns differ in length")
        keep += [op, od, tr]
        arr[i] = cp_plan_model(float(m["kappa_bytes"]), float(m["arrival_rate"]), len(op), op, od, tr)
    o = cp_plan_opts(float(horizon_s), int(n_obs), float(quantile), int(seed) & ((1 << 64) - 1), int(chunk_bytes))
    r = cp_plan_result()
    _check(LIB.cp_plan_pool(arr, len(models), C.byref(o), C.byref(r)))
    return dict(quantile_bytes=r.quantile_bytes, mean_bytes=r.mean_bytes, max_bytes=r.max_bytes,
                pool_bytes=r.pool_bytes, n_arrivals=r.n_arrivals)


# -------------------------------------------------------- convenience ----

class Pool:
    """Owns one cp_pool handle; methods forward to the C names above."""

    def __init__(self, **desc):
        self.handle = cp_pool_create(**desc)
        self.device = desc.get("device", 0)
        self.page_tokens = desc.get("page_tokens", 64)

    def register(self, kind: int, n_q_heads: int, n_kv_heads: int, **kw) -> int:
        return cp_model_register(self.handle, kind, n_q_heads, n_kv_heads, **kw)

    def register_spec(self, spec, n_layers: int = 1) -> int:
        """Register a model described by an object with kind / head fields."""
        if spec.kind == "mla":
            return self.register(CP_KIND_MLA, spec.n_q_heads, 1, latent_dim=spec.latent_dim,
                                 rope_dim=spec.rope_dim, softmax_scale=spec.scale, n_layers=n_layers)
        return self.register(CP_KIND_GQA, spec.n_q_heads, spec.n_kv_heads, head_dim=spec.head_dim,
                             softmax_scale=spec.scale, n_layers=n_layers)

    def info(self, model_id: int) -> dict:
        return cp_model_info(self.handle, model_id)

    def open(self, model_id: int, reserve_tokens: int) -> int:
        return cp_request_open(self.handle, model_id, reserve_tokens)

    def close(self, req_id: int) -> None:
        cp_request_close(self.handle, req_id)

    def ctx_len(self, req_id: int) -> int:
        return cp_request_len(self.handle, req_id)

    def cursor(self, req_id: int):
        return cp_request_cursor(self.handle, req_id)

    def pages(self, req_id: int, first: int = 0, count: Optional[int] = None, layers: int = 1) -> np.ndarray:
        if count is None:
            count = -(-self.ctx_len(req_id) // self.page_tokens) - first
        return cp_request_pages(self.handle, req_id, first, count, layers)

    def stats(self) -> dict:
        return cp_pool_stats(self.handle)

    def append(self, req_ids, n_new, rows, stream=None) -> None:
        cp_kv_append(self.handle, req_ids, n_new, rows, stream)

    def decode(self, req_ids, q, out, lse, stream=None, **opts) -> None:
        if opts:
            cp_attn_decode_ex(self.handle, req_ids, q, out, lse, stream, **opts)
        else:
            cp_attn_decode(self.handle, req_ids, q, out, lse, stream)

    def decode_noalloc(self, req_ids, q, out, lse, stream=None, **opts) -> None:
        cp_attn_decode_noalloc(self.handle, req_ids, q, out, lse, stream, **opts)

    def decode_step(self, req_ids, n_new, rows, q, out, lse, stream=None, **opts) -> None:
        cp_attn_decode_step(self.handle, req_ids, n_new, rows, q, out, lse, stream, **opts)

    def decode_layers(self, req_ids, n_new, rows, q, out, lse, stream=None, **opts) -> None:
        cp_attn_decode_layers(self.handle, req_ids, n_new, rows, q, out, lse, stream, **opts)

    def layer_state(self, req_id: int):
        return cp_request_layer_state(self.handle, req_id)

    def gather(self, req_id, start, n_tok, dst, stream=None) -> None:
        cp_kv_gather(self.handle, req_id, start, n_tok, dst, stream)

    def destroy(self) -> None:
        if self.handle:
            cp_pool_destroy(self.handle)
            self.handle = None
