"""ctypes binding of libpkv (see ``include/pkv.h``).

Argument marshalling only: every step of the restore runs in the library.
The functions keep the C names.  ``load()`` raises if ``libpkv.so`` has not
been built (``python -m paper_2609_26219_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Iterable, List, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpkv.so")

PKV_OK = 0
PKV_ERR_INVALID_ARGUMENT = -1
PKV_ERR_BAD_TAG = -2
PKV_ERR_PAGE_OUT_OF_RANGE = -3
PKV_ERR_PAGE_UNMAPPED = -4
PKV_ERR_PAGE_ALIAS = -5
PKV_ERR_OUT_OF_MEMORY = -6
PKV_ERR_DEVICE = -7

# Every symbol include/pkv.h declares.
EXPORTED = ("pkv_payload_size", "pkv_restore_plan", "pkv_restore", "pkv_restore_from_host", "pkv_free",
            "pkv_plan_query", "pkv_status_string", "pkv_checkpoint_plan", "pkv_quantize_gather", "pkv_plan_repair",
            "pkv_plan_payload_bytes", "pkv_restore_from_host_noalloc")


class PkvModel(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_tokens", ctypes.c_int32), ("page_size", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("pool_pages", ctypes.c_int64), ("rope_theta", ctypes.c_double), ("rope_style", ctypes.c_int32),
                ("rotary_dim", ctypes.c_int32), ("inv_freq", ctypes.c_void_p), ("kv_layout", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class PkvRequest(ctypes.Structure):
    _fields_ = [("suffix_tokens", ctypes.c_int32), ("delta", ctypes.c_int32), ("dst_row0", ctypes.c_int64),
                ("tags", ctypes.c_void_p), ("repair_mask", ctypes.c_void_p), ("page_table", ctypes.c_void_p),
                ("num_logical_pages", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("payload_offset", ctypes.c_uint64), ("scale_offset", ctypes.c_uint64)]


class PkvCheckpointRequest(ctypes.Structure):
    _fields_ = [("suffix_tokens", ctypes.c_int32), ("reserved", ctypes.c_int32), ("src_row0", ctypes.c_int64),
                ("tags", ctypes.c_void_p), ("page_table", ctypes.c_void_p), ("num_logical_pages", ctypes.c_int32),
                ("reserved2", ctypes.c_int32), ("payload_offset", ctypes.c_uint64), ("scale_offset", ctypes.c_uint64)]


class PkvPlanInfo(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int64), ("num_units", ctypes.c_int64), ("restored_rows", ctypes.c_int64),
                ("payload_bytes", ctypes.c_uint64), ("scale_bytes", ctypes.c_uint64),
                ("cache_bytes", ctypes.c_uint64), ("bytes_read", ctypes.c_uint64),
                ("bytes_written", ctypes.c_uint64), ("device", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("host_copy_bytes", ctypes.c_uint64), ("host_copies", ctypes.c_int64)]


class PkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {pkv_status_string(status)} ({status})")


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libpkv.so (once).  Raises ImportError when it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libpkv.so not built at {path}; run python -m paper_2609_26219_amd.build")
    lib = ctypes.CDLL(path)
    vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32
    lib.pkv_payload_size.argtypes = [ctypes.POINTER(PkvModel), ctypes.POINTER(PkvRequest),
                                     ctypes.POINTER(u64), ctypes.POINTER(u64)]
    lib.pkv_payload_size.restype = i32
    lib.pkv_restore_plan.argtypes = [ctypes.POINTER(PkvModel), ctypes.POINTER(PkvRequest), i32, ctypes.POINTER(vp)]
    lib.pkv_restore_plan.restype = i32
    lib.pkv_restore.argtypes = [vp, vp, u64, vp, u64, vp, vp, u64, vp]
    lib.pkv_restore.restype = i32
    lib.pkv_restore_from_host.argtypes = [vp, vp, u64, vp, u64, vp, u64, vp, u64, vp, vp, u64, vp]
    lib.pkv_restore_from_host.restype = i32
    lib.pkv_free.argtypes = [vp]
    lib.pkv_free.restype = None
    lib.pkv_plan_query.argtypes = [vp, ctypes.POINTER(PkvPlanInfo)]
    lib.pkv_plan_query.restype = i32
    lib.pkv_status_string.argtypes = [i32]
    lib.pkv_status_string.restype = ctypes.c_char_p
    lib.pkv_checkpoint_plan.argtypes = [ctypes.POINTER(PkvModel), ctypes.POINTER(PkvCheckpointRequest), i32,
                                        ctypes.POINTER(vp)]
    lib.pkv_checkpoint_plan.restype = i32
    lib.pkv_quantize_gather.argtypes = [vp, vp, vp, u64, vp, u64, vp, u64, vp]
    lib.pkv_quantize_gather.restype = i32
    lib.pkv_plan_repair.argtypes = [i32, i32, ctypes.c_int64, vp, ctypes.c_double, vp, ctypes.POINTER(ctypes.c_int64)]
    lib.pkv_plan_repair.restype = i32
    lib.pkv_restore_from_host_noalloc.argtypes = [vp, vp, u64, vp, u64, vp, vp, u64, vp]
    lib.pkv_restore_from_host_noalloc.restype = i32
    lib.pkv_plan_payload_bytes.argtypes = [vp, i32, ctypes.POINTER(u64)]
    lib.pkv_plan_payload_bytes.restype = i32
    _lib = lib
    return lib


def pkv_status_string(status: int) -> str:
    return load().pkv_status_string(int(status)).decode()


def make_model(shape) -> PkvModel:
    """PkvModel from any object with the pkv_model_t field names (the RoPE
    fields are optional).  The returned structure keeps the frequency array
    it points to alive."""
    inv = getattr(shape, "inv_freq", None)
    freq = None if inv is None else np.ascontiguousarray(inv, dtype=np.float64)
    m = PkvModel(int(shape.num_layers), int(shape.num_kv_heads), int(shape.head_dim), int(shape.block_tokens),
                 int(shape.page_size), int(shape.out_dtype), int(shape.pool_pages), float(shape.rope_theta),
                 int(getattr(shape, "rope_style", 0)), int(getattr(shape, "rotary_dim", 0)),
                 freq.ctypes.data if freq is not None and freq.size else None, int(getattr(shape, "kv_layout", 0)), 0)
    m.keep = freq
    return m


class _Requests:
    """A ctypes array of PkvRequest plus the host arrays it points into."""

    def __init__(self, requests: Sequence):
        self.keep: List[np.ndarray] = []
        self.array = (PkvRequest * max(1, len(requests)))()
        self.count = len(requests)
        for i, r in enumerate(requests):
            tags = np.ascontiguousarray(r.tags, dtype=np.uint8)
            rep = np.ascontiguousarray(r.repair, dtype=np.uint8)
            pt = np.ascontiguousarray(r.page_table, dtype=np.int32)
            self.keep += [tags, rep, pt]
            self.array[i] = PkvRequest(int(r.suffix_tokens), int(r.delta), int(r.dst_row0),
                                       tags.ctypes.data if tags.size else None,
                                       rep.ctypes.data if rep.size else None,
                                       pt.ctypes.data if pt.size else None, int(pt.size),
                                       int(getattr(r, "reserved", 0)), int(r.payload_offset), int(r.scale_offset))


class _CheckpointRequests:
    """A ctypes array of PkvCheckpointRequest plus the host arrays it points into.
    Request objects need suffix_tokens, src_row0, tags, src_page_table (or
    page_table), payload_offset and scale_offset."""

    def __init__(self, requests: Sequence):
        self.keep: List[np.ndarray] = []
        self.array = (PkvCheckpointRequest * max(1, len(requests)))()
        self.count = len(requests)
        for i, r in enumerate(requests):
            tags = np.ascontiguousarray(r.tags, dtype=np.uint8)
            pt = np.ascontiguousarray(getattr(r, "src_page_table", None) if getattr(r, "src_page_table", None)
                                      is not None else r.page_table, dtype=np.int32)
            self.keep += [tags, pt]
            self.array[i] = PkvCheckpointRequest(int(r.suffix_tokens), int(getattr(r, "reserved", 0)),
                                                 int(r.src_row0), tags.ctypes.data if tags.size else None,
                                                 pt.ctypes.data if pt.size else None, int(pt.size),
                                                 int(getattr(r, "reserved2", 0)), int(r.payload_offset),
                                                 int(r.scale_offset))


def pkv_checkpoint_plan_status(shape, requests: Sequence) -> int:
    lib = load()
    m = make_model(shape)
    reqs = _CheckpointRequests(requests)
    out = ctypes.c_void_p()
    st = lib.pkv_checkpoint_plan(ctypes.byref(m), reqs.array, reqs.count, ctypes.byref(out))
    if out.value:
        lib.pkv_free(out.value)
    return st


def pkv_checkpoint_plan(shape, requests: Sequence) -> "Plan":
    lib = load()
    m = make_model(shape)
    reqs = _CheckpointRequests(requests)
    out = ctypes.c_void_p()
    st = lib.pkv_checkpoint_plan(ctypes.byref(m), reqs.array, reqs.count, ctypes.byref(out))
    if st != PKV_OK:
        raise PkvError(st, "pkv_checkpoint_plan")
    return Plan(out.value)


def pkv_quantize_gather(plan: "Plan", k_cache: int, v_cache: int, cache_bytes: int, payload: int,
                        payload_bytes: int, scales: int, scale_bytes: int, stream: int = 0) -> None:
    st = load().pkv_quantize_gather(plan.handle, k_cache, v_cache, cache_bytes, payload, payload_bytes, scales,
                                    scale_bytes, stream or None)
    if st != PKV_OK:
        raise PkvError(st, "pkv_quantize_gather")


def cache_nbytes(k_cache, v_cache) -> int:
    """The cache_bytes argument for torch caches: a tensor's bytes, or, when
    k_cache and v_cache are the K and V views of one paired cache, the bytes
    of their shared storage from k_cache on."""
    ks, vs = k_cache.untyped_storage(), v_cache.untyped_storage()
    if ks.data_ptr() == vs.data_ptr():
        return ks.nbytes() - (k_cache.data_ptr() - ks.data_ptr())
    return k_cache.numel() * k_cache.element_size()


def quantize_gather_tensors(plan: "Plan", k_cache, v_cache, payload, scales, stream=None) -> None:
    """Marshal torch device tensors (contiguous) and the current stream into pkv_quantize_gather."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(k_cache.device)
    nbytes = lambda t: t.numel() * t.element_size()
    pkv_quantize_gather(plan, k_cache.data_ptr(), v_cache.data_ptr(), cache_nbytes(k_cache, v_cache), payload.data_ptr(),
                        nbytes(payload), scales.data_ptr(), nbytes(scales), stream.cuda_stream)


def pkv_plan_repair(suffix_tokens: int, block_tokens: int, dirty_tokens: int, importance, kappa: float):
    """Resume planner: (repair mask uint8 [ceil(N/B)], |H|)."""
    imp = np.ascontiguousarray(importance, dtype=np.float32)
    assert imp.size == suffix_tokens
    nb = -(-int(suffix_tokens) // int(block_tokens)) if block_tokens > 0 else 0
    mask = np.zeros(max(1, nb), np.uint8)
    h = ctypes.c_int64()
    st = load().pkv_plan_repair(int(suffix_tokens), int(block_tokens), int(dirty_tokens),
                                imp.ctypes.data if imp.size else None, float(kappa), mask.ctypes.data,
                                ctypes.byref(h))
    if st != PKV_OK:
        raise PkvError(st, "pkv_plan_repair")
    return mask[:nb], int(h.value)


def pkv_plan_repair_status(suffix_tokens, block_tokens, dirty_tokens, importance_ptr, kappa, mask_ptr) -> int:
    return load().pkv_plan_repair(int(suffix_tokens), int(block_tokens), int(dirty_tokens), importance_ptr,
                                  float(kappa), mask_ptr, None)


def pkv_payload_size(shape, request):
    lib = load()
    m = make_model(shape)
    reqs = _Requests([request])
    pb, se = ctypes.c_uint64(), ctypes.c_uint64()
    st = lib.pkv_payload_size(ctypes.byref(m), reqs.array, ctypes.byref(pb), ctypes.byref(se))
    if st != PKV_OK:
        raise PkvError(st, "pkv_payload_size")
    return pb.value, se.value


class Plan:
    """Owns a pkv_plan_t*; freed by ``pkv_free`` or on garbage collection."""

    def __init__(self, handle: int):
        self.handle = handle

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.pkv_free(self.handle)
            self.handle = None


def pkv_restore_plan_status(shape, requests: Sequence) -> int:
    """Status of pkv_restore_plan (the plan, if built, is freed at once)."""
    lib = load()
    m = make_model(shape)
    reqs = _Requests(requests)
    out = ctypes.c_void_p()
    st = lib.pkv_restore_plan(ctypes.byref(m), reqs.array, reqs.count, ctypes.byref(out))
    if out.value:
        lib.pkv_free(out.value)
    return st


def pkv_restore_plan(shape, requests: Sequence) -> Plan:
    lib = load()
    m = make_model(shape)
    reqs = _Requests(requests)
    out = ctypes.c_void_p()
    st = lib.pkv_restore_plan(ctypes.byref(m), reqs.array, reqs.count, ctypes.byref(out))
    if st != PKV_OK:
        raise PkvError(st, "pkv_restore_plan")
    return Plan(out.value)


def pkv_plan_query(plan: Plan) -> dict:
    info = PkvPlanInfo()
    st = load().pkv_plan_query(plan.handle, ctypes.byref(info))
    if st != PKV_OK:
        raise PkvError(st, "pkv_plan_query")
    return {name: getattr(info, name) for name, _ in PkvPlanInfo._fields_}


def pkv_plan_payload_bytes(plan: Plan, req: int) -> int:
    """Bytes of request ``req``'s checkpoint payload, all layers."""
    out = ctypes.c_uint64()
    st = load().pkv_plan_payload_bytes(plan.handle, int(req), ctypes.byref(out))
    if st != PKV_OK:
        raise PkvError(st, "pkv_plan_payload_bytes")
    return int(out.value)


def pkv_plan_payload_bytes_status(plan_handle, req: int, out_ptr) -> int:
    return load().pkv_plan_payload_bytes(plan_handle, int(req), out_ptr)


def pkv_restore(plan: Plan, payload: int, payload_bytes: int, scales: int, scale_bytes: int, k_cache: int,
                v_cache: int, cache_bytes: int, stream: int = 0) -> None:
    """Enqueue a restore; pointers are device addresses, stream a hipStream_t (0 = default)."""
    st = load().pkv_restore(plan.handle, payload, payload_bytes, scales, scale_bytes, k_cache, v_cache,
                            cache_bytes, stream or None)
    if st != PKV_OK:
        raise PkvError(st, "pkv_restore")


def pkv_restore_status(plan: Plan, *args) -> int:
    return load().pkv_restore(plan.handle, *args)


def pkv_restore_from_host(plan: Plan, host_payload: int, host_payload_bytes: int, host_scales: int,
                          host_scale_bytes: int, payload: int, payload_bytes: int, scales: int, scale_bytes: int,
                          k_cache: int, v_cache: int, cache_bytes: int, stream: int = 0) -> None:
    """Enqueue a streamed restore from host memory; host_* are host addresses."""
    st = load().pkv_restore_from_host(plan.handle, host_payload, host_payload_bytes, host_scales, host_scale_bytes,
                                      payload, payload_bytes, scales, scale_bytes, k_cache, v_cache, cache_bytes,
                                      stream or None)
    if st != PKV_OK:
        raise PkvError(st, "pkv_restore_from_host")


def pkv_restore_from_host_status(plan: Plan, *args) -> int:
    return load().pkv_restore_from_host(plan.handle, *args)


def restore_from_host_tensors(plan: Plan, host_payload, host_scales, payload, scales, k_cache, v_cache,
                              stream=None) -> None:
    """Marshal torch tensors (host ones ideally pinned) into pkv_restore_from_host."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(k_cache.device)
    nbytes = lambda t: t.numel() * t.element_size()
    pkv_restore_from_host(plan, host_payload.data_ptr(), nbytes(host_payload), host_scales.data_ptr(),
                          nbytes(host_scales), payload.data_ptr(), nbytes(payload), scales.data_ptr(),
                          nbytes(scales), k_cache.data_ptr(), v_cache.data_ptr(), cache_nbytes(k_cache, v_cache),
                          stream.cuda_stream)


def pkv_restore_from_host_noalloc(plan: Plan, host_payload: int, host_payload_bytes: int, host_scales: int,
                                  host_scale_bytes: int, k_cache: int, v_cache: int, cache_bytes: int,
                                  stream: int = 0) -> None:
    """Enqueue the allocation-free streamed restore; host_* are pinned host addresses."""
    st = pkv_restore_from_host_noalloc_status(plan, host_payload, host_payload_bytes, host_scales, host_scale_bytes,
                                              k_cache, v_cache, cache_bytes, stream)
    if st != PKV_OK:
        raise PkvError(st, "pkv_restore_from_host_noalloc")


def pkv_restore_from_host_noalloc_status(plan: Plan, host_payload, host_payload_bytes, host_scales,
                                         host_scale_bytes, k_cache, v_cache, cache_bytes, stream=0) -> int:
    return load().pkv_restore_from_host_noalloc(plan.handle, host_payload, host_payload_bytes, host_scales,
                                                host_scale_bytes, k_cache, v_cache, cache_bytes, stream or None)


def restore_from_host_noalloc_tensors(plan: Plan, host_payload, host_scales, k_cache, v_cache, stream=None) -> None:
    """Marshal pinned host tensors and device caches into pkv_restore_from_host_noalloc."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(k_cache.device)
    nbytes = lambda t: t.numel() * t.element_size()
    pkv_restore_from_host_noalloc(plan, host_payload.data_ptr(), nbytes(host_payload), host_scales.data_ptr(),
                                  nbytes(host_scales), k_cache.data_ptr(), v_cache.data_ptr(),
                                  cache_nbytes(k_cache, v_cache), stream.cuda_stream)


def pkv_free(plan: Plan) -> None:
    if plan.handle:
        load().pkv_free(plan.handle)
        plan.handle = None


def restore_tensors(plan: Plan, payload, scales, k_cache, v_cache, stream=None) -> None:
    """Marshal torch device tensors (contiguous) and the current stream into pkv_restore."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(k_cache.device)
    nbytes = lambda t: t.numel() * t.element_size()
    pkv_restore(plan, payload.data_ptr(), nbytes(payload), scales.data_ptr(), nbytes(scales), k_cache.data_ptr(),
                v_cache.data_ptr(), cache_nbytes(k_cache, v_cache), stream.cuda_stream)
