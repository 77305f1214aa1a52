"""Device buffers for checkpoint writes and restores: torch supplies memory
and streams only.

* :class:`OldCaches` places the drawn suffix rows of every request into the
  old context's paged caches on the GPU (every other slot holds NaN).
* :class:`DeviceCheckpoint` writes the checkpoint from them with
  ``pkv_quantize_gather``.
* :class:`DeviceRestore` holds a checkpoint and the destination caches
  (pre-filled with a recomputable pattern), builds the restore plan and
  launches ``pkv_restore`` on the current stream.

No step of the method's arithmetic happens here.
"""
from __future__ import annotations

import atexit
import dataclasses
import multiprocessing as mp
import sys
from typing import Dict, Iterator, Optional, Sequence, Tuple

import numpy as np

from . import binding
from . import workloads as wl

_CHUNK = 1 << 26  # elements per pattern-fill / check chunk


def _to_int16(t):
    import torch
    return torch.where(t >= 32768, t - 65536, t).to(torch.int16)


# Worker processes that draw suffix rows (numpy only).  They are forked by
# start_workers() before the process first touches the GPU, so no worker
# inherits GPU state, and closed and joined by stop_workers() (also at exit).
_POOL = None


def start_workers(workers: Optional[int] = None):
    """Fork the draw workers now (call before any GPU work); returns the pool,
    or None for one worker."""
    global _POOL
    n = workers or wl.default_workers()
    if _POOL is None and n > 1:
        _POOL = mp.get_context("fork").Pool(n)
        atexit.register(stop_workers)
    return _POOL


def stop_workers() -> None:
    global _POOL
    if _POOL is not None:
        pool, _POOL = _POOL, None
        pool.close()
        pool.join()


def worker_pool():
    """The pool of :func:`start_workers`, or None."""
    return _POOL


def _gpu_initialised() -> bool:
    torch = sys.modules.get("torch")
    return torch is not None and torch.cuda.is_initialized()


def _draw_job(args):
    case, key = args
    return key, case.suffix_bits(*key)


def suffix_rows(case: wl.Case, layers: Sequence[int], workers: Optional[int] = None
                ) -> Iterator[Tuple[int, int, Tuple[np.ndarray, np.ndarray, np.ndarray]]]:
    """Yield (request, layer, (old slots, K bits, V bits)) for every layer in
    ``layers`` (layer-major) and every request.  Each distinct draw is made
    once and dropped after its last use: in the workers of
    :func:`start_workers` if they run; else, before the GPU is touched, in a
    pool forked for this call; else (``workers`` 1, or the GPU already in
    use, where forking is not safe) in this process."""
    order = [(ri, layer) for layer in layers for ri in range(len(case.requests))]
    keys = list(dict.fromkeys((ri, case.source_layer(l)) for ri, l in order))
    last_use = {(ri, case.source_layer(l)): i for i, (ri, l) in enumerate(order)}
    workers = min(workers or wl.default_workers(), len(keys))
    pool, own = None, False
    if workers > 1:
        pool = _POOL
        if pool is None and not _gpu_initialised():
            pool, own = mp.get_context("fork").Pool(workers), True
    results = pool.imap(_draw_job, [(case, k) for k in keys]) if pool is not None else \
        ((k, case.suffix_bits(*k)) for k in keys)
    try:
        drawn: Dict[Tuple[int, int], Tuple[np.ndarray, np.ndarray, np.ndarray]] = {}
        for i, (ri, layer) in enumerate(order):
            key = (ri, case.source_layer(layer))
            while key not in drawn:
                k, val = next(results)
                drawn[k] = val
            val = drawn[key]
            if last_use[key] == i:
                del drawn[key]
            yield ri, layer, val
    finally:
        if own:
            pool.terminate()
            pool.join()


def alloc_caches(shape, device, fill: Optional[int] = None):
    """K and V caches of ``shape`` on the device, each seen as
    ``[L][pool_pages][P][H][D]`` int16: two tensors (``KV_SEPARATE``), or the
    K and V views ``[:, :, 0]`` / ``[:, :, 1]`` of one
    ``[L][pool_pages][2][P][H][D]`` tensor (``KV_PAIRED``)."""
    import torch

    dims = (shape.num_layers, shape.pool_pages, shape.page_size, shape.num_kv_heads, shape.head_dim)
    make = (lambda d: torch.empty(d, dtype=torch.int16, device=device)) if fill is None else \
        (lambda d: torch.full(d, fill, dtype=torch.int16, device=device))
    if getattr(shape, "kv_layout", wl.KV_SEPARATE) == wl.KV_PAIRED:
        kv = make(dims[:2] + (2,) + dims[2:])
        return kv[:, :, 0], kv[:, :, 1]
    return make(dims), make(dims)


def _scatter_rows(cache_layer, slots, bits):
    """Write rows ``bits`` ``[n, H, D]`` into slots of one layer ``[pool_pages][P][H][D]``."""
    import torch

    P = cache_layer.shape[1]
    idx = torch.from_numpy(np.asarray(slots, dtype=np.int64)).to(cache_layer.device)
    cache_layer[idx // P, idx % P] = torch.from_numpy(bits.view(np.int16)).to(cache_layer.device)


class OldCaches:
    """The old context's K and V caches on the device, all layers."""

    def __init__(self, case: wl.Case, device: str = "cuda", workers: Optional[int] = None):
        import torch

        self.case = case
        s = case.src_shape
        nan = wl.cache_nan_bits(s.out_dtype)
        nan = nan - 65536 if nan >= 32768 else nan
        self.k, self.v = alloc_caches(s, device, nan)
        for ri, layer, (slots, kb, vb) in suffix_rows(case, range(s.num_layers), workers):
            _scatter_rows(self.k[layer], slots, kb)
            _scatter_rows(self.v[layer], slots, vb)
        torch.cuda.synchronize(device)


def alloc_checkpoint(case: wl.Case, device: str = "cuda"):
    """Zeroed payload (uint8) and scale (int16) device buffers of a case."""
    import torch

    payload = torch.zeros(max(16, case.payload_nbytes), dtype=torch.uint8, device=device)
    scales = torch.zeros(max(4, case.scale_elems), dtype=torch.int16, device=device)
    return payload, scales


class DeviceCheckpoint:
    """Checkpoint write of all layers from :class:`OldCaches` (one launch)."""

    def __init__(self, case: wl.Case, old: OldCaches, device: str = "cuda"):
        self.case = case
        self.old = old
        self.payload, self.scales = alloc_checkpoint(case, device)
        self.plan = binding.pkv_checkpoint_plan(case.src_shape, case.requests)
        self.info = binding.pkv_plan_query(self.plan)

    def write(self, stream=None) -> None:
        binding.quantize_gather_tensors(self.plan, self.old.k, self.old.v, self.payload, self.scales, stream)


def write_checkpoint_layerwise(case: wl.Case, payload, scales, device: str = "cuda",
                               workers: Optional[int] = None) -> None:
    """Write a case's checkpoint on the GPU one layer at a time, through one
    reusable old-cache layer (for cases whose old caches do not fit at once)."""
    import torch

    s1 = dataclasses.replace(case.src_shape, num_layers=1)
    nan = wl.cache_nan_bits(s1.out_dtype)
    nan = nan - 65536 if nan >= 32768 else nan
    k, v = alloc_caches(s1, device)
    current = None
    rows = []

    def flush(layer):
        k.fill_(nan)
        v.fill_(nan)
        for ri, (slots, kb, vb) in rows:
            _scatter_rows(k[0], slots, kb)
            _scatter_rows(v[0], slots, vb)
        reqs = [dataclasses.replace(r, payload_offset=case.layer_payload_offset(ri, layer),
                                    scale_offset=case.layer_scale_offset(ri, layer))
                for ri, r in enumerate(case.requests)]
        plan = binding.pkv_checkpoint_plan(s1, reqs)
        binding.quantize_gather_tensors(plan, k, v, payload, scales)
        torch.cuda.synchronize(device)
        binding.pkv_free(plan)

    for ri, layer, drawn in suffix_rows(case, range(case.shape.num_layers), workers):
        if current is not None and layer != current:
            flush(current)
            rows = []
        current = layer
        rows.append((ri, drawn))
    if current is not None:
        flush(current)


class DeviceRestore:
    """A checkpoint and the destination caches of a case, with its restore plan.

    ``checkpoint`` is ``None`` (write it on the GPU from the drawn old
    caches), a pair of host arrays (payload uint8, scales uint16) to upload, or
    a pair of device tensors to copy."""

    def __init__(self, case: wl.Case, device: str = "cuda", checkpoint=None, workers: Optional[int] = None):
        import torch

        self.case = case
        self.device = torch.device(device)
        s = case.shape
        self.payload, self.scales = alloc_checkpoint(case, device)
        if checkpoint is None:
            write_checkpoint_layerwise(case, self.payload, self.scales, device, workers)
        else:
            p, sc = checkpoint
            if isinstance(p, np.ndarray):
                self.payload[:p.size].copy_(torch.from_numpy(p))
                self.scales[:sc.size].copy_(torch.from_numpy(np.asarray(sc, np.uint16).view(np.int16)))
            else:
                self.payload.copy_(p)
                self.scales.copy_(sc)
        self.k_cache, self.v_cache = alloc_caches(s, self.device)
        self.prefill()
        self.plan = binding.pkv_restore_plan(s, case.requests)
        self.info = binding.pkv_plan_query(self.plan)

    def prefill(self) -> None:
        """Fill both caches with the generator's position-dependent pattern."""
        import torch

        s = self.case.shape
        page = s.page_size * s.row_elems
        pages_per_chunk = max(1, _CHUNK // page)
        for which, cache in ((0, self.k_cache), (1, self.v_cache)):
            seed = self.case.prefill_seed(which)
            for layer in range(s.num_layers):
                for p0 in range(0, s.pool_pages, pages_per_chunk):
                    p1 = min(s.pool_pages, p0 + pages_per_chunk)
                    start = layer * s.layer_elems + p0 * page
                    idx = torch.arange(start, start + (p1 - p0) * page, dtype=torch.int64, device=self.device)
                    cache[layer, p0:p1] = _to_int16(wl.prefill_bits_torch(idx, seed)).view(cache[layer, p0:p1].shape)
        torch.cuda.synchronize(self.device)

    def run(self, stream=None) -> None:
        binding.restore_tensors(self.plan, self.payload, self.scales, self.k_cache, self.v_cache, stream)

    def untouched_mismatches(self, written_slots: np.ndarray) -> int:
        """Elements outside ``written_slots`` (bool [pool_slots], same in every
        layer) that differ from the pre-fill pattern."""
        import torch

        s = self.case.shape
        row = s.row_elems
        keep = torch.from_numpy(~written_slots).to(self.device)
        bad = 0
        P = s.page_size
        pages_per_chunk = max(1, _CHUNK // (P * row))
        for which, cache in ((0, self.k_cache), (1, self.v_cache)):
            seed = self.case.prefill_seed(which)
            for layer in range(s.num_layers):
                base = layer * s.layer_elems
                for p0 in range(0, s.pool_pages, pages_per_chunk):
                    p1 = min(s.pool_pages, p0 + pages_per_chunk)
                    s0, s1 = p0 * P, p1 * P
                    idx = torch.arange(base + s0 * row, base + s1 * row, dtype=torch.int64, device=self.device)
                    want = _to_int16(wl.prefill_bits_torch(idx, seed)).view(s1 - s0, row)
                    got = cache[layer, p0:p1].reshape(s1 - s0, row)
                    diff = (got != want) & keep[s0:s1, None]
                    bad += int(diff.sum().item())
        return bad

    def rows(self, which: int, layer: int, slots: np.ndarray) -> np.ndarray:
        """uint16 bits of the given slots of one layer, ``[n, H, D]``."""
        import torch

        cache = self.k_cache if which == 0 else self.v_cache
        P = self.case.shape.page_size
        idx = torch.from_numpy(np.asarray(slots, dtype=np.int64)).to(self.device)
        return cache[layer][idx // P, idx % P].cpu().numpy().view(np.uint16)

    def host_caches(self):
        """Both caches on the host, ``[L][pool_pages][P][H][D]`` uint16 each, whatever the device layout."""
        return (self.k_cache.contiguous().cpu().numpy().view(np.uint16),
                self.v_cache.contiguous().cpu().numpy().view(np.uint16))
