"""Device buffers for a restore: torch supplies memory and streams only.

``DeviceRestore`` uploads a generated checkpoint, pre-fills the two caches
with a recomputable pattern, builds the plan through the C ABI and launches
``pkv_restore`` on the current torch stream.  No restore arithmetic happens
here.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import binding
from . import workloads as wl

_CHUNK = 1 << 26  # elements per pattern-fill / check chunk


def _to_int16(t):
    import torch
    return torch.where(t >= 32768, t - 65536, t).to(torch.int16)


class DeviceRestore:
    def __init__(self, case: wl.Case, device: str = "cuda", workers: Optional[int] = None):
        import torch

        self.case = case
        self.device = torch.device(device)
        s = case.shape
        case.warm(workers)
        self.payload = torch.empty(max(16, case.payload_nbytes), dtype=torch.uint8, device=self.device)
        self.scales = torch.empty(max(4, case.scale_elems), dtype=torch.int16, device=self.device)
        self.scales.fill_(wl.FP16_NAN_BITS)
        self._upload()
        cache_shape = (s.num_layers, s.pool_pages, s.page_size, s.num_kv_heads, s.head_dim)
        self.k_cache = torch.empty(cache_shape, dtype=torch.int16, device=self.device)
        self.v_cache = torch.empty(cache_shape, dtype=torch.int16, device=self.device)
        self.prefill()
        self.plan = binding.pkv_restore_plan(s, case.requests)
        self.info = binding.pkv_plan_query(self.plan)

    def _upload(self) -> None:
        import torch

        c = self.case
        for ri, r in enumerate(c.requests):
            first = {}
            for layer in range(c.shape.num_layers):
                pb, sb = c.encoded_layer(ri, layer)
                o = c.layer_payload_offset(ri, layer)
                so = c.layer_scale_offset(ri, layer)
                src = c.source_layer(layer)
                if src in first:  # repeated layer: device-to-device copy of its source
                    fo, fso = first[src]
                    self.payload[o:o + pb.size].copy_(self.payload[fo:fo + pb.size])
                    self.scales[so:so + sb.size].copy_(self.scales[fso:fso + sb.size])
                    continue
                first[src] = (o, so)
                self.payload[o:o + pb.size].copy_(torch.from_numpy(pb))
                self.scales[so:so + sb.size].copy_(torch.from_numpy(sb.reshape(-1).view(np.int16)))
        torch.cuda.synchronize(self.device)

    def prefill(self) -> None:
        """Fill both caches with the generator's position-dependent pattern."""
        import torch

        for which, cache in ((0, self.k_cache), (1, self.v_cache)):
            flat = cache.view(-1)
            seed = self.case.prefill_seed(which)
            for start in range(0, flat.numel(), _CHUNK):
                end = min(flat.numel(), start + _CHUNK)
                idx = torch.arange(start, end, dtype=torch.int64, device=self.device)
                flat[start:end] = _to_int16(wl.prefill_bits_torch(idx, seed))
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
        for which, cache in ((0, self.k_cache), (1, self.v_cache)):
            seed = self.case.prefill_seed(which)
            flat = cache.view(s.num_layers, s.pool_slots, row)
            slots_per_chunk = max(1, _CHUNK // row)
            for layer in range(s.num_layers):
                base = layer * s.layer_elems
                for s0 in range(0, s.pool_slots, slots_per_chunk):
                    s1 = min(s.pool_slots, s0 + slots_per_chunk)
                    idx = torch.arange(base + s0 * row, base + s1 * row, dtype=torch.int64, device=self.device)
                    want = _to_int16(wl.prefill_bits_torch(idx, seed)).view(s1 - s0, row)
                    diff = (flat[layer, s0:s1] != want) & keep[s0:s1, None]
                    bad += int(diff.sum().item())
        return bad

    def rows(self, which: int, layer: int, slots: np.ndarray) -> np.ndarray:
        """uint16 bits of the given slots of one layer, ``[n, H, D]``."""
        import torch

        cache = self.k_cache if which == 0 else self.v_cache
        s = self.case.shape
        flat = cache.view(s.num_layers, s.pool_slots, s.num_kv_heads, s.head_dim)
        idx = torch.from_numpy(np.asarray(slots, dtype=np.int64)).to(self.device)
        return flat[layer].index_select(0, idx).cpu().numpy().view(np.uint16)

    def host_caches(self):
        return (self.k_cache.cpu().numpy().view(np.uint16), self.v_cache.cpu().numpy().view(np.uint16))
