"""Seeded synthetic suffix-restore workloads.

This module is the one place where inputs are drawn; the CPU oracle
(``oracle/``), the tests and the benchmark consume what it draws.  It holds
none of the method's arithmetic: it draws the random parts of an edit and
resume (per-block precision tags, the repair mask, old and new page tables,
the edit shift, key and value tensors) and places the drawn values in the old
context's paged cache.  Checkpoints are written from those caches by the
quantize-and-gather step itself (the oracle's on the host, libpkv's on the
GPU); nothing here quantizes, dequantizes, rotates or places a restored row.

Value model (synthetic stand-in for the paper's long-context models, whose
weights and QA datasets are not available here): stored keys and values are
N(0, 1); a few rotary channel *pairs* ``(i, i + D/2)`` per (layer, head) are
outliers scaled by 8.  Because the outlier scale is applied to both channels
of a rotary pair, each pair stays an isotropic Gaussian, so a key rotated to
any old position has the same distribution as the pre-rotation key and the
stored (post-rotation) keys can be drawn directly.

Checkpoint sizes follow the format of ``include/pkv.h``: per layer, per tag,
per block a K tile and a V tile of B rows x H heads x D channels at 16, 8 or
4 bits per channel.
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

TAG_FP16, TAG_K8V8, TAG_K8V4, TAG_K4V4 = 0, 1, 2, 3
ROPE_HALF, ROPE_INTERLEAVED = 0, 1
TAG_NAMES = ("FP16", "K8V8", "K8V4", "K4V4")
KEY_BITS = (16, 8, 8, 4)
VALUE_BITS = (16, 8, 4, 4)
OUT_FP16, OUT_BF16 = 0, 1
KV_SEPARATE, KV_PAIRED = 0, 1  # device cache layouts (pkv_kv_layout_t)

FP16_NAN_BITS = 0x7E00

# Seed streams (spawn keys) so every piece can be regenerated in isolation.
_STREAM_TAGS, _STREAM_REPAIR, _STREAM_PAGES, _STREAM_POS, _STREAM_K, _STREAM_V = range(6)

CONFIG_NAMES = ("tiny", "llama8b_1l", "llama8b_32l", "llama70b", "batched16", "qwen3_32b_1l", "glm4_9b_1l",
                "llama33_70b_1l")
BASE_SEED = 26090


@dataclasses.dataclass(frozen=True)
class Shape:
    """Model and cache geometry shared by every request of a restore."""

    num_layers: int
    num_kv_heads: int
    head_dim: int
    block_tokens: int
    page_size: int
    pool_pages: int
    rope_theta: float
    out_dtype: int  # OUT_FP16 or OUT_BF16
    rope_style: int = 0  # ROPE_HALF or ROPE_INTERLEAVED
    rotary_dim: int = 0  # 0 = head_dim
    inv_freq: Optional[Tuple[float, ...]] = None  # explicit pair frequencies, else theta^(-2i/rotary_dim)
    kv_layout: int = 0  # KV_SEPARATE or KV_PAIRED (device caches only; host caches are always two arrays)

    @property
    def pool_slots(self) -> int:
        return self.pool_pages * self.page_size

    @property
    def row_elems(self) -> int:
        """Elements of one cache slot (all heads)."""
        return self.num_kv_heads * self.head_dim

    @property
    def layer_elems(self) -> int:
        return self.pool_slots * self.row_elems

    @property
    def cache_elems(self) -> int:
        return self.num_layers * self.layer_elems


@dataclasses.dataclass
class Request:
    """One resumed request: suffix geometry, edit shift, tags, repair mask, pages."""

    suffix_tokens: int
    delta: int
    dst_row0: int
    tags: np.ndarray  # uint8 [NB]
    repair: np.ndarray  # uint8 [NB], nonzero = block in the repair set
    page_table: np.ndarray  # int32 [num_logical_pages], -1 = unmapped
    payload_offset: int = 0  # bytes
    scale_offset: int = 0  # fp16 elements
    # The old context the checkpoint was written from (offload side):
    src_row0: int = 0  # omega_0, old logical row of suffix token 0 (= dst_row0 - delta)
    src_page_table: Optional[np.ndarray] = None  # int32, old context's logical -> physical pages

    @property
    def num_blocks(self) -> int:
        return len(self.tags)


def num_blocks(n_tokens: int, block_tokens: int) -> int:
    return -(-n_tokens // block_tokens)


def tile_nbytes(bits: int, shape: Shape) -> int:
    """Bytes of one K or V tile ([B][H][D]) stored with ``bits`` per channel."""
    return shape.block_tokens * shape.num_kv_heads * shape.head_dim * bits // 8


def encoded_layer_nbytes(shape: Shape, tags: np.ndarray) -> int:
    counts = np.bincount(np.asarray(tags, dtype=np.int64), minlength=4)
    return int(sum(int(counts[t]) * (tile_nbytes(KEY_BITS[t], shape) + tile_nbytes(VALUE_BITS[t], shape))
                   for t in range(4)))


def encoded_request_nbytes(shape: Shape, req: Request) -> Tuple[int, int]:
    """(payload bytes, scale fp16 elements) of one request's checkpoint."""
    return (shape.num_layers * encoded_layer_nbytes(shape, req.tags),
            shape.num_layers * req.num_blocks * shape.num_kv_heads * 4)


# ----------------------------------------------------------------------------
# Draws
# ----------------------------------------------------------------------------

def draw_layer(shape: Shape, seed: int, req_index: int, layer: int, n_tokens: int,
               outlier_pairs: int) -> Tuple[np.ndarray, np.ndarray]:
    """Stored (post-rotation) K and V of one layer: float32 ``[NB*B, H, D]``.

    Rows ``>= n_tokens`` (padding of the last block) are zero.
    """
    B, H, D = shape.block_tokens, shape.num_kv_heads, shape.head_dim
    rows = num_blocks(n_tokens, B) * B
    rk = _rng(seed, _STREAM_K, req_index, layer)
    rv = _rng(seed, _STREAM_V, req_index, layer)
    k = rk.standard_normal((rows, H, D), dtype=np.float32)
    v = rv.standard_normal((rows, H, D), dtype=np.float32)
    if outlier_pairs > 0:
        for h in range(H):
            pairs = rk.choice(D // 2, size=outlier_pairs, replace=False)
            ch = np.concatenate([pairs, pairs + D // 2])
            k[:, h, ch] *= np.float32(8.0)
    k[n_tokens:] = 0
    v[n_tokens:] = 0
    return k, v


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy=seed, spawn_key=tuple(key))))


# ----------------------------------------------------------------------------
# Pool pre-fill: a counter-based pattern so any region can be recomputed.
# ----------------------------------------------------------------------------

_PF_C1 = 0x45D9F3B  # < 2^31, so 32-bit x constant stays inside int64
_PF_C2 = 0x2C1B3C6D


def prefill_bits_np(flat_index: np.ndarray, seed: int) -> np.ndarray:
    """uint16 pre-fill pattern of cache elements at the given flat indices."""
    i = np.asarray(flat_index, dtype=np.int64)
    x = ((i & 0xFFFFFFFF) ^ ((i >> 32) * 0x9E37) ^ (seed & 0xFFFF)) & 0xFFFFFFFF
    x = ((x ^ (x >> 16)) * _PF_C1) & 0xFFFFFFFF
    x = ((x ^ (x >> 15)) * _PF_C2) & 0xFFFFFFFF
    x = x ^ (x >> 13)
    return ((x >> 8) & 0xFFFF).astype(np.uint16)


def prefill_bits_torch(flat_index, seed: int):
    """Same pattern as :func:`prefill_bits_np` on an int64 torch tensor."""
    i = flat_index
    x = ((i & 0xFFFFFFFF) ^ ((i >> 32) * 0x9E37) ^ (seed & 0xFFFF)) & 0xFFFFFFFF
    x = ((x ^ (x >> 16)) * _PF_C1) & 0xFFFFFFFF
    x = ((x ^ (x >> 15)) * _PF_C2) & 0xFFFFFFFF
    x = x ^ (x >> 13)
    return (x >> 8) & 0xFFFF


# ----------------------------------------------------------------------------
# Cases
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Case:
    """A complete synthetic restore problem.

    Layer ``l`` of request ``r`` is drawn with key ``(r, l % distinct_layers)``:
    with ``distinct_layers < num_layers`` later layers repeat the encoded
    bytes of earlier ones (still stored at their own addresses).
    """

    name: str
    shape: Shape
    requests: List[Request]
    seed: int
    distinct_layers: int
    outlier_pairs: int
    payload_nbytes: int = 0
    scale_elems: int = 0
    src_pool_pages: int = 0  # pages per layer of the old context's caches

    def __post_init__(self):
        self._assign_source_pages()
        off, soff = 0, 0
        for r in self.requests:
            r.payload_offset = off
            r.scale_offset = soff
            pb, se = encoded_request_nbytes(self.shape, r)
            off += _round_up(pb, 256)
            soff += _round_up(se, 64)
        self.payload_nbytes = off
        self.scale_elems = soff

    def _assign_source_pages(self) -> None:
        """Old-context placement: omega_0 = rho_0 - delta, each request's old
        logical pages on distinct random pages of a shared old pool (twice the
        pages needed)."""
        P = self.shape.page_size
        need = []
        for r in self.requests:
            # Hand-built test cases may pick rho_0 < delta; their old rows start at 0.
            r.src_row0 = max(0, int(r.dst_row0) - int(r.delta))
            need.append(-(-(r.src_row0 + r.suffix_tokens) // P))
        self.src_pool_pages = max(1, 2 * sum(need))
        perm = _rng(self.seed, 7).permutation(self.src_pool_pages).astype(np.int32)
        k = 0
        for r, n in zip(self.requests, need):
            r.src_page_table = perm[k:k + n].copy()
            k += n

    @property
    def src_shape(self) -> Shape:
        """Geometry of the old context's caches."""
        return dataclasses.replace(self.shape, pool_pages=self.src_pool_pages)

    def old_cache_layer(self, which: int, layer: int) -> np.ndarray:
        """Bit patterns (cache dtype) of one layer of the old K (0) or V (1)
        cache, ``[src_pool_pages, P, H, D]``: each request's suffix rows hold
        its drawn values at their old slots; every other slot holds NaN, so a
        read of a wrong slot shows."""
        s = self.src_shape
        flat = np.full((s.pool_slots, s.num_kv_heads, s.head_dim), cache_nan_bits(s.out_dtype), dtype=np.uint16)
        for ri in range(len(self.requests)):
            slots, k, v = self.suffix_bits(ri, layer)
            flat[slots] = k if which == 0 else v
        return flat.reshape(s.pool_pages, s.page_size, s.num_kv_heads, s.head_dim)

    def host_old_caches(self) -> Tuple[np.ndarray, np.ndarray]:
        """Old K and V caches ``[L, src_pool_pages, P, H, D]`` (small cases)."""
        L = self.shape.num_layers
        return (np.stack([self.old_cache_layer(0, l) for l in range(L)]),
                np.stack([self.old_cache_layer(1, l) for l in range(L)]))

    # -- raw draws ---------------------------------------------------------
    def source_layer(self, layer: int) -> int:
        return layer % self.distinct_layers

    def raw_layer(self, req_index: int, layer: int) -> Tuple[np.ndarray, np.ndarray]:
        r = self.requests[req_index]
        return draw_layer(self.shape, self.seed, req_index, self.source_layer(layer), r.suffix_tokens,
                          self.outlier_pairs)

    def suffix_bits(self, req_index: int, layer: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """(old slots [N], K bits [N, H, D], V bits [N, H, D]) of one request's
        suffix rows in one layer of the old caches (cache dtype)."""
        r = self.requests[req_index]
        k, v = self.raw_layer(req_index, layer)
        P = self.shape.page_size
        rows = r.src_row0 + np.arange(r.suffix_tokens)
        slots = r.src_page_table[rows // P].astype(np.int64) * P + rows % P
        return (slots, to_cache_bits(k[:r.suffix_tokens], self.shape.out_dtype),
                to_cache_bits(v[:r.suffix_tokens], self.shape.out_dtype))

    def layer_payload_offset(self, req_index: int, layer: int) -> int:
        r = self.requests[req_index]
        return r.payload_offset + layer * encoded_layer_nbytes(self.shape, r.tags)

    def layer_scale_offset(self, req_index: int, layer: int) -> int:
        r = self.requests[req_index]
        return r.scale_offset + layer * r.num_blocks * self.shape.num_kv_heads * 4

    # -- pool ------------------------------------------------------------
    def prefill_seed(self, which: int) -> int:
        return (self.seed * 2 + which) & 0xFFFF

    def host_prefill(self, which: int) -> np.ndarray:
        """uint16 ``[L, pool_pages, P, H, D]`` pre-fill of the K (0) or V (1) cache."""
        n = self.shape.cache_elems
        bits = prefill_bits_np(np.arange(n, dtype=np.int64), self.prefill_seed(which))
        s = self.shape
        return bits.reshape(s.num_layers, s.pool_pages, s.page_size, s.num_kv_heads, s.head_dim)

    # -- accounting (data volume, not arithmetic) -------------------------
    def restored_tokens(self) -> int:
        """Tokens restored per layer summed over requests (rows of F blocks)."""
        total = 0
        B = self.shape.block_tokens
        for r in self.requests:
            n_valid = np.minimum(B, r.suffix_tokens - np.arange(r.num_blocks) * B)
            total += int(n_valid[np.asarray(r.repair) == 0].sum())
        return total

    def algorithmic_bytes(self) -> Dict[str, int]:
        """Bytes a restore must move: payload of F blocks, their scales, output rows."""
        s = self.shape
        B, H, D = s.block_tokens, s.num_kv_heads, s.head_dim
        read = 0
        scales = 0
        for r in self.requests:
            f = np.asarray(r.repair) == 0
            n_valid = np.minimum(B, r.suffix_tokens - np.arange(r.num_blocks) * B)
            for tag in range(4):
                sel = f & (np.asarray(r.tags) == tag)
                rows = int(n_valid[sel].sum())
                read += rows * H * D * (KEY_BITS[tag] + VALUE_BITS[tag]) // 8
                if tag != TAG_FP16:
                    scales += int(sel.sum()) * H * 4 * 2
        tok = self.restored_tokens()
        written = tok * H * D * 2 * 2
        L = s.num_layers
        return {"payload_read": L * read, "scale_read": L * scales, "written": L * written,
                "total": L * (read + scales + written)}


def cache_nan_bits(out_dtype: int) -> int:
    return FP16_NAN_BITS if out_dtype == OUT_FP16 else 0x7FC0


def to_cache_bits(x: np.ndarray, out_dtype: int) -> np.ndarray:
    """Bit patterns of finite float values stored in a fp16 or bf16 cache
    (round to nearest even; no torch, so it is safe in forked workers)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if out_dtype == OUT_FP16:
        return x.astype(np.float16).view(np.uint16)
    assert np.isfinite(x).all()
    b = x.view(np.uint32)
    return ((b + (((b >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def default_workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _round_up(x: int, a: int) -> int:
    return (x + a - 1) // a * a


# ----------------------------------------------------------------------------
# Draws of tags, repair sets, positions and page tables
# ----------------------------------------------------------------------------

def draw_tags(rng: np.random.Generator, nb: int, mix: Sequence[float], int4_tag: int = TAG_K8V4) -> np.ndarray:
    """Per-block tags from a (int4, int8, fp16) mix; int4 maps to K8V4 (or K4V4)."""
    choices = np.array([int4_tag, TAG_K8V8, TAG_FP16], dtype=np.uint8)
    p = np.asarray(mix, dtype=np.float64)
    return choices[rng.choice(3, size=nb, p=p / p.sum())]


def draw_repair_edit_local(rng: np.random.Generator, nb: int, frac: float, local_share: float = 0.8) -> np.ndarray:
    """Repair mask: a contiguous run from block 0 (the edit-local dirty window)
    holding ``local_share`` of the repaired blocks, plus sparse random blocks."""
    n_rep = int(round(frac * nb))
    n_local = min(n_rep, int(round(local_share * n_rep)))
    mask = np.zeros(nb, dtype=np.uint8)
    mask[:n_local] = 1
    rest = np.arange(n_local, nb)
    extra = rng.choice(rest, size=min(len(rest), n_rep - n_local), replace=False)
    mask[extra] = 1
    return mask


def draw_positions(rng: np.random.Generator, delta: int, min_old: int = 1024, max_old: int = 8191) -> int:
    """rho_0 = omega_0 + delta with omega_0 uniform so that rho_0 >= min_old."""
    lo = max(0, -delta) + min_old
    omega0 = int(rng.integers(lo, max(lo, max_old) + 1))
    return omega0 + delta


def private_page_table(rng: np.random.Generator, rows_end: int, page_size: int, pool_factor: int = 2):
    """Map every logical page covering ``[0, rows_end)`` to a distinct random
    page of a pool ``pool_factor`` times larger.  Returns (table, pool_pages)."""
    nlp = -(-rows_end // page_size)
    pool = pool_factor * nlp
    return rng.choice(pool, size=nlp, replace=False).astype(np.int32), pool


def llama3_inv_freq(theta: float, dim: int, factor: float = 8.0, low_freq_factor: float = 1.0,
                    high_freq_factor: float = 4.0, original_max_position: int = 8192) -> Tuple[float, ...]:
    """Rotary frequencies with Llama-3's published long-context scaling (a
    model-configuration input): pairs whose wavelength is below
    original/high_freq_factor keep theta^(-2i/dim), those above
    original/low_freq_factor are divided by `factor`, and the band between
    is a linear blend in original/wavelength."""
    base = theta ** (-np.arange(0, dim, 2, dtype=np.float64) / dim)
    wavelen = 2 * math.pi / base
    low_wl = original_max_position / low_freq_factor
    high_wl = original_max_position / high_freq_factor
    smooth = (original_max_position / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    blended = (1 - smooth) * base / factor + smooth * base
    out = np.where(wavelen < high_wl, base, np.where(wavelen > low_wl, base / factor, blended))
    return tuple(float(x) for x in out)


# Public architecture facts of the paper's model families (KV heads, head
# dim, RoPE), at one layer and an 8K-token suffix.
MODEL_ROPE = {
    # name: (num_kv_heads, head_dim, theta, rope_style, rotary_dim, scaled frequencies)
    "qwen3_32b_1l": (8, 128, 1.0e6, ROPE_HALF, 0, False),
    "glm4_9b_1l": (2, 128, 1.0e4, ROPE_INTERLEAVED, 64, False),
    "llama33_70b_1l": (8, 128, 5.0e5, ROPE_HALF, 0, True),
}


def make_case(name: str, seed: Optional[int] = None, distinct_layers: Optional[int] = None,
              int4_tag: int = TAG_K8V4) -> Case:
    """One of the five named workloads (see ``CONFIG_NAMES``)."""
    idx = CONFIG_NAMES.index(name)
    seed = BASE_SEED + idx if seed is None else seed
    g = lambda stream: _rng(seed, stream)
    if name == "tiny":
        B, P, N = 16, 16, 512
        nb = num_blocks(N, B)
        tags = g(_STREAM_TAGS).integers(0, 3, size=nb).astype(np.uint8)
        tags = np.array([int4_tag, TAG_K8V8, TAG_FP16], dtype=np.uint8)[tags]
        repair = np.zeros(nb, np.uint8)
        repair[g(_STREAM_REPAIR).choice(nb, size=4, replace=False)] = 1
        pt = g(_STREAM_PAGES).permutation(64).astype(np.int32)
        shape = Shape(1, 2, 64, B, P, 64, 10000.0, OUT_FP16)
        req = Request(N, 37, 337, tags, repair, pt)
        return Case(name, shape, [req], seed, distinct_layers or 1, outlier_pairs=0)
    if name in ("llama8b_1l", "llama8b_32l", "llama70b"):
        if name == "llama8b_1l":
            L, B, P, N, out, theta = 1, 32, 16, 8192, OUT_FP16, 500000.0
            mix, rep = (0.7, 0.2, 0.1), 0.10
            delta = int(g(_STREAM_POS).integers(-2048, 2049))
        elif name == "llama8b_32l":
            L, B, P, N, out, theta = 32, 32, 16, 32768, OUT_BF16, 500000.0
            mix, rep, delta = (0.7, 0.2, 0.1), 0.15, -1500
        else:
            L, B, P, N, out, theta = 80, 64, 32, 65536, OUT_BF16, 500000.0
            mix, rep, delta = (0.6, 0.3, 0.1), 0.12, 4096
        nb = num_blocks(N, B)
        tags = draw_tags(g(_STREAM_TAGS), nb, mix, int4_tag)
        repair = draw_repair_edit_local(g(_STREAM_REPAIR), nb, rep)
        rho0 = draw_positions(g(_STREAM_POS) if name != "llama8b_1l" else _rng(seed, _STREAM_POS, 1), delta)
        pt, pool = private_page_table(g(_STREAM_PAGES), rho0 + N, P)
        shape = Shape(L, 8, 128, B, P, pool, theta, out)
        req = Request(N, delta, rho0, tags, repair, pt)
        return Case(name, shape, [req], seed, distinct_layers or L, outlier_pairs=1)
    if name == "batched16":
        return make_batched(seed, distinct_layers=distinct_layers or 2, int4_tag=int4_tag)
    if name in MODEL_ROPE:
        H, D, theta, style, rdim, scaled = MODEL_ROPE[name]
        B, P, N = 32, 16, 8192
        nb = num_blocks(N, B)
        tags = draw_tags(g(_STREAM_TAGS), nb, (0.7, 0.2, 0.1), int4_tag)
        repair = draw_repair_edit_local(g(_STREAM_REPAIR), nb, 0.10)
        delta = int(g(_STREAM_POS).integers(-4096, 4097))
        rho0 = draw_positions(_rng(seed, _STREAM_POS, 1), delta)
        pt, pool = private_page_table(g(_STREAM_PAGES), rho0 + N, P)
        inv = llama3_inv_freq(theta, D) if scaled else None
        shape = Shape(1, H, D, B, P, pool, theta, OUT_BF16, style, rdim, inv)
        req = Request(N, delta, rho0, tags, repair, pt)
        return Case(name, shape, [req], seed, distinct_layers or 1, outlier_pairs=1)
    raise ValueError(name)


def make_batched(seed: int, n_req: int = 16, num_layers: int = 32, pool_slots: int = 1 << 20,
                 n_range: Tuple[int, int] = (4096, 65536), delta_range: Tuple[int, int] = (-8192, 8192),
                 distinct_layers: int = 2, int4_tag: int = TAG_K8V4, B: int = 32, P: int = 16,
                 H: int = 8, D: int = 128) -> Case:
    """Batched resumes sharing one paged pool with interleaved page ownership."""
    r_pos = _rng(seed, _STREAM_POS)
    r_tags = _rng(seed, _STREAM_TAGS)
    r_rep = _rng(seed, _STREAM_REPAIR)
    r_pages = _rng(seed, _STREAM_PAGES)
    pool_pages = pool_slots // P
    reqs = []
    spans = []
    for _ in range(n_req):
        N = int(r_pos.integers(n_range[0], n_range[1] + 1))
        delta = int(r_pos.integers(delta_range[0], delta_range[1] + 1))
        rho0 = draw_positions(r_pos, delta)
        nb = num_blocks(N, B)
        mix = r_tags.dirichlet((1.0, 1.0, 1.0))
        tags = draw_tags(r_tags, nb, mix, int4_tag)
        repair = draw_repair_edit_local(r_rep, nb, float(r_rep.uniform(0.05, 0.20)))
        first, last = rho0 // P, (rho0 + N - 1) // P
        spans.append((first, last))
        reqs.append([N, delta, rho0, tags, repair])
    need = sum(l - f + 1 for f, l in spans)
    if need > pool_pages:
        raise ValueError(f"batched case needs {need} pages, pool has {pool_pages}")
    perm = r_pages.permutation(pool_pages).astype(np.int32)
    tables = [np.full(l + 1, -1, dtype=np.int32) for f, l in spans]
    cursor = [f for f, l in spans]
    k = 0
    live = True
    while live:  # deal pool pages round-robin so ownership interleaves
        live = False
        for i, (f, l) in enumerate(spans):
            if cursor[i] <= l:
                tables[i][cursor[i]] = perm[k]
                k += 1
                cursor[i] += 1
                live = True
    shape = Shape(num_layers, H, D, B, P, pool_pages, 500000.0, OUT_BF16)
    requests = [Request(N, d, r0, t, rp, tables[i]) for i, (N, d, r0, t, rp) in enumerate(reqs)]
    return Case("batched16", shape, requests, seed, distinct_layers, outlier_pairs=1)


def make_custom(seed: int, *, L: int = 1, H: int = 2, D: int = 64, B: int = 16, P: int = 16,
                n_tokens: Sequence[int] = (100,), deltas: Sequence[int] = (5,), rho0s: Optional[Sequence[int]] = None,
                mix: Sequence[float] = (1 / 3, 1 / 3, 1 / 3), tag_set: Sequence[int] = (TAG_K8V4, TAG_K8V8, TAG_FP16),
                repair_frac: float = 0.2, repair_all: bool = False, out_dtype: int = OUT_FP16,
                theta: float = 10000.0, outlier_pairs: int = 0, pool_factor: int = 2) -> Case:
    """Small parametrised case for property tests (shared private pool, disjoint pages)."""
    r = _rng(seed, 99)
    reqs = []
    ends = []
    for i, N in enumerate(n_tokens):
        delta = int(deltas[i % len(deltas)])
        rho0 = int(rho0s[i]) if rho0s is not None else int(r.integers(0, 3 * P)) + max(0, 0)
        nb = num_blocks(N, B)
        p = np.asarray(mix, dtype=np.float64)
        tags = np.asarray(tag_set, dtype=np.uint8)[r.choice(len(tag_set), size=nb, p=p / p.sum())]
        if repair_all:
            repair = np.ones(nb, np.uint8)
        else:
            repair = (r.random(nb) < repair_frac).astype(np.uint8)
        reqs.append([N, delta, rho0, tags, repair])
        ends.append(rho0 + N)
    nlps = [max(1, -(-e // P)) for e in ends]
    pool = pool_factor * sum(nlps)
    perm = r.permutation(pool).astype(np.int32)
    tables = []
    k = 0
    for n in nlps:
        tables.append(perm[k:k + n].copy())
        k += n
    shape = Shape(L, H, D, B, P, pool, float(theta), out_dtype)
    requests = [Request(N, d, r0, t, rp, tables[i]) for i, (N, d, r0, t, rp) in enumerate(reqs)]
    return Case("custom", shape, requests, seed, L, outlier_pairs)
