"""CPU oracle of PatchKV's offload-side quantize-and-gather.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  It states in plain fp64 NumPy what the offload kernel
computes when a checkpoint is written (PatchKV Section IV-D: a fused kernel
gathers block rows, computes scales, packs FP16 / 8-bit / 4-bit payloads and
clusters same-representation blocks into contiguous runs; the resume side is
``oracle/restore.py``):

for every request, layer and block ``b`` of the suffix (all blocks: the repair
set is not known when the checkpoint is written):

1. gather the block's valid rows from the old context's paged cache: token
   ``t`` sits on old logical row ``omega_0 + b*B + t``, i.e. slot
   ``row mod P`` of page ``page_table[row div P]``;
2. per KV head and per K/V, over the valid rows only:
   * FP16 tag: store the binary16 value nearest to the cache value;
   * b-bit tag (b = 8 or 4): zero = the largest binary16 not above the
     minimum, scale = the smallest binary16 not below (max - zero)/(2^b - 1),
     code = round-half-even((x - zero) / scale) in double precision, clipped
     to [0, 2^b - 1] (a zero scale means every value equals the zero: code 0);
3. write the tiles token-major ``[B][H][D]`` (padding rows of a partial last
   block are code 0 / +0.0) in the clustered layout: per layer, runs of
   FP16, K8V8, K8V4, K4V4 blocks, ascending blocks within a run, K tile then
   V tile; 4-bit codes two per byte, channel 2j in the low nibble of byte j;
4. scales as binary16 ``[L][NB][H][2 (K, V)][2 (scale, zero)]``; FP16 tiles
   get scale 0 and zero 0.

The rounding directions (readings of the paper, which only says scales are
computed) make ``|x - (code*scale + zero)| <= scale/2`` hold exactly.
"""
from __future__ import annotations

from typing import Dict, Sequence, Tuple

import numpy as np

FP16, K8V8, K8V4, K4V4 = 0, 1, 2, 3
KEY_BITS = {FP16: 16, K8V8: 8, K8V4: 8, K4V4: 4}
VALUE_BITS = {FP16: 16, K8V8: 8, K8V4: 4, K4V4: 4}
OUT_FP16, OUT_BF16 = 0, 1

_F16_MAX = 65504.0


# --------------------------------------------------------------------------
# binary16 helpers written from the format's definition
# --------------------------------------------------------------------------

def _f16_values_from_bits(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def _f16_next_down(bits: np.ndarray) -> np.ndarray:
    """Bit pattern of the next binary16 toward -inf (finite inputs)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.int32)
    neg = (b & 0x8000) != 0
    mag = b & 0x7FFF
    out = np.where(neg, b + 1, np.where(mag == 0, 0x8001, b - 1))
    return out.astype(np.uint16)


def _f16_next_up(bits: np.ndarray) -> np.ndarray:
    """Bit pattern of the next binary16 toward +inf (finite inputs)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.int32)
    neg = (b & 0x8000) != 0
    mag = b & 0x7FFF
    out = np.where(~neg, b + 1, np.where(mag == 0, 0x0001, b - 1))
    return out.astype(np.uint16)


def f16_floor(x: np.ndarray) -> np.ndarray:
    """Bits of the largest binary16 <= x (x finite, |x| <= 65504)."""
    x = np.asarray(x, dtype=np.float64)
    near = x.astype(np.float16).view(np.uint16)
    above = _f16_values_from_bits(near) > x
    return np.where(above, _f16_next_down(near), near).astype(np.uint16)


def f16_ceil(x: np.ndarray) -> np.ndarray:
    """Bits of the smallest binary16 >= x (x finite, |x| <= 65504)."""
    x = np.asarray(x, dtype=np.float64)
    near = x.astype(np.float16).view(np.uint16)
    below = _f16_values_from_bits(near) < x
    return np.where(below, _f16_next_up(near), near).astype(np.uint16)


def cache_values(bits: np.ndarray, cache_dtype: int) -> np.ndarray:
    """fp64 values of fp16 / bf16 cache bit patterns."""
    bits = np.asarray(bits, dtype=np.uint16)
    if cache_dtype == OUT_FP16:
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Step 1: gather
# --------------------------------------------------------------------------

def source_slots(shape, req, block: int) -> np.ndarray:
    """Old-cache slot of every valid token of a block (``req.src_row0`` and
    the old context's page table ``req.src_page_table``)."""
    B, P = shape.block_tokens, shape.page_size
    n = min(B, req.suffix_tokens - block * B)
    slots = np.empty(n, dtype=np.int64)
    for t in range(n):
        row = req.src_row0 + block * B + t
        page = int(req.src_page_table[row // P])
        if page < 0 or page >= shape.pool_pages:
            raise ValueError("source row on an unmapped or out-of-range page")
        slots[t] = page * P + row % P
    return slots


# --------------------------------------------------------------------------
# Step 2: quantize one (block, head) tile of n valid rows x D channels
# --------------------------------------------------------------------------

def quantize_tile(x: np.ndarray, bits: int) -> Tuple[np.ndarray, int, int]:
    """(codes uint8 [n, D], scale bits, zero bits) of one head's tile."""
    qmax = (1 << bits) - 1
    # Signed zeros: a -0.0 extreme counts as +0.0 (adding +0.0 maps -0 to +0).
    zero_bits = int(f16_floor(np.array(float(x.min()) + 0.0)))
    zero = float(_f16_values_from_bits(np.array(zero_bits)))
    span = (float(x.max()) - zero) + 0.0  # exact: both are short binary fractions
    scale_bits = int(f16_ceil(np.array(span / qmax)))
    scale = float(_f16_values_from_bits(np.array(scale_bits)))
    if scale == 0.0:
        return np.zeros(x.shape, dtype=np.uint8), scale_bits, zero_bits
    codes = np.clip(np.rint((x - zero) / scale), 0, qmax)
    return codes.astype(np.uint8), scale_bits, zero_bits


def pack_tile(codes: np.ndarray, bits: int) -> np.ndarray:
    """Bytes of a code tile ``[B, H, D]`` (8-bit: one per channel; 4-bit: channel 2j low nibble)."""
    flat = codes.reshape(-1).astype(np.uint8)
    if bits == 8:
        return flat
    lo, hi = flat[0::2], flat[1::2]
    return (lo | (hi << 4)).astype(np.uint8)


def encode_tile(x: np.ndarray, n_valid: int, bits: int) -> Tuple[np.ndarray, np.ndarray]:
    """Encode one K or V tile ``[B, H, D]`` (rows >= n_valid are padding).
    Returns (bytes, per-head [H, 2] (scale bits, zero bits))."""
    B, H, D = x.shape
    sz = np.zeros((H, 2), dtype=np.uint16)
    if bits == 16:
        h = np.zeros((B, H, D), dtype=np.float16)
        h[:n_valid] = x[:n_valid].astype(np.float16)  # nearest binary16
        return h.view(np.uint8).reshape(-1), sz
    codes = np.zeros((B, H, D), dtype=np.uint8)
    for head in range(H):
        c, s, z = quantize_tile(x[:n_valid, head, :], bits)
        codes[:n_valid, head, :] = c
        sz[head] = (s, z)
    return pack_tile(codes, bits), sz


# --------------------------------------------------------------------------
# Steps 3-4: clustered layout
# --------------------------------------------------------------------------

def layer_layout_bytes(tags: Sequence[int], B: int, H: int, D: int) -> int:
    return sum(B * H * D * (KEY_BITS[int(t)] + VALUE_BITS[int(t)]) // 8 for t in tags)


def quantize_tiles_many(x: np.ndarray, n_valid: np.ndarray, bits: int) -> Tuple[np.ndarray, np.ndarray]:
    """The per-tile definition of :func:`quantize_tile` applied to many tiles
    at once: ``x`` fp64 ``[nb, B, H, D]``, rows ``>= n_valid[i]`` are padding.
    Returns (codes uint8 [nb, B, H, D] with padding rows 0, bits [nb, H, 2] (scale, zero))."""
    nb, B, H, D = x.shape
    qmax = (1 << bits) - 1
    valid = (np.arange(B)[None, :] < np.asarray(n_valid)[:, None])[:, :, None, None]
    lo = np.where(valid, x, np.inf).min(axis=(1, 3)) + 0.0  # -0 counts as +0
    hi = np.where(valid, x, -np.inf).max(axis=(1, 3))
    zero_bits = f16_floor(lo)
    zero = _f16_values_from_bits(zero_bits)
    scale_bits = f16_ceil(((hi - zero) + 0.0) / qmax)
    scale = _f16_values_from_bits(scale_bits)
    safe = np.where(scale > 0, scale, 1.0)[:, None, :, None]
    q = np.clip(np.rint((x - zero[:, None, :, None]) / safe), 0, qmax)
    q = np.where((scale > 0)[:, None, :, None] & valid, q, 0)
    return q.astype(np.uint8), np.stack([scale_bits, zero_bits], axis=-1)


def gather_rows(shape, req, layer_cache: np.ndarray) -> np.ndarray:
    """Step 1 for one layer: the request's suffix rows, in token order, from
    one layer of an old cache (uint16 ``[pool_pages, P, H, D]``)."""
    H, D = shape.num_kv_heads, shape.head_dim
    flat = np.asarray(layer_cache, dtype=np.uint16).reshape(-1, H, D)
    nb = len(req.tags)
    if nb == 0:
        return np.zeros((0, H, D), np.uint16)
    return np.concatenate([flat[source_slots(shape, req, b)] for b in range(nb)])


def quantize_rows(shape, req, k_rows: np.ndarray, v_rows: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Steps 2-4 for one layer of one request from its gathered suffix rows
    (uint16 cache bit patterns ``[suffix_tokens, H, D]``): (payload bytes,
    scale bits ``[NB, H, 2, 2]``)."""
    B, H, D = shape.block_tokens, shape.num_kv_heads, shape.head_dim
    nb = len(req.tags)
    n_valid = np.minimum(B, req.suffix_tokens - np.arange(nb) * B)
    scales = np.zeros((nb, H, 2, 2), dtype=np.uint16)
    tiles = []
    for rows in (k_rows, v_rows):
        rows = np.asarray(rows, dtype=np.uint16).reshape(-1, H, D)
        assert rows.shape[0] == req.suffix_tokens
        x = np.zeros((nb * B, H, D), dtype=np.float64)
        x[:req.suffix_tokens] = cache_values(rows, shape.out_dtype)
        tiles.append(x.reshape(nb, B, H, D))
    pieces = []
    tags = np.asarray(req.tags)
    for tag in (FP16, K8V8, K8V4, K4V4):
        blocks = np.nonzero(tags == tag)[0]
        if len(blocks) == 0:
            continue
        parts = []
        for which, bits in ((0, KEY_BITS[tag]), (1, VALUE_BITS[tag])):
            x = tiles[which][blocks]
            if bits == 16:
                h = x.astype(np.float16)
                h[np.arange(B)[None, :] >= n_valid[blocks][:, None]] = 0
                parts.append(h.view(np.uint8).reshape(len(blocks), -1))
            else:
                codes, sz = quantize_tiles_many(x, n_valid[blocks], bits)
                scales[blocks, :, which, :] = sz
                parts.append(pack_tile(codes, bits).reshape(len(blocks), -1))
        pieces.append(np.concatenate(parts, axis=1).reshape(-1))  # K tile then V tile, per block
    payload = np.concatenate(pieces) if pieces else np.zeros(0, np.uint8)
    return payload, scales


def quantize_layer(shape, req, k_layer: np.ndarray, v_layer: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """One layer of one request's checkpoint from that layer of the old caches
    (uint16 ``[pool_pages, P, H, D]``): (payload bytes, scale bits ``[NB, H, 2, 2]``)."""
    return quantize_rows(shape, req, gather_rows(shape, req, k_layer), gather_rows(shape, req, v_layer))


def quantize_gather(shape, requests: Sequence, k_cache: np.ndarray, v_cache: np.ndarray,
                    payload_bytes: int, scale_elems: int) -> Tuple[np.ndarray, np.ndarray]:
    """Encode every block of every request from the caches (uint16 bit
    patterns ``[L, pool_pages, P, H, D]`` of dtype ``shape.out_dtype``) into a
    payload (uint8 [payload_bytes]) and scales (uint16 [scale_elems]).
    Bytes outside the requests' checkpoints are left 0."""
    L, B, H, D = shape.num_layers, shape.block_tokens, shape.num_kv_heads, shape.head_dim
    payload = np.zeros(payload_bytes, dtype=np.uint8)
    scales = np.zeros(scale_elems, dtype=np.uint16)
    for req in requests:
        nb = len(req.tags)
        layer_bytes = layer_layout_bytes(req.tags, B, H, D)
        for layer in range(L):
            pb, sb = quantize_layer(shape, req, k_cache[layer], v_cache[layer])
            o = req.payload_offset + layer * layer_bytes
            payload[o:o + pb.size] = pb
            so = req.scale_offset + layer * nb * H * 4
            scales[so:so + sb.size] = sb.reshape(-1)
    return payload, scales


def quantize_gather_per_tile(shape, requests: Sequence, k_cache: np.ndarray, v_cache: np.ndarray,
                             payload_bytes: int, scale_elems: int) -> Tuple[np.ndarray, np.ndarray]:
    """The same result tile by tile with :func:`encode_tile` (slow; for small cases)."""
    L, B, H, D = shape.num_layers, shape.block_tokens, shape.num_kv_heads, shape.head_dim
    payload = np.zeros(payload_bytes, dtype=np.uint8)
    scales = np.zeros(scale_elems, dtype=np.uint16)
    kf = np.asarray(k_cache, dtype=np.uint16).reshape(L, -1, H, D)
    vf = np.asarray(v_cache, dtype=np.uint16).reshape(L, -1, H, D)
    for req in requests:
        nb = len(req.tags)
        order = [b for tag in (FP16, K8V8, K8V4, K4V4) for b in range(nb) if int(req.tags[b]) == tag]
        for layer in range(L):
            pos = req.payload_offset + layer * layer_layout_bytes(req.tags, B, H, D)
            for b in order:
                tag = int(req.tags[b])
                n = min(B, req.suffix_tokens - b * B)
                slots = source_slots(shape, req, b)
                for which, (cache, bits) in enumerate(((kf, KEY_BITS[tag]), (vf, VALUE_BITS[tag]))):
                    x = np.zeros((B, H, D), dtype=np.float64)
                    x[:n] = cache_values(cache[layer, slots], shape.out_dtype)
                    data, sz = encode_tile(x, n, bits)
                    payload[pos:pos + data.size] = data
                    pos += data.size
                    base = req.scale_offset + ((layer * nb + b) * H) * 4 + which * 2
                    for head in range(H):
                        scales[base + head * 4] = sz[head, 0]
                        scales[base + head * 4 + 1] = sz[head, 1]
    return payload, scales
