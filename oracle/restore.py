"""CPU oracle for PatchKV's suffix restore.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path (the ``libpkv`` HIP library and its
binding) never does.  It is a plain, slow, fp64 statement of what the fused
restore computes (PatchKV, Section IV-D "Quality-Constrained Quantized
Transport" and the resume path in Section IV-A, steps 5-6):

for every request, every layer, every block ``b`` of the aligned suffix ``S``
that is in the reuse set ``F = B(S) minus R`` (Eq. 12; blocks of ``R`` are
recomputed elsewhere and never touched here), and every KV head:

1. read the block's K and V tiles from the checkpoint payload, whose blocks
   are clustered into same-tag runs (Section IV-D);
2. decode each tile by the block's frozen precision tag (Eq. 14 tiers FP16,
   K8/V8, K8/V4, plus the uniform 4-bit K4/V4 of the transport ablation in
   Section V-C): FP16 is taken as is, a quantized channel is
   ``code * scale + zero`` with the block-head's fp16 scale and zero;
3. correct the key phase by the edit shift (Eq. 3):
   ``K_corr = R(rho_i) R(omega_i)^-1 K_old = R(Delta) K_old`` with
   ``Delta = rho_i - omega_i``, the same for every suffix token after a middle
   edit (Eq. 1).  Values are never rotated (Section IV-C);
4. round once, from the exact fp64 value, to the cache dtype (fp16 or bf16,
   round to nearest even);
5. write token ``t`` of block ``b`` to logical row ``rho_0 + b*B + t`` of the
   request, i.e. slot ``row mod P`` of physical page ``page_table[row div P]``
   (the old-to-new token map of Section IV-D); nothing else is written.

Readings where the paper is silent (each is listed with its reason in the
design notes): the model's own RoPE (the paper calls the correction
model-aware): rotate-half pairs ``(i, i + R/2)`` or interleaved pairs
``(2i, 2i + 1)`` over the first ``R`` channels, frequencies
``theta^(-2i/R)`` unless the model gives its own table, and channels past
``R`` untouched; rotation skipped when ``Delta == 0``; tiles are token-major
``[B][H][D]``; 4-bit codes put channel ``2j`` in the low nibble.

Objects passed in only need the attributes used below (``Shape`` /
``Request``-like); this module imports nothing from the product package.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

FP16, K8V8, K8V4, K4V4 = 0, 1, 2, 3
# Bits per channel of the key and value representation of each tag (Eq. 14;
# keys never go below 8 bits in PatchKV's own tiers, K4V4 is the ablation's
# uniform INT4).
KEY_BITS = {FP16: 16, K8V8: 8, K8V4: 8, K4V4: 4}
VALUE_BITS = {FP16: 16, K8V8: 8, K8V4: 4, K4V4: 4}
OUT_FP16, OUT_BF16 = 0, 1


# --------------------------------------------------------------------------
# Step 1: locate a block's tiles in the clustered checkpoint (Section IV-D)
# --------------------------------------------------------------------------

def block_layout(tags: Sequence[int], B: int, H: int, D: int) -> Tuple[Dict[int, Tuple[int, int]], int]:
    """Byte offsets, inside one layer, of every block's (K tile, V tile),
    and the layer's size.  Same-tag blocks form one contiguous run; runs go
    FP16, K8V8, K8V4, K4V4; blocks ascend inside a run."""
    offsets: Dict[int, Tuple[int, int]] = {}
    pos = 0
    for tag in (FP16, K8V8, K8V4, K4V4):
        for b in range(len(tags)):
            if int(tags[b]) == tag:
                k_bytes = B * H * D * KEY_BITS[tag] // 8
                v_bytes = B * H * D * VALUE_BITS[tag] // 8
                offsets[b] = (pos, pos + k_bytes)
                pos += k_bytes + v_bytes
    return offsets, pos


def request_payload_bytes(shape, req) -> int:
    return shape.num_layers * block_layout(req.tags, shape.block_tokens, shape.num_kv_heads, shape.head_dim)[1]


# --------------------------------------------------------------------------
# Step 2: decode by tag
# --------------------------------------------------------------------------

def read_tile(payload: np.ndarray, offset: int, bits: int, B: int, H: int, D: int) -> np.ndarray:
    """A tile's channels as fp64 ``[B, H, D]``: fp16 values, or integer codes."""
    n = B * H * D
    raw = payload[offset: offset + n * bits // 8]
    if bits == 16:
        vals = raw.view("<f2").astype(np.float64)
    elif bits == 8:
        vals = raw.astype(np.float64)
    elif bits == 4:
        vals = np.empty(n, dtype=np.float64)
        vals[0::2] = raw & 0x0F  # channel 2j: low nibble of byte j
        vals[1::2] = raw >> 4
    else:
        raise ValueError(bits)
    return vals.reshape(B, H, D)


def dequantize(codes: np.ndarray, scale: np.ndarray, zero: np.ndarray) -> np.ndarray:
    """``code * scale + zero`` per head (``scale``/``zero`` are ``[H]``), in fp64."""
    return codes * scale[None, :, None] + zero[None, :, None]


def block_scales(scales: np.ndarray, req, shape, layer: int, block: int) -> np.ndarray:
    """fp64 ``[H, 2 (K, V), 2 (scale, zero)]`` of one (layer, block)."""
    H = shape.num_kv_heads
    nb = len(req.tags)
    start = req.scale_offset + ((layer * nb + block) * H) * 4
    bits = np.asarray(scales[start: start + H * 4], dtype=np.uint16)
    return bits.view(np.float16).astype(np.float64).reshape(H, 2, 2)


def decode_block(payload: np.ndarray, scales: np.ndarray, shape, req, layer: int, block: int,
                 layout: Optional[Tuple[Dict[int, Tuple[int, int]], int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Decoded (K_old, V) of one block, fp64 ``[B, H, D]`` (padding rows included).
    ``layout`` is the request's ``block_layout`` if already computed."""
    B, H, D = shape.block_tokens, shape.num_kv_heads, shape.head_dim
    offsets, layer_bytes = layout if layout is not None else block_layout(req.tags, B, H, D)
    base = req.payload_offset + layer * layer_bytes
    k_off, v_off = offsets[block]
    tag = int(req.tags[block])
    k = read_tile(payload, base + k_off, KEY_BITS[tag], B, H, D)
    v = read_tile(payload, base + v_off, VALUE_BITS[tag], B, H, D)
    if tag != FP16:
        sz = block_scales(scales, req, shape, layer, block)
        k = dequantize(k, sz[:, 0, 0], sz[:, 0, 1])
        v = dequantize(v, sz[:, 1, 0], sz[:, 1, 1])
    return k, v


# --------------------------------------------------------------------------
# Step 3: RoPE phase correction of keys (Eq. 2, Eq. 3)
# --------------------------------------------------------------------------

ROPE_HALF, ROPE_INTERLEAVED = 0, 1


def rope_frequencies(theta: float, rotary_dim: int, inv_freq=None) -> np.ndarray:
    """Frequency of rotary pair ``i < rotary_dim/2``: the given table, else
    ``theta^(-2i/rotary_dim)``."""
    if inv_freq is not None:
        f = np.asarray(inv_freq, dtype=np.float64)
        assert f.shape == (rotary_dim // 2,)
        return f
    i = np.arange(rotary_dim // 2, dtype=np.float64)
    return theta ** (-2.0 * i / rotary_dim)


def rope_angles(position: float, theta: float, D: int, inv_freq=None) -> np.ndarray:
    """Angle of rotary pair ``i`` at a position: ``position * f_i``."""
    return position * rope_frequencies(theta, D, inv_freq)


def rope_pairs(D: int, rotary_dim: int, style: int) -> Tuple[np.ndarray, np.ndarray]:
    """Channel indices (first, second) of every rotary pair ``i``:
    rotate-half ``(i, i + R/2)`` or interleaved ``(2i, 2i + 1)``, R = rotary_dim."""
    i = np.arange(rotary_dim // 2)
    if style == ROPE_HALF:
        return i, i + rotary_dim // 2
    if style == ROPE_INTERLEAVED:
        return 2 * i, 2 * i + 1
    raise ValueError(style)


def rotate(x: np.ndarray, angles: np.ndarray, style: int = ROPE_HALF, rotary_dim: Optional[int] = None) -> np.ndarray:
    """Apply ``R`` to the last axis: pair ``i`` (by ``style``) turns by
    ``angles[i]`` counter-clockwise; channels from ``rotary_dim`` on are
    returned unchanged."""
    D = x.shape[-1]
    R = D if rotary_dim is None else rotary_dim
    a, b = rope_pairs(D, R, style)
    c, s = np.cos(angles), np.sin(angles)
    out = np.array(x, dtype=np.float64, copy=True)
    xa, xb = x[..., a], x[..., b]
    out[..., a] = xa * c - xb * s
    out[..., b] = xb * c + xa * s
    return out


def correct_key_phase(k_old: np.ndarray, delta: int, theta: float, style: int = ROPE_HALF,
                      rotary_dim: Optional[int] = None, inv_freq=None) -> np.ndarray:
    """``R(rho) R(omega)^-1 K_old = R(rho - omega) K_old = R(Delta) K_old``
    with the model's pairing, rotated channels and frequencies.  ``R(0)`` is
    the identity, so no arithmetic is applied when ``Delta == 0``."""
    if delta == 0:
        return k_old.copy()
    D = k_old.shape[-1]
    R = D if not rotary_dim else rotary_dim
    return rotate(k_old, delta * rope_frequencies(theta, R, inv_freq), style, R)


def shape_rope(shape) -> Tuple[int, Optional[int], object]:
    """(style, rotary_dim or None, inv_freq or None) of a shape; absent
    attributes mean full rotate-half RoPE with theta frequencies."""
    return (int(getattr(shape, "rope_style", ROPE_HALF)), int(getattr(shape, "rotary_dim", 0)) or None,
            getattr(shape, "inv_freq", None))


# --------------------------------------------------------------------------
# Step 4: one rounding to the cache dtype
# --------------------------------------------------------------------------

def round_fp16_bits(x: np.ndarray) -> np.ndarray:
    """binary16 bit patterns of fp64 values, round to nearest even (numpy's
    direct double -> half conversion)."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns of fp64 values, rounded once to nearest even.

    bf16 keeps 8 significant bits; subnormals (below 2^-126) are multiples of
    2^-133.  ``m * 2^e`` with ``m`` in [0.5, 1) is scaled so the kept bits are
    the integer part, rounded by ``rint`` (ties to even), and scaled back; the
    result is exactly representable in float32, whose top 16 bits are the bf16
    pattern."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.float64)
    finite = np.isfinite(x)
    xf = np.where(finite, x, 0.0)
    _, e = np.frexp(xf)
    e = np.maximum(e, -125)
    r = np.ldexp(np.rint(np.ldexp(xf, 8 - e)), e - 8)
    out[finite] = r[finite]
    out[~finite] = x[~finite]
    with np.errstate(over="ignore"):
        f32 = out.astype(np.float32)
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    bits[nan] = 0x7FC0
    return bits


def round_to_output(x: np.ndarray, out_dtype: int) -> np.ndarray:
    return round_fp16_bits(x) if out_dtype == OUT_FP16 else round_bf16_bits(x)


def output_values(bits: np.ndarray, out_dtype: int) -> np.ndarray:
    """fp64 values of fp16 / bf16 output bit patterns."""
    bits = np.asarray(bits, dtype=np.uint16)
    if out_dtype == OUT_FP16:
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Which outputs are correct (reading: several correct results near ties)
# --------------------------------------------------------------------------
#
# The exact result is the one rounding of the fp64 value above.  An
# implementation that first rounds to single precision and then to the cache
# dtype can land on the other side of a rounding midpoint m of the cache
# dtype, but only when the value lies within that first rounding (at most
# 2^-24 |x|) of m.  Both neighbours of such a near-tie are accepted, and
# nothing else: away from a midpoint only the exactly rounded value is.

TIE_WINDOW_REL = 2.0 ** -23  # twice half a single-precision ulp, relative to |x|


def rotation_slack(exact_k: np.ndarray, delta: int) -> Optional[np.ndarray]:
    """Absolute slack for rotated keys ``[..., D]`` (``None`` when Delta is 0:
    no rotation, so the result is a plain rounding).  A rotation computed from
    a differently rounded angle Delta*f_i (f_i <= 1) and cos/sin differs from
    this module's by at most about 2^-51 (1 + |Delta|) (|x| + |y|) for the pair
    (x, y); a rotation keeps each pair's norm, so |x| + |y| <= 2 max|x'| over
    the head's outputs.  The slack is 4x that bound."""
    if delta == 0:
        return None
    row_max = np.abs(np.asarray(exact_k, dtype=np.float64)).max(axis=-1, keepdims=True)
    return 2.0 ** -47 * (1.0 + abs(float(delta))) * row_max


def classify_outputs(got_bits: np.ndarray, exact: np.ndarray, out_dtype: int,
                     slack: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """(exactly rounded, accepted near-tie) masks of output bit patterns
    against exact fp64 values.  An element that is neither is wrong.

    Near-tie: the bits are the other neighbour of the midpoint m between
    them and the exactly rounded value (the two are adjacent), and
    ``|x - m| <= 2^-23 |x| + slack``.  ``slack`` (absolute, broadcastable)
    is given for rotated keys only (:func:`rotation_slack`); for them a zero
    of either sign is also accepted where the exact result rounds to zero
    (x*c - y*s can give -0 or +0).  Elsewhere signed zeros must match."""
    got = np.asarray(got_bits, dtype=np.uint16)
    x = np.asarray(exact, dtype=np.float64)
    want = round_to_output(x, out_dtype)
    same = got == want
    gv = output_values(got, out_dtype)
    wv = output_values(want, out_dtype)
    mid = (gv + wv) / 2.0  # exact in fp64: both are short binary fractions
    # adjacent: no representable value strictly between them, i.e. their
    # sign-magnitude orders differ by one
    def order(b):
        b = b.astype(np.int32)
        return np.where(b & 0x8000, -(b & 0x7FFF), b)
    adjacent = np.abs(order(got) - order(want)) == 1
    window = TIE_WINDOW_REL * np.abs(x) + (0.0 if slack is None else slack)
    with np.errstate(invalid="ignore"):
        near = ~same & adjacent & np.isfinite(gv) & (np.abs(x - mid) <= window)
    if slack is not None:
        near |= ~same & (gv == 0.0) & (wv == 0.0)
    return same, near


# --------------------------------------------------------------------------
# Step 5: placement (old-to-new token map + page table)
# --------------------------------------------------------------------------

def valid_tokens(req, B: int, block: int) -> int:
    return min(B, req.suffix_tokens - block * B)


def destination_slots(shape, req, block: int) -> np.ndarray:
    """Physical slot of every valid token of a block."""
    B, P = shape.block_tokens, shape.page_size
    n = valid_tokens(req, B, block)
    slots = np.empty(n, dtype=np.int64)
    for t in range(n):
        row = req.dst_row0 + block * B + t
        lp = row // P
        if lp >= len(req.page_table):
            raise ValueError("row beyond the page table")
        page = int(req.page_table[lp])
        if page < 0 or page >= shape.pool_pages:
            raise ValueError("row on an unmapped or out-of-range page")
        slots[t] = page * P + row % P
    return slots


def reused_blocks(req) -> List[int]:
    """Blocks of F (not in the repair set R), ascending."""
    return [b for b in range(len(req.tags)) if int(req.repair[b]) == 0]


def restore_block(payload, scales, shape, req, layer: int, block: int, layout=None
                  ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(slots [n], K exact fp64 [n, H, D], V exact fp64 [n, H, D]) of one reused block."""
    n = valid_tokens(req, shape.block_tokens, block)
    k_old, v = decode_block(payload, scales, shape, req, layer, block, layout)
    style, rdim, inv = shape_rope(shape)
    k = correct_key_phase(k_old[:n], int(req.delta), float(shape.rope_theta), style, rdim, inv)
    return destination_slots(shape, req, block), k, v[:n]


def restore(shape, requests: Sequence, payload: np.ndarray, scales: np.ndarray,
            k_cache: np.ndarray, v_cache: np.ndarray, layers: Optional[Iterable[int]] = None
            ) -> Tuple[np.ndarray, np.ndarray]:
    """Full restore on copies of the two caches (uint16 bit patterns,
    ``[L, pool_pages, P, H, D]``).  Returns the new caches."""
    L, H, D = shape.num_layers, shape.num_kv_heads, shape.head_dim
    k_out = np.array(k_cache, dtype=np.uint16, copy=True)
    v_out = np.array(v_cache, dtype=np.uint16, copy=True)
    kf = k_out.reshape(L, -1, H, D)
    vf = v_out.reshape(L, -1, H, D)
    layer_list = range(L) if layers is None else list(layers)
    check_pages(shape, requests)
    for req in requests:
        layout = block_layout(req.tags, shape.block_tokens, H, D)
        for layer in layer_list:
            for b in reused_blocks(req):
                slots, k, v = restore_block(payload, scales, shape, req, layer, b, layout)
                kf[layer, slots] = round_to_output(k, shape.out_dtype)
                vf[layer, slots] = round_to_output(v, shape.out_dtype)
    return k_out, v_out


def written_slots(shape, requests: Sequence) -> np.ndarray:
    """Boolean ``[pool_pages * P]``: slots a restore writes (in every layer)."""
    mask = np.zeros(shape.pool_pages * shape.page_size, dtype=bool)
    for req in requests:
        for b in reused_blocks(req):
            mask[destination_slots(shape, req, b)] = True
    return mask


def check_pages(shape, requests: Sequence) -> None:
    """Every page a restore writes must belong to exactly one (request,
    logical page); otherwise two rows would land in one slot."""
    owner: Dict[int, Tuple[int, int]] = {}
    P = shape.page_size
    for ri, req in enumerate(requests):
        for b in reused_blocks(req):
            first = req.dst_row0 + b * shape.block_tokens
            last = first + valid_tokens(req, shape.block_tokens, b) - 1
            for lp in range(first // P, last // P + 1):
                destination_slots(shape, req, b)  # raises on unmapped / out of range pages
                page = int(req.page_table[lp])
                if owner.setdefault(page, (ri, lp)) != (ri, lp):
                    raise ValueError("two logical pages share a physical page")
