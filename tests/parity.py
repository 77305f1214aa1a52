"""Element-by-element comparison of GPU cache rows with the CPU oracle.

Tolerance (reading of the 1-ulp bar with several correct results): every
restored element is the oracle's exactly rounded value, or the other
neighbour of a rounding midpoint that the exact value lies within the
double-rounding window of (the kernel rounds double -> float -> cache dtype;
:func:`oracle.classify_outputs`); for fp16 output, max |GPU - exact| <= 2e-3
over unit-scale elements (|exact| < 8; the N(0,1) channels); every other
element of both caches bit-identical to the pre-fill.
"""
from __future__ import annotations

import contextlib
import ctypes
import dataclasses
import sys

import numpy as np

import oracle

FP16_ABS_TOL = 2e-3
UNIT_SCALE = 8.0


def _ordered(bits: np.ndarray) -> np.ndarray:
    b = bits.astype(np.int32)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance in representable steps between fp16 or bf16 bit patterns (+0 == -0)."""
    return np.abs(_ordered(a) - _ordered(b))


def bits_to_f64(bits: np.ndarray, out_dtype: int) -> np.ndarray:
    bits = np.asarray(bits, dtype=np.uint16)
    if out_dtype == oracle.OUT_FP16:
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@dataclasses.dataclass
class Stats:
    n: int = 0
    n_bit_exact: int = 0
    n_near_tie: int = 0   # the other neighbour of a near-tie (accepted)
    n_wrong: int = 0      # neither: any of these fails the check
    max_ulp: int = 0
    max_abs_unit: float = 0.0
    n_nan: int = 0
    first_wrong: tuple = ()

    def add(self, got: np.ndarray, exact: np.ndarray, out_dtype: int, delta: int = 0) -> None:
        """``delta``: the request's shift when ``exact`` holds rotated keys
        (0 for values and unrotated keys)."""
        got = np.asarray(got, dtype=np.uint16)
        slack = oracle.rotation_slack(exact, delta) if delta else None
        same, near = oracle.classify_outputs(got, exact, out_dtype, slack)
        want = oracle.round_to_output(exact, out_dtype)
        d = ulp_distance(got, want)
        self.n += d.size
        self.n_bit_exact += int(same.sum())
        self.n_near_tie += int(near.sum())
        wrong = ~(same | near)
        if wrong.any() and not self.first_wrong:
            i = np.unravel_index(int(np.argmax(wrong)), wrong.shape)
            self.first_wrong = (tuple(int(x) for x in i), f"{int(got[i]):04x}", f"{int(want[i]):04x}",
                                float(np.asarray(exact)[i]))
        self.n_wrong += int(wrong.sum())
        self.max_ulp = max(self.max_ulp, int(d.max()) if d.size else 0)
        vals = bits_to_f64(got, out_dtype)
        self.n_nan += int(np.isnan(vals).sum())
        unit = np.abs(exact) < UNIT_SCALE
        if unit.any():
            self.max_abs_unit = max(self.max_abs_unit, float(np.abs(vals - exact)[unit].max()))

    @property
    def bit_exact_fraction(self) -> float:
        return self.n_bit_exact / max(1, self.n)

    @property
    def near_tie_fraction(self) -> float:
        return self.n_near_tie / max(1, self.n)

    def assert_ok(self, out_dtype: int) -> None:
        assert self.n > 0
        assert self.n_nan == 0, f"{self.n_nan} NaN outputs (a repair block or a poisoned scale was read)"
        assert self.n_wrong == 0, (f"{self.n_wrong} of {self.n} elements neither exactly rounded nor a near-tie "
                                   f"neighbour; first (index, got, want, exact): {self.first_wrong}")
        assert self.max_ulp <= 1, f"max ulp distance {self.max_ulp}"
        if out_dtype == oracle.OUT_FP16:
            assert self.max_abs_unit <= FP16_ABS_TOL, self.max_abs_unit


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


# ---------------------------------------------------------------------------
# Checkpoints for the restore tests
# ---------------------------------------------------------------------------

POISON_BYTE = 0xFF        # an FP16 tile of 0xFFFF is NaN
POISON_SCALE = 0x7E00     # binary16 NaN: a quantised tile decodes to NaN


def oracle_checkpoint(case, poison: bool = True):
    """(payload uint8, scales uint16) of a small case, written by the oracle's
    quantize-and-gather from the case's old caches; with ``poison`` every
    repair block's tiles and scales are overwritten with NaN encodings, so a
    restore that reads one shows it."""
    from oracle import quantize as oq

    k_old, v_old = case.host_old_caches()
    payload, scales = oq.quantize_gather(case.src_shape, case.requests, k_old, v_old,
                                         case.payload_nbytes, case.scale_elems)
    if poison:
        pr, sr = repair_ranges(case)
        for a, b in pr:
            payload[a:b] = POISON_BYTE
        for a, b in sr:
            scales[a:b] = POISON_SCALE
    return payload, scales


def repair_ranges(case):
    """Half-open (payload byte ranges, scale element ranges) of every repair
    block's K and V tiles and scales, all layers, adjacent ranges merged."""
    s = case.shape
    B, H, D = s.block_tokens, s.num_kv_heads, s.head_dim
    pr, sr = [], []
    for ri, req in enumerate(case.requests):
        layout = oracle.block_layout(req.tags, B, H, D)[0]
        for layer in range(s.num_layers):
            po = case.layer_payload_offset(ri, layer)
            so = case.layer_scale_offset(ri, layer)
            for b in range(len(req.tags)):
                if not req.repair[b]:
                    continue
                tag = int(req.tags[b])
                k0, v0 = layout[b]
                pr.append((po + k0, po + v0 + B * H * D * oracle.VALUE_BITS[tag] // 8))
                sr.append((so + b * H * 4, so + (b + 1) * H * 4))
    return _merge(pr), _merge(sr)


def _merge(ranges):
    out = []
    for a, b in sorted(ranges):
        if out and a <= out[-1][1]:
            out[-1] = (out[-1][0], max(out[-1][1], b))
        else:
            out.append((a, b))
    return out


def poison_device(case, payload, scales) -> None:
    """:func:`oracle_checkpoint`'s poisoning applied to device buffers."""
    pr, sr = repair_ranges(case)
    for a, b in pr:
        payload[a:b].fill_(POISON_BYTE)
    nan = POISON_SCALE - 65536 if POISON_SCALE >= 32768 else POISON_SCALE
    for a, b in sr:
        scales[a:b].fill_(nan)


def oracle_layer_checkpoint(case, ri: int, layer: int):
    """The oracle's checkpoint of one (request, layer) from the drawn rows:
    (payload bytes, scale bits [NB, H, 2, 2])."""
    from oracle import quantize as oq

    _, kb, vb = case.suffix_bits(ri, layer)
    return oq.quantize_rows(case.shape, case.requests[ri], kb, vb)


# Start orders of the restore kernel (pkv_internal_set_restore_order): by
# launch size, or forced to the early or the late order.
ORDERS = {"auto": 0, "early": 1, "late": 2}


@contextlib.contextmanager
def restore_order(order: str):
    """Force the restore kernel's start order for the launches inside."""
    from paper_2609_26219_amd import binding as pb

    fn = pb.load().pkv_internal_set_restore_order
    fn.argtypes = [ctypes.c_int32]
    fn.restype = ctypes.c_int32
    assert fn(ORDERS[order]) == 0
    try:
        yield
    finally:
        assert fn(0) == 0


def restore_small(case, poison: bool = True, order: str = "auto"):
    """Restore a small case on the GPU from the oracle's checkpoint.
    Returns (DeviceRestore after one run, (payload, scales) on the host)."""
    import torch

    from paper_2609_26219_amd.device import DeviceRestore

    ckpt = oracle_checkpoint(case, poison)
    dr = DeviceRestore(case, checkpoint=ckpt)
    with restore_order(order):
        dr.run()
        torch.cuda.synchronize()
    return dr, ckpt


def check_both_orders(case, poison: bool = True) -> None:
    """Full-cache parity of the restore in the early and the late start order."""
    for order in ("early", "late"):
        st = check_full(*restore_small(case, poison, order))
        log(f"  {order} order: {st}")


# ---------------------------------------------------------------------------
# Comparisons
# ---------------------------------------------------------------------------

def check_full(dr, ckpt) -> Stats:
    """Whole-cache comparison against a full oracle restore from the same
    checkpoint (small cases)."""
    case = dr.case
    s = case.shape
    payload, scales = ckpt
    pre_k, pre_v = case.host_prefill(0), case.host_prefill(1)
    k_got, v_got = dr.host_caches()
    written = oracle.written_slots(s, case.requests)
    kg = k_got.reshape(s.num_layers, s.pool_slots, s.row_elems)
    vg = v_got.reshape(kg.shape)
    # untouched: bit-identical to the pre-fill
    assert np.array_equal(kg[:, ~written], pre_k.reshape(kg.shape)[:, ~written]), "stray K write"
    assert np.array_equal(vg[:, ~written], pre_v.reshape(vg.shape)[:, ~written]), "stray V write"
    st = Stats()
    for req in case.requests:
        layout = oracle.block_layout(req.tags, s.block_tokens, s.num_kv_heads, s.head_dim)
        for layer in range(s.num_layers):
            for b in oracle.reused_blocks(req):
                slots, k, v = oracle.restore_block(payload, scales, s, req, layer, b, layout)
                st.add(kg[layer, slots].reshape(k.shape), k, s.out_dtype, int(req.delta))
                st.add(vg[layer, slots].reshape(v.shape), v, s.out_dtype)
    st.assert_ok(s.out_dtype)
    return st


def check_device_checkpoint(case, payload, scales, refs) -> None:
    """Bit-exact comparison of device-written checkpoint slices with the
    oracle's, for the (request, layer) keys of ``refs``."""
    for (ri, layer), (pb, sb) in refs.items():
        po = case.layer_payload_offset(ri, layer)
        so = case.layer_scale_offset(ri, layer)
        got_p = payload[po:po + pb.size].cpu().numpy()
        got_s = scales[so:so + sb.size].cpu().numpy().view(np.uint16)
        bad_p = int((got_p != pb).sum())
        bad_s = int((got_s != sb.reshape(-1)).sum())
        log(f"  checkpoint request {ri} layer {layer}: {pb.size} bytes, {sb.size} scales, "
            f"{bad_p} + {bad_s} mismatches")
        assert bad_p == 0 and bad_s == 0


def check_sampled(dr, refs, check_untouched: bool = True) -> Stats:
    """Compare every reused block of the sampled (request, layer) pairs with
    the oracle's restore of the oracle's checkpoint ``refs[(request, layer)]``;
    check all untouched elements of every layer on the device."""
    case = dr.case
    s = case.shape
    st = Stats()
    shape1 = dataclasses.replace(s, num_layers=1)
    for (ri, layer), (pb, sb) in refs.items():
        req = case.requests[ri]
        one = dataclasses.replace(req, payload_offset=0, scale_offset=0)
        blocks = oracle.reused_blocks(req)
        all_slots = np.concatenate([oracle.destination_slots(s, req, b) for b in blocks]) if blocks else np.zeros(0, int)
        kg = dr.rows(0, layer, all_slots)
        vg = dr.rows(1, layer, all_slots)
        pos = 0
        layout = oracle.block_layout(req.tags, s.block_tokens, s.num_kv_heads, s.head_dim)
        for b in blocks:
            slots, k, v = oracle.restore_block(pb, sb.reshape(-1), shape1, one, 0, b, layout)
            n = len(slots)
            st.add(kg[pos:pos + n], k, s.out_dtype, int(req.delta))
            st.add(vg[pos:pos + n], v, s.out_dtype)
            pos += n
        log(f"  sampled request {ri} layer {layer}: {len(blocks)} blocks, max ulp {st.max_ulp}, "
            f"bit-exact {st.bit_exact_fraction:.7f}, near-ties {st.n_near_tie}, wrong {st.n_wrong}")
    st.assert_ok(s.out_dtype)
    if check_untouched:
        written = oracle.written_slots(s, case.requests)
        bad = dr.untouched_mismatches(written)
        log(f"  untouched check over {s.num_layers} layers: {bad} mismatches")
        assert bad == 0
    return st


def host_gap_bytes() -> int:
    import ctypes

    from paper_2609_26219_amd import binding as pb

    fn = pb.load().pkv_internal_host_gap_bytes
    fn.restype = ctypes.c_uint64
    return int(fn())


def streamed_payload_ranges(case, gap: int):
    """Per layer, the (offset, length) payload copies a streamed restore
    issues: every reused block's K and V tiles, requests in order, blocks in
    layout order (runs by tag, ascending), a copy extended over a following
    one of the same request that starts at most `gap` bytes after it ends."""
    s = case.shape
    B, H, D, L = s.block_tokens, s.num_kv_heads, s.head_dim, s.num_layers
    out = []
    for layer in range(L):
        ranges = []
        for ri, req in enumerate(case.requests):
            offsets, _ = oracle.block_layout(req.tags, B, H, D)
            base = case.layer_payload_offset(ri, layer)
            first = len(ranges)
            for tag in range(4):
                for b in range(len(req.tags)):
                    if int(req.tags[b]) != tag or req.repair[b]:
                        continue
                    k0, v0 = offsets[b]
                    off, end = base + k0, base + v0 + B * H * D * oracle.VALUE_BITS[tag] // 8
                    if len(ranges) > first and ranges[-1][1] <= off and off - ranges[-1][1] <= gap:
                        ranges[-1][1] = end
                    else:
                        ranges.append([off, end])
        out.append([(a, e - a) for a, e in ranges])
    return out


def reused_byte_masks(case, gap: int = 0):
    """Boolean masks over the payload bytes and the scale elements that a
    streamed restore copies: every reused block's K and V tiles in every
    layer (plus repair blocks inside gaps of at most `gap` bytes), and the
    whole per-layer scale block of each request that has a reused quantized
    block in that layer."""
    s = case.shape
    H, L = s.num_kv_heads, s.num_layers
    pmask = np.zeros(case.payload_nbytes, bool)
    smask = np.zeros(case.scale_elems, bool)
    for layer_ranges in streamed_payload_ranges(case, gap):
        for off, ln in layer_ranges:
            pmask[off: off + ln] = True
    for ri, req in enumerate(case.requests):
        nb = len(req.tags)
        for layer in range(L):
            if any(not req.repair[b] and int(req.tags[b]) != 0 for b in range(nb)):
                so = case.layer_scale_offset(ri, layer)
                smask[so: so + nb * H * 4] = True
    return pmask, smask


# ---------------------------------------------------------------------------
# Checkpoint write
# ---------------------------------------------------------------------------

FILL = 0xAB  # checkpoint-write tests: payload bytes outside every checkpoint range keep this


def gpu_checkpoint(case, torch, caches=None):
    """Write a case's checkpoint on the GPU from its old caches (host arrays
    unless given); payload and scales start filled with marker values."""
    from paper_2609_26219_amd import binding as pb

    from paper_2609_26219_amd.device import alloc_caches

    s = case.src_shape
    kc, vc = case.host_old_caches() if caches is None else caches
    dk, dv = alloc_caches(s, "cuda")  # in the shape's layout
    dk.copy_(torch.from_numpy(kc.view(np.int16)))
    dv.copy_(torch.from_numpy(vc.view(np.int16)))
    payload = torch.full((case.payload_nbytes,), FILL, dtype=torch.uint8, device="cuda")
    scales = torch.full((case.scale_elems,), 0x5A5A, dtype=torch.int16, device="cuda")
    plan = pb.pkv_checkpoint_plan(s, case.requests)
    info = pb.pkv_plan_query(plan)
    assert info["kind"] == 1
    pb.quantize_gather_tensors(plan, dk, dv, payload, scales)
    torch.cuda.synchronize()
    return kc, vc, payload.cpu().numpy(), scales.cpu().numpy().view(np.uint16), info


def check_checkpoint_write(case, torch, caches=None):
    """The GPU checkpoint write against the oracle quantizer, bit for bit;
    bytes outside every request's ranges keep their marker values."""
    from oracle import quantize as oq
    from paper_2609_26219_amd import workloads as wl

    kc, vc, payload, scales, info = gpu_checkpoint(case, torch, caches)
    ref_p, ref_s = oq.quantize_gather(case.src_shape, case.requests, kc, vc, case.payload_nbytes, case.scale_elems)
    inside_p = np.zeros(case.payload_nbytes, bool)
    inside_s = np.zeros(case.scale_elems, bool)
    for r in case.requests:
        pbytes, selems = wl.encoded_request_nbytes(case.shape, r)
        inside_p[r.payload_offset: r.payload_offset + pbytes] = True
        inside_s[r.scale_offset: r.scale_offset + selems] = True
    bad = np.nonzero(payload[inside_p] != ref_p[inside_p])[0]
    assert bad.size == 0, f"{bad.size} payload bytes differ, first at {bad[:5]}"
    assert np.array_equal(scales[inside_s], ref_s[inside_s])
    assert (payload[~inside_p] == FILL).all() and (scales[~inside_s] == 0x5A5A).all()
    assert info["bytes_written"] == int(inside_p.sum()) + 2 * int(inside_s.sum())
    return payload, scales, ref_p, ref_s
