"""Pins of the quantize-and-gather oracle (the offload side of the checkpoint).

Against: a hand-worked fixture; the half-step bound checked through the
restore oracle's decode; the defining extremal properties of the fp16
zero/scale roundings; code-range and tie behaviour; and agreement of the
whole write -> read cycle with the original values."""
import json
import os
import types

import numpy as np
import pytest

import oracle
from oracle import quantize as oq

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _ns(**kw):
    return types.SimpleNamespace(**kw)


@pytest.mark.parametrize("fixture", ["hand_quantize_d4.json", "hand_quantize_d4_bf16.json"])
def test_hand_worked_checkpoint_write(fixture):
    """The binary16 fixture and its bfloat16 twin: same K8V4 values, an FP16
    block whose bfloat16 values need rounding to binary16 (ties included)."""
    d = json.load(open(os.path.join(GOLDEN, fixture)))
    s = d["shape"]
    shape = _ns(num_layers=1, num_kv_heads=1, head_dim=4, block_tokens=2, page_size=2, pool_pages=3,
                out_dtype=s["cache_dtype"])
    r = d["request"]
    req = _ns(suffix_tokens=r["suffix_tokens"], src_row0=r["src_row0"], tags=np.array(r["tags"], np.uint8),
              src_page_table=np.array(r["page_table"], np.int32), payload_offset=0, scale_offset=0)
    caches = []
    fill = int(d.get("fill_hex", "7e00"), 16)  # NaN of the cache dtype
    old = d.get("old_cache_hex") or d["old_cache_f16_hex"]
    for kv in ("k", "v"):
        c = np.full((1, 3, 2, 1, 4), fill, dtype=np.uint16).reshape(1, 6, 1, 4)
        for slot, words in old[kv].items():
            c[0, int(slot), 0] = [int(w, 16) for w in words]
        caches.append(c.reshape(1, 3, 2, 1, 4))
    payload, scales = oq.quantize_gather(shape, [req], caches[0], caches[1], 44, 8)
    want = bytearray()
    for seg in d["expected_payload"]:
        if "u16" in seg:
            for w in seg["u16"]:
                want += int(w, 16).to_bytes(2, "little")
        else:
            want += bytes(int(b, 16) for b in seg["u8"])
    assert payload.tobytes() == bytes(want)
    assert [f"{x:04x}" for x in scales] == d["expected_scales_f16_hex"]


def test_cache_values_from_literal_bits():
    """Cache bit patterns decode by their own format's definition (hand-derived
    values): bfloat16 = sign, 8 exponent bits (bias 127), 7 fraction bits;
    binary16 = sign, 5 exponent bits (bias 15), 10 fraction bits."""
    bf = np.array([0x3F80, 0xC000, 0x8000, 0x0001, 0x7F7F, 0x3581, 0x4049, 0x0080], np.uint16)
    got = oq.cache_values(bf, oq.OUT_BF16)
    want = [1.0, -2.0, -0.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, (1 + 2 ** -7) * 2.0 ** -20, 3.140625,
            2.0 ** -126]
    assert got.tolist() == want
    assert np.signbit(got[2])
    hf = np.array([0x3C00, 0xC000, 0x8000, 0x0001, 0x7BFF, 0x3555, 0x0400], np.uint16)
    got = oq.cache_values(hf, oq.OUT_FP16)
    assert got.tolist() == [1.0, -2.0, -0.0, 2.0 ** -24, 65504.0, (1 + 0x155 / 1024) * 2.0 ** -2, 2.0 ** -14]
    assert np.signbit(got[2])


def test_fp16_floor_ceil_are_extremal():
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000) * 4, rng.standard_normal(2000) * 1e-6, [0.0, -0.0, 1.0, -2.5]])
    lo = oq.f16_floor(x)
    hi = oq.f16_ceil(x)
    lo_v = lo.view(np.float16).astype(np.float64)
    hi_v = hi.view(np.float16).astype(np.float64)
    assert (lo_v <= x).all() and (hi_v >= x).all()
    # nothing representable in between: the neighbour beyond each bound crosses x
    assert (oq._f16_next_up(lo).view(np.float16).astype(np.float64) > x).all()
    assert (oq._f16_next_down(hi).view(np.float16).astype(np.float64) < x).all()
    exact = x.astype(np.float16).astype(np.float64) == x
    assert (lo_v[exact] == x[exact]).all() and (hi_v[exact] == x[exact]).all()


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("cache_dtype", [oq.OUT_FP16, oq.OUT_BF16])
def test_round_trip_within_half_step(bits, cache_dtype):
    rng = np.random.default_rng(bits + 10 * cache_dtype)
    qmax = (1 << bits) - 1
    for trial in range(200):
        n = int(rng.integers(1, 40))
        raw = rng.standard_normal((n, 16)) * rng.choice([1e-6, 1e-3, 1.0, 8.0, 100.0])
        if trial % 17 == 0:
            raw[:] = raw[0, 0]  # constant tile
        # values as the cache holds them
        if cache_dtype == oq.OUT_FP16:
            x = raw.astype(np.float16).astype(np.float64)
        else:
            x = oracle.round_bf16_bits(raw)
            x = oq.cache_values(x, oq.OUT_BF16)
        codes, s_bits, z_bits = oq.quantize_tile(x, bits)
        s = float(np.array(s_bits, np.uint16).view(np.float16))
        z = float(np.array(z_bits, np.uint16).view(np.float16))
        assert codes.max() <= qmax
        assert z <= x.min()
        assert s * qmax >= x.max() - z
        dec = oracle.dequantize(codes.astype(np.float64)[:, None, :], np.array([s]), np.array([z]))[:, 0, :]
        assert (np.abs(dec - x) <= s / 2 * (1 + 1e-12)).all()


def test_rint_ties_go_to_even():
    x = np.array([[0.0, 0.25, 0.75, 1.25, 7.5]])  # scale 0.5: 0.5 -> 0, 1.5 -> 2, 2.5 -> 2
    codes, s, z = oq.quantize_tile(x, 4)
    assert codes.tolist() == [[0, 0, 2, 2, 15]]


def test_write_then_read_cycle_recovers_values():
    """Checkpoint written by the quantize oracle and read back by the restore
    oracle (with Delta = 0, same page layout) reproduces every value to half a step."""
    rng = np.random.default_rng(9)
    B, H, D, P, L = 8, 2, 16, 4, 2
    N = 21
    nb = -(-N // B)
    tags = np.array([0, 1, 2, 3][:nb] + [2] * max(0, nb - 4), np.uint8)
    pool = 16
    pt = rng.permutation(pool)[:8].astype(np.int32)
    shape = _ns(num_layers=L, num_kv_heads=H, head_dim=D, block_tokens=B, page_size=P, pool_pages=pool,
                out_dtype=oq.OUT_FP16, rope_theta=1e4)
    k = rng.standard_normal((L, pool, P, H, D)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((L, pool, P, H, D)).astype(np.float16).view(np.uint16)
    src = _ns(suffix_tokens=N, src_row0=3, tags=tags, src_page_table=pt, payload_offset=0, scale_offset=0)
    layer_bytes = sum(B * H * D * (oq.KEY_BITS[int(t)] + oq.VALUE_BITS[int(t)]) // 8 for t in tags)
    payload, scales = oq.quantize_gather(shape, [src], k, v, L * layer_bytes, L * nb * H * 4)
    dst = _ns(suffix_tokens=N, delta=0, dst_row0=3, tags=tags, repair=np.zeros(nb, np.uint8), page_table=pt,
              payload_offset=0, scale_offset=0)
    for layer in range(L):
        for b in range(nb):
            slots, kk, vv = oracle.restore_block(payload, scales, shape, dst, layer, b)
            tag = int(tags[b])
            for got, cache, bits in ((kk, k, oq.KEY_BITS[tag]), (vv, v, oq.VALUE_BITS[tag])):
                want = cache.reshape(L, -1, H, D)[layer, slots].view(np.float16).astype(np.float64)
                if bits == 16:
                    assert np.array_equal(got, want)
                else:
                    sz = oracle.block_scales(scales, dst, shape, layer, b)
                    step = sz[:, 0 if cache is k else 1, 0][None, :, None]
                    assert (np.abs(got - want) <= step / 2 * (1 + 1e-12)).all()


@pytest.mark.parametrize("seed", [0, 1])
def test_layer_form_equals_tile_by_tile(seed):
    """The vectorised per-layer form gives the same bytes as the per-tile form."""
    from paper_2609_26219_amd import workloads as wl
    for dtype in (wl.OUT_FP16, wl.OUT_BF16):
        case = wl.make_custom(seed, L=2, H=3, D=32, B=8, P=4, n_tokens=(37, 5, 16), deltas=(3, 0, -2),
                              rho0s=(9, 4, 30), tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), out_dtype=dtype,
                              outlier_pairs=1)
        k, v = case.host_old_caches()
        a = oq.quantize_gather(case.src_shape, case.requests, k, v, case.payload_nbytes, case.scale_elems)
        b = oq.quantize_gather_per_tile(case.src_shape, case.requests, k, v, case.payload_nbytes, case.scale_elems)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
