"""CPU emulation of the checkpoint (quantize-and-gather) kernel's addressing.

Replays, for every thread of every workgroup of the host-built work list, the
address formulas of ``gather.hip`` and checks: every cache read is a suffix
row of a request (in bounds); every byte of each request's checkpoint range
and every scale element is written exactly once; nothing else is written.
Keep the constants in step with the kernel."""
import ctypes

import numpy as np
import pytest

from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

MAX_WAVES = 16  # waves per workgroup at most
KBITS = (16, 8, 8, 4)
VBITS = (16, 8, 4, 4)
UNIT_DTYPE = np.dtype([("k_off", "<u8"), ("v_off", "<u8"), ("scale_off", "<u8"), ("row0", "<i8"), ("pt_off", "<i8"),
                       ("table_off", "<i4"), ("layer", "<i4"), ("tag", "<i4"), ("n_valid", "<i4"),
                       ("page1", "<i4"), ("page2", "<i4")])


def loads_per_chunk(nload):
    return 2 if nload <= 2 else 4 if nload <= 4 else 8 if nload <= 8 else 16


def checkpoint_units(shape, requests):
    lib = pb.load()
    fn = lib.pkv_internal_checkpoint_units
    fn.argtypes = [ctypes.POINTER(pb.PkvModel), ctypes.POINTER(pb.PkvCheckpointRequest), ctypes.c_int32,
                   ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32)]
    fn.restype = ctypes.c_int32
    m = pb.make_model(shape)
    reqs = pb._CheckpointRequests(requests)
    count, wg = ctypes.c_int64(), ctypes.c_int32()
    assert fn(ctypes.byref(m), reqs.array, reqs.count, None, 0, ctypes.byref(count), ctypes.byref(wg)) == 0
    units = np.zeros(count.value, dtype=UNIT_DTYPE)
    assert fn(ctypes.byref(m), reqs.array, reqs.count, units.ctypes.data, count.value, ctypes.byref(count),
              ctypes.byref(wg)) == 0
    return units, wg.value


def emulate(case):
    """Workgroup 2u + which encodes the K (0) or V (1) tile of unit u; wave w
    of it encodes heads w, w + waves, ...; lane l holds channels
    [8c, 8c + 8) of row r of every load (r = l // (D/8), c = l % (D/8))."""
    s = case.src_shape
    H, D, B, P, L = s.num_kv_heads, s.head_dim, s.block_tokens, s.page_size, s.num_layers
    units, WG = checkpoint_units(s, case.requests)
    assert WG == 64 * min(H, MAX_WAVES)
    nwaves = WG // 64
    lpr = D // 8
    rpl = 64 // lpr
    lane = np.arange(64)
    r, c = lane // lpr, lane % lpr
    on = r < rpl
    nload = -(-B // rpl)
    NL = loads_per_chunk(nload)
    nchunk = -(-nload // NL)
    paired = s.kv_layout == wl.KV_PAIRED
    shift = int(np.log2(P)) + int(paired)  # slot rows from a layer's start to page p: p << shift
    layer_elems = (2 if paired else 1) * s.pool_pages * P * H * D
    v_offset = P * H * D if paired else 0  # V reads in the one paired buffer; separate caches share cache_read
    cache_read = np.zeros(L * layer_elems, dtype=np.int32)
    pw = np.zeros(case.payload_nbytes, dtype=np.int32)
    sw = np.zeros(case.scale_elems, dtype=np.int32)
    pt_all = np.concatenate([r_.src_page_table for r_ in case.requests]).astype(np.int64)
    assert len(units) == L * sum(r_.num_blocks for r_ in case.requests)
    passes_of = {}
    for u in units:
        tag = int(u["tag"]) & 0xFF
        n_valid = int(u["n_valid"])
        assert 1 <= n_valid <= B
        for which, (off, bits) in enumerate(((int(u["k_off"]), KBITS[tag]), (int(u["v_off"]), VBITS[tag]))):
            passes = 1 if bits == 16 or nchunk == 1 else 2
            passes_of[(int(u["layer"]), int(u["row0"]), which)] = passes
            for w in range(nwaves):
                for head in range(w, H, nwaves):
                    for ch in range(nchunk):
                        for i in range(NL):
                            t = (ch * NL + i) * rpl + r
                            rd = on & (t < n_valid)
                            rows = int(u["row0"]) + t[rd]
                            pages = pt_all[int(u["pt_off"]) + rows // P]
                            assert ((pages >= 0) & (pages < s.pool_pages)).all()
                            base = (int(u["layer"]) * layer_elems + ((pages << shift) | (rows % P)) * H * D + head * D
                                    + 8 * c[rd] + which * v_offset)
                            for e in range(8):
                                np.add.at(cache_read, base + e, passes)
                            wr = on & (t < B)
                            tt, cc = t[wr], c[wr]
                            if bits == 16:
                                st, ln = off + (tt * H + head) * D * 2 + 16 * cc, 16
                            elif bits == 8:
                                st, ln = off + (tt * H + head) * D + 8 * cc, 8
                            else:
                                st, ln = off + (tt * H + head) * (D // 2) + 4 * cc, 4
                            assert (st >= 0).all() and (st + ln <= pw.size).all()
                            for b in range(ln):
                                np.add.at(pw, st + b, 1)
                    e0 = int(u["scale_off"]) + 4 * head + 2 * which
                    sw[e0: e0 + 2] += 1
    # every checkpoint byte / scale element exactly once, nothing else
    want_p = np.zeros_like(pw)
    want_s = np.zeros_like(sw)
    for r_ in case.requests:
        pbytes, selems = wl.encoded_request_nbytes(case.shape, r_)
        want_p[r_.payload_offset: r_.payload_offset + pbytes] = 1
        want_s[r_.scale_offset: r_.scale_offset + selems] = 1
    assert np.array_equal(pw, want_p)
    assert np.array_equal(sw, want_s)
    # reads: exactly the suffix rows, once per pass of each (layer, K|V) tile
    want_r = np.zeros_like(cache_read)
    for r_ in case.requests:
        for b in range(r_.num_blocks):
            tag = int(r_.tags[b])
            n = min(B, r_.suffix_tokens - b * B)
            rows = r_.src_row0 + b * B + np.arange(n)
            slot_rows = (r_.src_page_table[rows // P].astype(np.int64) << shift) | (rows % P)
            for layer in range(L):
                for which, bits in enumerate((KBITS[tag], VBITS[tag])):
                    k = 1 if bits == 16 or nchunk == 1 else 2
                    for sl in slot_rows:
                        b0 = layer * layer_elems + sl * H * D + which * v_offset
                        want_r[b0: b0 + H * D] += k
    assert np.array_equal(cache_read, want_r)


@pytest.mark.parametrize("maker", [
    lambda: wl.make_case("tiny"),
    lambda: wl.make_case("tiny", int4_tag=wl.TAG_K4V4),
    lambda: wl.make_custom(1, L=2, H=3, D=128, B=32, P=16, n_tokens=(70,), deltas=(12,), rho0s=(29,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    lambda: wl.make_custom(2, L=1, H=8, D=64, B=4, P=16, n_tokens=(23, 9), deltas=(5, 0), rho0s=(7, 40),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    lambda: wl.make_custom(3, L=1, H=4, D=128, B=64, P=32, n_tokens=(130,), deltas=(-9,), rho0s=(31,),
                           tag_set=(0, 2), mix=(1, 1)),
    lambda: wl.make_custom(5, L=2, H=8, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    # D = 48: 6 lanes per row, lanes 60..63 idle; D = 512 with B = 64: two chunks (rows streamed twice)
    lambda: wl.make_custom(6, L=1, H=2, D=48, B=16, P=16, n_tokens=(37,), deltas=(2,), rho0s=(5,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    lambda: wl.make_custom(7, L=1, H=2, D=512, B=64, P=16, n_tokens=(150,), deltas=(-2,), rho0s=(9,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    lambda: wl.make_custom(8, L=1, H=20, D=16, B=8, P=8, n_tokens=(21,), deltas=(1,), rho0s=(3,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
], ids=["tiny", "tiny_k4v4", "h3_d128", "h8_b4_two_requests", "h4_b64", "h8_d128", "d48_idle_lanes",
        "d512_two_chunks", "h20_heads_loop"])
def test_gather_addresses(maker):
    emulate(maker())


def _paired(case):
    import dataclasses
    case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    return case


@pytest.mark.parametrize("maker", [
    lambda: _paired(wl.make_case("tiny")),
    lambda: _paired(wl.make_custom(2, L=1, H=8, D=64, B=4, P=16, n_tokens=(23, 9), deltas=(5, 0), rho0s=(7, 40),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1))),
    lambda: _paired(wl.make_custom(5, L=2, H=8, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1))),
    # general kernel: blocks over more than three pages
    lambda: _paired(wl.make_custom(9, L=1, H=4, D=64, B=32, P=8, n_tokens=(77,), deltas=(1,), rho0s=(6,),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1))),
], ids=["tiny", "h8_b4_two_requests", "h8_d128", "general_kernel"])
def test_gather_addresses_paired_pages(maker):
    emulate(maker())


@pytest.mark.parametrize("maker", [
    lambda: wl.make_case("tiny"),
    lambda: wl.make_custom(2, L=1, H=8, D=64, B=4, P=16, n_tokens=(23, 9), deltas=(5, 0), rho0s=(7, 40),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    lambda: wl.make_custom(3, L=1, H=4, D=64, B=64, P=32, n_tokens=(130,), deltas=(-9,), rho0s=(31,),
                           tag_set=(0, 2), mix=(1, 1)),
    lambda: wl.make_custom(5, L=2, H=8, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    lambda: wl.make_custom(8, L=1, H=20, D=16, B=8, P=8, n_tokens=(21,), deltas=(1,), rho0s=(3,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    # 70B-shaped blocks: 64 tokens over 32-token pages, 16 loads per lane in 8-wave workgroups
    lambda: wl.make_custom(13, L=1, H=8, D=128, B=64, P=32, n_tokens=(150, 64), deltas=(4096, 0), rho0s=(31, 96),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
], ids=["tiny", "h8_b4_two_requests", "h4_d64_b64", "h8_d128", "h20_heads_loop", "h8_d128_b64_p32"])
def test_tile_kernel_tiles_and_pages(maker):
    """Tile kernel (blocks of at most 2P + 1 tokens, at most 16 loads per lane):
    wave w of workgroup b encodes tile b * waves + w of the (unit, K|V, head)
    order, so a grid of ceil(tiles / waves) workgroups encodes every tile
    exactly once; the three source pages carried in each unit give every
    valid row's page, and rows past n_valid read the block's first row."""
    case = maker()
    s = case.src_shape
    H, D, B, P = s.num_kv_heads, s.head_dim, s.block_tokens, s.page_size
    assert B <= 2 * P + 1
    units, WG = checkpoint_units(s, case.requests)
    nwaves = WG // 64
    ntiles = len(units) * 2 * H
    grid = -(-ntiles // nwaves)
    T = (np.arange(grid)[:, None] * nwaves + np.arange(nwaves)[None, :]).reshape(-1)
    T = T[T < ntiles]
    assert np.array_equal(np.sort(T), np.arange(ntiles))
    # tile -> (unit, K|V, head)
    ui, rest = T // (2 * H), T % (2 * H)
    assert ((rest >= H) == (rest // H == 1)).all() and (ui < len(units)).all()
    pt_all = np.concatenate([r_.src_page_table for r_ in case.requests]).astype(np.int64)
    lpr = D // 8
    rpl = 64 // lpr
    nload = -(-B // rpl)
    assert loads_per_chunk(nload) <= 16 and loads_per_chunk(nload) >= nload
    for u in units:
        pages = [int(u["table_off"]), int(u["page1"]), int(u["page2"])]  # page0 shares table_off's slot
        first = int(u["row0"]) // P
        for t in range(B):
            row = int(u["row0"]) + (t if t < int(u["n_valid"]) else 0)
            k = row // P - first
            assert 0 <= k <= 2
            assert pages[k] == pt_all[int(u["pt_off"]) + row // P]
            assert 0 <= pages[k] < s.pool_pages


HALF_WAVES = 8  # waves per workgroup of the half-tile kernel


@pytest.mark.parametrize("maker", [
    lambda: wl.make_custom(13, L=1, H=8, D=128, B=64, P=32, n_tokens=(150, 64), deltas=(4096, 0), rho0s=(31, 96),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
    # 12 loads per lane (a 16-load chunk), three heads: tiles of different (unit, K|V) share workgroups
    lambda: wl.make_custom(14, L=2, H=3, D=128, B=48, P=32, n_tokens=(100,), deltas=(7,), rho0s=(5,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1)),
], ids=["h8_d128_b64_p32", "h3_d128_b48"])
def test_half_tile_kernel_mapping(maker):
    """Half-tile kernel (9 to 16 loads per lane): wave w of workgroup b is
    half-tile W = 8b + w, tile W >> 1, half W & 1, so both halves of a tile sit
    in one workgroup (the range exchange), every tile is covered exactly once
    by its two halves' rows, and each tile's scale word is written once."""
    case = maker()
    s = case.src_shape
    H, D, B = s.num_kv_heads, s.head_dim, s.block_tokens
    units, _ = checkpoint_units(s, case.requests)
    lpr = D // 8
    rpl = 64 // lpr
    nload = -(-B // rpl)
    assert 8 < nload <= 16 and loads_per_chunk(nload) == 16
    ntiles = len(units) * 2 * H
    grid = -(-2 * ntiles // HALF_WAVES)
    lane = np.arange(64)
    r, c = lane // lpr, lane % lpr
    on = r < rpl
    rows_of = np.zeros((ntiles, B, lpr), dtype=np.int32)  # (tile, row, channel piece) writes
    scale_writes = np.zeros(ntiles, dtype=np.int32)
    for b in range(grid):
        for w in range(HALF_WAVES):
            W = b * HALF_WAVES + w
            T, half = W >> 1, W & 1
            assert (W ^ 1) // HALF_WAVES == b  # the partner half is in the same workgroup
            if T >= ntiles:
                continue  # such waves read tile 0, store nothing, and still pass the barrier
            for i in range(8):
                t = half * 8 * rpl + i * rpl + r
                st = on & (t < B)
                np.add.at(rows_of[T], (t[st], c[st]), 1)
            if half == 0:
                scale_writes[T] += 1
    assert (rows_of == 1).all() and (scale_writes == 1).all()
