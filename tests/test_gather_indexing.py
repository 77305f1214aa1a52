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

GATHER_TOKENS = 4  # tokens per thread
KBITS = (16, 8, 8, 4)
VBITS = (16, 8, 4, 4)
UNIT_DTYPE = np.dtype([("k_off", "<u8"), ("v_off", "<u8"), ("scale_off", "<u8"), ("row0", "<i8"), ("pt_off", "<i8"),
                       ("table_off", "<i4"), ("layer", "<i4"), ("tag", "<i4"), ("n_valid", "<i4"),
                       ("reserved", "<i8")])


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
    s = case.src_shape
    H, D, B, P, L = s.num_kv_heads, s.head_dim, s.block_tokens, s.page_size, s.num_layers
    units, WG = checkpoint_units(s, case.requests)
    cols = H * D // 16
    tpp = WG // cols
    assert WG % 64 == 0 and WG <= 1024 and tpp * GATHER_TOKENS >= B
    dq = D // 16
    tid = np.arange(WG)
    t0 = tid // cols
    active = t0 < tpp
    c = tid % cols
    head = c // dq
    j = c % dq
    layer_elems = s.pool_pages * P * H * D
    cache_read = np.zeros(L * layer_elems, dtype=np.int32)
    pw = np.zeros(case.payload_nbytes, dtype=np.int32)
    sw = np.zeros(case.scale_elems, dtype=np.int32)
    pt_all = np.concatenate([r.src_page_table for r in case.requests]).astype(np.int64)
    assert len(units) == L * sum(r.num_blocks for r in case.requests)
    for u in units:
        tag = int(u["tag"]) & 0xFF
        n_valid = int(u["n_valid"])
        assert 1 <= n_valid <= B
        for which, (off, bits) in enumerate(((int(u["k_off"]), KBITS[tag]), (int(u["v_off"]), VBITS[tag]))):
            for i in range(GATHER_TOKENS):
                t = t0 + i * tpp
                rd = active & (t < n_valid)
                wr = active & (t < B)
                for th in np.nonzero(rd)[0]:
                    row = int(u["row0"]) + int(t[th])
                    page = int(pt_all[int(u["pt_off"]) + (row // P)])
                    assert 0 <= page < s.pool_pages
                    base = int(u["layer"]) * layer_elems + (page * P + row % P) * H * D + int(head[th]) * D
                    for o in (8 * int(j[th]), D // 2 + 8 * int(j[th])):
                        assert base + o + 8 <= cache_read.size
                        cache_read[base + o: base + o + 8] += 1
                for th in np.nonzero(wr)[0]:
                    r = int(t[th]) * H + int(head[th])
                    jj = int(j[th])
                    if bits == 16:
                        spans = [(off + r * D * 2 + 16 * jj, 16), (off + r * D * 2 + D + 16 * jj, 16)]
                    elif bits == 8:
                        spans = [(off + r * D + 8 * jj, 8), (off + r * D + D // 2 + 8 * jj, 8)]
                    else:
                        spans = [(off + r * (D // 2) + 4 * jj, 4), (off + r * (D // 2) + D // 4 + 4 * jj, 4)]
                    for st, ln in spans:
                        assert 0 <= st and st + ln <= pw.size
                        pw[st: st + ln] += 1
            writers = np.nonzero(active & (t0 == 0) & (j == 0))[0]
            for th in writers:
                e = int(u["scale_off"]) + 4 * int(head[th]) + 2 * which
                sw[e: e + 2] += 1
    # every checkpoint byte / scale element exactly once, nothing else
    want_p = np.zeros_like(pw)
    want_s = np.zeros_like(sw)
    for r in case.requests:
        pbytes, selems = wl.encoded_request_nbytes(case.shape, r)
        want_p[r.payload_offset: r.payload_offset + pbytes] = 1
        want_s[r.scale_offset: r.scale_offset + selems] = 1
    assert np.array_equal(pw, want_p)
    assert np.array_equal(sw, want_s)
    # reads: exactly the suffix rows, each element of each row read once per (layer, K|V) pass
    want_r = np.zeros_like(cache_read)
    for r in case.requests:
        rows = r.src_row0 + np.arange(r.suffix_tokens)
        slots = r.src_page_table[rows // P].astype(np.int64) * P + rows % P
        for layer in range(L):
            for sl in slots:
                b0 = layer * layer_elems + sl * H * D
                want_r[b0: b0 + H * D] += 2
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
], ids=["tiny", "tiny_k4v4", "h3_d128", "h8_b4_two_requests", "h4_b64", "h8_d128"])
def test_gather_addresses(maker):
    emulate(maker())
