"""CPU replay of the staged streamed restore (pkv_restore_from_host_noalloc):
every unit restored in exactly one step, every payload and scale byte it
reads copied into the stage by that step (or, for scales, by an earlier step
of the same request-layer), every stage address inside the stage, and only
reused blocks (plus repair blocks between close reused ones) copied."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl
from parity import host_gap_bytes
from test_kernel_indexing import host_units

STAGE_PAYLOAD = 64 << 20
STAGE_SCALES = 4 << 20
KBITS = (16, 8, 8, 4)
VBITS = (16, 8, 4, 4)


def stage_schedule(shape, requests):
    fn = pb.load().pkv_internal_stage_schedule
    fn.argtypes = [ctypes.POINTER(pb.PkvModel), ctypes.POINTER(pb.PkvRequest), ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64),
                   ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32)]
    fn.restype = ctypes.c_int32
    m = pb.make_model(shape)
    reqs = pb._Requests(requests)
    ns, nc, ok = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
    assert fn(ctypes.byref(m), reqs.array, reqs.count, None, 0, None, 0, ctypes.byref(ns), ctypes.byref(nc),
              ctypes.byref(ok)) == 0
    steps = np.zeros((ns.value, 8), np.int64)
    copies = np.zeros((nc.value, 3), np.uint64)
    assert fn(ctypes.byref(m), reqs.array, reqs.count, steps.ctypes.data, len(steps), copies.ctypes.data, len(copies),
              ctypes.byref(ns), ctypes.byref(nc), ctypes.byref(ok)) == 0
    return steps, copies.astype(np.int64), bool(ok.value)


def _covered(ranges, a, b):
    """[a, b) inside the union of half-open ranges (sorted, merged here)."""
    for lo, hi in ranges:
        if lo <= a and b <= hi:
            return True
    return False


CASES = [
    ("tiny", lambda: wl.make_case("tiny")),
    ("three_requests_3l", lambda: wl.make_custom(4, L=3, H=2, D=64, B=16, P=16, n_tokens=(137, 16, 50),
                                                 deltas=(3, 0, -7), rho0s=(0, 6, 13), tag_set=(0, 1, 2, 3),
                                                 mix=(1, 1, 1, 1), repair_frac=0.3, out_dtype=wl.OUT_BF16)),
    ("fp16_only", lambda: wl.make_custom(7, L=2, H=2, D=64, B=16, P=16, n_tokens=(90,), deltas=(5,), tag_set=(0,),
                                         mix=(1,), repair_frac=0.25)),
    ("all_repair", lambda: wl.make_custom(6, L=2, H=2, D=64, B=16, P=16, n_tokens=(64, 20), deltas=(4, 2),
                                          repair_all=True)),
    # 16 MiB FP16 blocks (1024 tokens x 32 heads x 128): request-layers span several 64 MiB windows
    ("windows", lambda: wl.make_custom(8, L=2, H=32, D=128, B=1024, P=1024, n_tokens=(9 * 1024 + 300, 2000),
                                       deltas=(-3, 9), rho0s=(7, 50), tag_set=(0, 1, 2, 3), mix=(0.7, 0.1, 0.1, 0.1),
                                       repair_frac=0.2)),
    ("llama8b_1l", lambda: wl.make_case("llama8b_1l")),
]


@pytest.mark.parametrize("name,maker", CASES, ids=[c[0] for c in CASES])
def test_stage_schedule_replay(name, maker):
    case = maker()
    s = case.shape
    B, H, D, L = s.block_tokens, s.num_kv_heads, s.head_dim, s.num_layers
    steps, copies, ok = stage_schedule(s, case.requests)
    assert ok
    units = host_units(s, case.requests)
    gap = host_gap_bytes()
    done = np.zeros(len(units), np.int32)
    staged_scales = None  # (scale0, count) held by the stage
    windows_per_rl = {}
    for u0, u1, lo, hi, scale0, scale_elems, c0, c1 in steps:
        assert 0 <= u0 < u1 <= len(units) and lo < hi and c0 < c1 <= len(copies)
        assert hi - lo <= STAGE_PAYLOAD
        if scale_elems:
            assert scale_elems * 2 <= STAGE_SCALES
            staged_scales = (scale0, scale_elems)
        cps = copies[c0:c1]
        assert (cps[:, 1] == cps[:, 0] - lo).all() and (cps[:, 1] + cps[:, 2] <= STAGE_PAYLOAD).all()
        src = [(int(a), int(a + n)) for a, _, n in cps]
        blk = units[u0:u1]
        layer = int(blk["layer"][0])
        ri = int(blk["table_off"][0]) // D
        assert (blk["layer"] == layer).all() and (blk["table_off"] == ri * D).all()
        windows_per_rl[(layer, ri)] = windows_per_rl.get((layer, ri), 0) + 1
        req = case.requests[ri]
        nb = len(req.tags)
        base = case.layer_payload_offset(ri, layer)
        # copies: whole reused blocks of this request-layer, plus repair blocks lying in short gaps between them
        offsets, _ = oracle.block_layout(req.tags, B, H, D)
        spans = sorted((base + offsets[b][0], base + offsets[b][1] + B * H * D * VBITS[int(req.tags[b])] // 8, b)
                       for b in range(nb))
        for a, e in src:
            inside = [(x, y, b) for x, y, b in spans if a <= x and y <= e]
            assert inside and inside[0][0] == a and inside[-1][1] == e
            assert not req.repair[inside[0][2]] and not req.repair[inside[-1][2]]
            for (x0, y0, b0), (x1, y1, b1) in zip(inside, inside[1:]):
                assert y0 == x1
        act = np.nonzero((blk["k_off"] >= lo) & (blk["k_off"] < hi))[0]
        for i in act:
            u = blk[i]
            tag = int(u["tag"]) & 0xFF
            n = int(u["n_valid"])
            for off, bits in ((int(u["k_off"]), KBITS[tag]), (int(u["v_off"]), VBITS[tag])):
                end = off + n * H * D * bits // 8
                assert lo <= off and end - lo <= STAGE_PAYLOAD
                assert _covered(src, off, end), (name, off, end)
            if tag != 0:
                so = int(u["scale_off"])
                assert staged_scales is not None and staged_scales[0] == req.scale_offset + layer * nb * H * 4
                assert staged_scales[0] <= so and so + 4 * H <= staged_scales[0] + staged_scales[1]
            done[u0 + i] += 1
    assert (done == 1).all(), "every unit is restored by exactly one step"
    if name == "windows":
        assert max(windows_per_rl.values()) >= 2
    # every reused byte of every request-layer is copied by some step
    for ri, req in enumerate(case.requests):
        offsets, _ = oracle.block_layout(req.tags, B, H, D)
        for layer in range(L):
            base = case.layer_payload_offset(ri, layer)
            for b in oracle.reused_blocks(req):
                a = base + offsets[b][0]
                e = base + offsets[b][1] + B * H * D * VBITS[int(req.tags[b])] // 8
                assert any(x <= a and e <= x + n for x, _, n in copies), (ri, layer, b)
    assert gap > 0


def test_stage_refused_when_scales_exceed_the_stage():
    # one request-layer holds ceil(N / B) * H * 8 bytes of scales: 8 bytes over 4 MiB
    big = wl.make_custom(3, L=1, H=1, D=32, B=1, P=1024, n_tokens=(524289,), deltas=(1,), rho0s=(0,), tag_set=(1,),
                         mix=(1.0,), repair_frac=0.0, out_dtype=wl.OUT_FP16)
    _, _, ok = stage_schedule(big.shape, big.requests)
    assert not ok
    fits = wl.make_custom(3, L=1, H=1, D=32, B=1, P=1024, n_tokens=(524288,), deltas=(1,), rho0s=(0,), tag_set=(1,),
                          mix=(1.0,), repair_frac=0.0, out_dtype=wl.OUT_FP16)
    _, _, ok = stage_schedule(fits.shape, fits.requests)
    assert ok
    # FP16 blocks read no scales, so any length stages
    fp16 = wl.make_custom(3, L=1, H=1, D=32, B=1, P=1024, n_tokens=(524289,), deltas=(1,), rho0s=(0,), tag_set=(0,),
                          mix=(1.0,), repair_frac=0.0, out_dtype=wl.OUT_FP16)
    _, _, ok = stage_schedule(fp16.shape, fp16.requests)
    assert ok
