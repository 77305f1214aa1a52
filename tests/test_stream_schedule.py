"""CPU checks of the streamed restore's schedule (pkv_restore_from_host):
layer-major work items, and host -> device copy ranges that cover exactly the
reused blocks' payload bytes of each layer plus that layer's scale entries."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl
from parity import host_gap_bytes, streamed_payload_ranges
from test_kernel_indexing import UNIT_DTYPE, host_units


def schedule(shape, requests):
    lib = pb.load()
    fn = lib.pkv_internal_stream_schedule
    fn.argtypes = [ctypes.POINTER(pb.PkvModel), ctypes.POINTER(pb.PkvRequest), ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_int64, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64), ctypes.c_void_p]
    fn.restype = ctypes.c_int32
    m = pb.make_model(shape)
    reqs = pb._Requests(requests)
    npay, nsc = ctypes.c_int64(), ctypes.c_int64()
    layers = np.zeros((3, shape.num_layers + 1), np.int64)
    assert fn(ctypes.byref(m), reqs.array, reqs.count, None, 0, ctypes.byref(npay), ctypes.byref(nsc),
              layers.ctypes.data) == 0
    ranges = np.zeros((npay.value + nsc.value, 2), np.uint64)
    assert fn(ctypes.byref(m), reqs.array, reqs.count, ranges.ctypes.data, len(ranges), ctypes.byref(npay),
              ctypes.byref(nsc), layers.ctypes.data) == 0
    return ranges[:npay.value].astype(np.int64), ranges[npay.value:].astype(np.int64), layers


CASES = [
    lambda: wl.make_custom(4, L=3, H=2, D=64, B=16, P=16, n_tokens=(137, 16, 50), deltas=(3, 0, -7),
                           rho0s=(0, 6, 13), tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.3,
                           out_dtype=wl.OUT_BF16, outlier_pairs=1),
    lambda: wl.make_case("tiny"),
    lambda: wl.make_custom(4, L=3, H=2, D=32, B=8, P=4, n_tokens=(37, 16, 5), deltas=(3, 0, -7), rho0s=(0, 6, 13),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.3),
    lambda: wl.make_custom(5, L=2, H=4, D=64, B=16, P=16, n_tokens=(100, 64), deltas=(1, 2), repair_frac=0.0),
    lambda: wl.make_custom(6, L=2, H=2, D=64, B=16, P=16, n_tokens=(64, 20), deltas=(4, 2), repair_all=True),
    lambda: wl.make_custom(7, L=2, H=2, D=64, B=16, P=16, n_tokens=(90,), deltas=(5,), tag_set=(0,), mix=(1,),
                           repair_frac=0.25),
]


@pytest.mark.parametrize("maker", CASES, ids=["three_requests_3l", "tiny", "three_requests", "no_repair", "all_repair", "fp16_only"])
def test_stream_schedule(maker):
    """The library's copy list equals an independent recomputation at the
    library's merge gap, covers every reused byte, and adds only repair-block
    bytes lying between reused ones."""
    case = maker()
    s = case.shape
    B, H, D, L = s.block_tokens, s.num_kv_heads, s.head_dim, s.num_layers
    pay, sc, layers = schedule(s, case.requests)
    units = host_units(s, case.requests)
    # layer-major work items: layer l owns units [layers[0][l], layers[0][l + 1])
    assert layers[0][0] == 0 and layers[0][-1] == len(units)
    for l in range(L):
        assert (units["layer"][layers[0][l]:layers[0][l + 1]] == l).all()
    lib_gap = host_gap_bytes()
    want_all = streamed_payload_ranges(case, lib_gap)
    exact = streamed_payload_ranges(case, 0)
    for l in range(L):
        got = [(int(o), int(n)) for o, n in pay[layers[1][l]:layers[1][l + 1]]]
        assert got == want_all[l], l
        # the merged copies cover every reused byte, and only repair bytes lie in between
        covered = set()
        for o, n in got:
            covered |= set(range(o, o + n))
        reused = set()
        for o, n in exact[l]:
            reused |= set(range(o, o + n))
        assert reused <= covered
        # copies of one layer never overlap each other
        ends = sorted((o, o + n) for o, n in got)
        assert all(a[1] <= b[0] for a, b in zip(ends, ends[1:]))
    # and copies of different layers never overlap either
    allr = sorted((int(o), int(o + n)) for o, n in pay)
    assert all(a[1] <= b[0] for a, b in zip(allr, allr[1:]))
    # scale copies: the whole per-layer scale block of each request with a reused quantized block
    for l in range(L):
        want_s = []
        for ri, req in enumerate(case.requests):
            nb = len(req.tags)
            if any(not req.repair[b] and int(req.tags[b]) != 0 for b in range(nb)):
                want_s.append(((req.scale_offset + l * nb * H * 4) * 2, nb * H * 8))
        got_s = [(int(o), int(n)) for o, n in sc[layers[2][l]:layers[2][l + 1]]]
        # adjacent requests' scale blocks may be one copy
        merged = []
        for o, n in want_s:
            if merged and merged[-1][0] + merged[-1][1] == o:
                merged[-1] = (merged[-1][0], merged[-1][1] + n)
            else:
                merged.append((o, n))
        assert got_s == merged, l
