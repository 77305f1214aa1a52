"""The allocation-free streamed restore (pkv_restore_from_host_noalloc)
against pkv_restore_from_host, through the C ABI: identical caches, bit for
bit, on two calls in a row (the second with a smaller plan), and the oracle's
restore on both.  The first case's request-layers span more than the 64 MiB
stage, so they run in several payload windows."""
import numpy as np
import pytest

from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

from parity import check_full, log, oracle_checkpoint

pytestmark = pytest.mark.gpu

FILL = 0x5A


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    pb.load()
    return _t


def _paired(case):
    import dataclasses
    case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    return case


def _big():
    # 32768 tokens x 8 heads x 128, mostly FP16: about 98 MiB per request-layer
    # (two windows), plus a short second request; two layers.
    return _paired(wl.make_custom(31, L=2, H=8, D=128, B=32, P=16, n_tokens=(32768, 900), deltas=(-1500, 37),
                                  rho0s=(5007, 40000), tag_set=(0, 1, 2, 3), mix=(0.6, 0.2, 0.1, 0.1),
                                  repair_frac=0.15, out_dtype=wl.OUT_BF16, theta=5e5, outlier_pairs=1))


def _both(case, torch):
    from paper_2609_26219_amd.device import DeviceRestore

    ckpt = oracle_checkpoint(case)
    hp = torch.from_numpy(ckpt[0]).pin_memory()
    hs = torch.from_numpy(ckpt[1].view(np.int16)).pin_memory()
    blank = (np.full(ckpt[0].shape, FILL, np.uint8), np.full(ckpt[1].shape, FILL * 0x101, np.uint16))
    dr = DeviceRestore(case, checkpoint=blank)
    pb.restore_from_host_tensors(dr.plan, hp, hs, dr.payload, dr.scales, dr.k_cache, dr.v_cache)
    torch.cuda.synchronize()
    ref = dr.host_caches()
    dr.prefill()
    nb = lambda t: t.numel() * t.element_size()
    st = pb.pkv_restore_from_host_noalloc_status(dr.plan, hp.data_ptr(), nb(hp), hs.data_ptr(), nb(hs),
                                                 dr.k_cache.data_ptr(), dr.v_cache.data_ptr(),
                                                 pb.cache_nbytes(dr.k_cache, dr.v_cache),
                                                 torch.cuda.current_stream().cuda_stream)
    assert st == pb.PKV_OK, pb.pkv_status_string(st)
    torch.cuda.synchronize()
    got = dr.host_caches()
    assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])
    stats = check_full(dr, ckpt)
    log(f"  {case.name}: identical to pkv_restore_from_host; oracle: {stats.n} elements, "
        f"{stats.n_near_tie} near-tie neighbours, 0 wrong")
    return dr, hp, hs


def test_noalloc_matches_streamed_restore_two_calls(torch):
    log("[gpu] allocation-free streamed restore: a two-window case, then tiny")
    _both(_big(), torch)
    _both(wl.make_case("tiny"), torch)


def test_noalloc_rejects_pageable_and_oversized(torch):
    """Pageable host memory, and a request-layer whose scales exceed the 4 MiB
    stage, are refused before anything is enqueued."""
    from paper_2609_26219_amd.device import DeviceRestore

    case = wl.make_case("tiny")
    ckpt = oracle_checkpoint(case)
    dr = DeviceRestore(case, checkpoint=ckpt)
    before = dr.host_caches()
    p, s = np.ascontiguousarray(ckpt[0]), np.ascontiguousarray(ckpt[1])
    cb = pb.cache_nbytes(dr.k_cache, dr.v_cache)
    st = pb.pkv_restore_from_host_noalloc_status(dr.plan, p.ctypes.data, p.nbytes, s.ctypes.data, s.nbytes,
                                                 dr.k_cache.data_ptr(), dr.v_cache.data_ptr(), cb)
    assert st == pb.PKV_ERR_INVALID_ARGUMENT
    # 1 KV head x 32 channels, blocks of 1 token: ceil(N / B) * H * 8 bytes of scales per layer, 8 bytes over
    big = wl.make_custom(3, L=1, H=1, D=32, B=1, P=1024, n_tokens=(524289,), deltas=(1,), rho0s=(0,),
                         tag_set=(1,), mix=(1.0,), repair_frac=0.0, out_dtype=wl.OUT_FP16)
    plan = pb.pkv_restore_plan(big.shape, big.requests)
    hp = torch.zeros(big.payload_nbytes, dtype=torch.uint8).pin_memory()
    hs = torch.zeros(big.scale_elems, dtype=torch.int16).pin_memory()
    k = torch.zeros(pb.pkv_plan_query(plan)["cache_bytes"] // 2, dtype=torch.int16, device="cuda")
    v = torch.zeros_like(k)
    st = pb.pkv_restore_from_host_noalloc_status(plan, hp.data_ptr(), big.payload_nbytes, hs.data_ptr(),
                                                 2 * big.scale_elems, k.data_ptr(), v.data_ptr(), 2 * k.numel())
    assert st == pb.PKV_ERR_INVALID_ARGUMENT
    torch.cuda.synchronize()
    after = dr.host_caches()
    assert np.array_equal(before[0], after[0]) and np.array_equal(before[1], after[1])
    assert int(k.abs().sum()) == 0 and int(v.abs().sum()) == 0
