"""GPU parity of the streamed restore from host memory (pkv_restore_from_host):
same caches as the oracle's restore and as pkv_restore, and only the reused
blocks' bytes (plus per-layer scales) copied into the device checkpoint."""
import numpy as np
import pytest

from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

from parity import check_full, host_gap_bytes, log, oracle_checkpoint, reused_byte_masks

pytestmark = pytest.mark.gpu

FILL = 0x5A


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    pb.load()
    return _t


def _streamed(case, torch, pinned=True, stream=None):
    from paper_2609_26219_amd.device import DeviceRestore
    ckpt = oracle_checkpoint(case)
    blank = (np.full(ckpt[0].shape, FILL, np.uint8), np.full(ckpt[1].shape, FILL * 0x101, np.uint16))
    dr = DeviceRestore(case, checkpoint=blank)
    hp = torch.from_numpy(ckpt[0])
    hs = torch.from_numpy(ckpt[1].view(np.int16))
    if pinned:
        hp, hs = hp.pin_memory(), hs.pin_memory()
    if stream is None:
        pb.restore_from_host_tensors(dr.plan, hp, hs, dr.payload, dr.scales, dr.k_cache, dr.v_cache)
    else:
        with torch.cuda.stream(stream):
            pb.restore_from_host_tensors(dr.plan, hp, hs, dr.payload, dr.scales, dr.k_cache, dr.v_cache)
    torch.cuda.synchronize()
    return dr, ckpt


def _check_copied_only_reused(case, dr, ckpt):
    pmask, smask = reused_byte_masks(case, host_gap_bytes())
    p = dr.payload.cpu().numpy()[:ckpt[0].size]
    sc = dr.scales.cpu().numpy().view(np.uint16)[:ckpt[1].size]
    assert np.array_equal(p[pmask], ckpt[0][pmask]) and (p[~pmask] == FILL).all()
    assert np.array_equal(sc[smask], ckpt[1][smask]) and (sc[~smask] == FILL * 0x101).all()
    info = dr.info
    assert info["host_copy_bytes"] == int(pmask.sum()) + 2 * int(smask.sum())
    log(f"  copied {info['host_copy_bytes']} of {ckpt[0].size + 2 * ckpt[1].size} checkpoint bytes "
        f"in {info['host_copies']} copies")


def _paired(case):
    import dataclasses
    case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    return case


CASES = [
    ("tiny", lambda: wl.make_case("tiny")),
    ("llama8b_1l", lambda: wl.make_case("llama8b_1l")),
    ("three_requests_3l", lambda: wl.make_custom(4, L=3, H=2, D=64, B=16, P=16, n_tokens=(137, 16, 50),
                                                 deltas=(3, 0, -7), rho0s=(0, 6, 13), tag_set=(0, 1, 2, 3),
                                                 mix=(1, 1, 1, 1), repair_frac=0.3, out_dtype=wl.OUT_BF16,
                                                 outlier_pairs=1)),
    ("llama8b_1l_paired_pages", lambda: _paired(wl.make_case("llama8b_1l"))),
]


@pytest.mark.parametrize("name,maker", CASES, ids=[c[0] for c in CASES])
def test_streamed_restore_parity(name, maker, torch):
    log(f"[gpu] streamed restore from pinned host memory: {name}")
    case = maker()
    dr, ckpt = _streamed(case, torch)
    st = check_full(dr, ckpt)
    log(f"  {st}")
    _check_copied_only_reused(case, dr, ckpt)


def test_streamed_equals_device_restore(torch):
    case = wl.make_case("llama8b_1l")
    dr, ckpt = _streamed(case, torch)
    k2 = torch.zeros_like(dr.k_cache)
    v2 = torch.zeros_like(dr.v_cache)
    dp = torch.from_numpy(ckpt[0]).cuda()
    ds = torch.from_numpy(ckpt[1].view(np.int16)).cuda()
    dr.prefill()
    pb.restore_tensors(dr.plan, dp, ds, dr.k_cache, dr.v_cache)
    torch.cuda.synchronize()
    k_dev, v_dev = dr.host_caches()
    dr2, _ = _streamed(case, torch)
    k_h, v_h = dr2.host_caches()
    assert np.array_equal(k_dev, k_h) and np.array_equal(v_dev, v_h)


def test_streamed_pageable_and_side_stream(torch):
    case = wl.make_custom(9, L=2, H=4, D=64, B=16, P=16, n_tokens=(70, 33), deltas=(2, -5), rho0s=(3, 40),
                          tag_set=(0, 1, 2), mix=(1, 1, 1), repair_frac=0.2)
    dr, ckpt = _streamed(case, torch, pinned=False)
    check_full(dr, ckpt)
    dr, ckpt = _streamed(case, torch, stream=torch.cuda.Stream())
    check_full(dr, ckpt)


def test_streamed_repeat_reuses_plan(torch):
    case = wl.make_case("tiny")
    dr, ckpt = _streamed(case, torch)
    hp = torch.from_numpy(ckpt[0]).pin_memory()
    hs = torch.from_numpy(ckpt[1].view(np.int16)).pin_memory()
    for _ in range(3):
        dr.prefill()
        pb.restore_from_host_tensors(dr.plan, hp, hs, dr.payload, dr.scales, dr.k_cache, dr.v_cache)
    torch.cuda.synchronize()
    check_full(dr, ckpt)


def test_streamed_argument_errors(torch):
    case = wl.make_case("tiny")
    dr, ckpt = _streamed(case, torch)
    hp = torch.from_numpy(ckpt[0]).pin_memory()
    hs = torch.from_numpy(ckpt[1].view(np.int16)).pin_memory()
    nb = lambda t: t.numel() * t.element_size()
    good = (hp.data_ptr(), nb(hp), hs.data_ptr(), nb(hs), dr.payload.data_ptr(), nb(dr.payload),
            dr.scales.data_ptr(), nb(dr.scales), dr.k_cache.data_ptr(), dr.v_cache.data_ptr(), nb(dr.k_cache), 0)
    bad = [
        (0,) + good[1:],                      # no host payload
        good[:1] + (nb(hp) - 16,) + good[2:],  # host payload too small
        good[:2] + (0,) + good[3:],           # no host scales
        good[:3] + (nb(hs) - 2,) + good[4:],  # host scales too small
        good[:4] + (0,) + good[5:],           # no device payload
        good[:8] + (dr.k_cache.data_ptr(), dr.k_cache.data_ptr()) + good[10:],  # K and V alias
    ]
    for args in bad:
        assert pb.pkv_restore_from_host_status(dr.plan, *args) == pb.PKV_ERR_INVALID_ARGUMENT, args
    ck = pb.pkv_checkpoint_plan(case.src_shape, case.requests)
    assert pb.load().pkv_restore_from_host(ck.handle, *good) == pb.PKV_ERR_INVALID_ARGUMENT
    torch.cuda.synchronize()
    check_full(dr, ckpt)  # nothing above wrote anything


def test_zero_copy_restore_from_pinned_memory(torch):
    """pkv_restore reading the checkpoint straight from pinned host memory:
    the same caches as the oracle and as a device-resident restore."""
    case = wl.make_custom(12, L=3, H=4, D=128, B=32, P=16, n_tokens=(300, 95), deltas=(-700, 3), rho0s=(900, 4),
                          tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2, out_dtype=wl.OUT_BF16,
                          outlier_pairs=1)
    dr, ckpt = _streamed(case, torch)  # device-resident reference via the streamed path
    k_ref, v_ref = dr.host_caches()
    hp = torch.from_numpy(ckpt[0]).pin_memory()
    hs = torch.from_numpy(ckpt[1].view(np.int16)).pin_memory()
    dr.prefill()
    pb.restore_tensors(dr.plan, hp, hs, dr.k_cache, dr.v_cache)
    torch.cuda.synchronize()
    k, v = dr.host_caches()
    assert np.array_equal(k, k_ref) and np.array_equal(v, v_ref)
    check_full(dr, ckpt)


def test_pageable_and_foreign_inputs_rejected(torch):
    """Inputs the kernel could not read are refused before any launch."""
    case = wl.make_case("tiny")
    dr, ckpt = _streamed(case, torch)
    before = dr.host_caches()
    nb = lambda t: t.numel() * t.element_size()
    pageable_p = np.ascontiguousarray(ckpt[0])
    pageable_s = np.ascontiguousarray(ckpt[1])
    args = (pageable_p.ctypes.data, pageable_p.nbytes, dr.scales.data_ptr(), nb(dr.scales), dr.k_cache.data_ptr(),
            dr.v_cache.data_ptr(), nb(dr.k_cache), 0)
    assert pb.pkv_restore_status(dr.plan, *args) == pb.PKV_ERR_INVALID_ARGUMENT
    args = (dr.payload.data_ptr(), nb(dr.payload), pageable_s.ctypes.data, pageable_s.nbytes, dr.k_cache.data_ptr(),
            dr.v_cache.data_ptr(), nb(dr.k_cache), 0)
    assert pb.pkv_restore_status(dr.plan, *args) == pb.PKV_ERR_INVALID_ARGUMENT
    # caches must be device memory
    hk = torch.empty(dr.k_cache.numel(), dtype=torch.int16, pin_memory=True)
    args = (dr.payload.data_ptr(), nb(dr.payload), dr.scales.data_ptr(), nb(dr.scales), hk.data_ptr(),
            dr.v_cache.data_ptr(), nb(dr.k_cache), 0)
    assert pb.pkv_restore_status(dr.plan, *args) == pb.PKV_ERR_INVALID_ARGUMENT
    torch.cuda.synchronize()
    after = dr.host_caches()
    assert np.array_equal(before[0], after[0]) and np.array_equal(before[1], after[1])
