"""GPU parity of the HIP restore against the CPU oracle, through the C ABI."""
import copy
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

from parity import (check_both_orders, check_device_checkpoint, check_full, check_sampled, log, oracle_checkpoint,
                    oracle_layer_checkpoint, poison_device, restore_order, restore_small)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    pb.load()
    return _t


@pytest.mark.parametrize("order", ["early", "late"])
@pytest.mark.parametrize("name", ["tiny", "llama8b_1l"])
def test_named_small_full(name, order, torch):
    log(f"[gpu] {name}, {order} order: full-cache parity")
    dr, ckpt = restore_small(wl.make_case(name), order=order)
    st = check_full(dr, ckpt)
    log(f"  {st}")
    assert st.bit_exact_fraction > 0.9999


def _paired(case):
    import dataclasses
    case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    return case


@pytest.mark.parametrize("order", ["early", "late"])
@pytest.mark.parametrize("name", ["tiny", "llama8b_1l"])
def test_named_small_full_paired_pages(name, order, torch):
    log(f"[gpu] {name}, paired K/V pages, {order} order: full-cache parity")
    dr, ckpt = restore_small(_paired(wl.make_case(name)), order=order)
    st = check_full(dr, ckpt)
    log(f"  {st}")
    assert st.bit_exact_fraction > 0.9999


def test_paired_pages_argument_errors(torch):
    """A paired cache is one buffer with v_cache = k_cache + P*H*D elements;
    any other placement, or a buffer smaller than both halves of every
    layer, is refused before any write."""
    from paper_2609_26219_amd.device import DeviceRestore
    case = _paired(wl.make_case("tiny"))
    ckpt = oracle_checkpoint(case)
    dr = DeviceRestore(case, checkpoint=ckpt)
    s_ = case.shape
    nb = lambda t: t.numel() * t.element_size()
    half = s_.page_size * s_.row_elems * 2
    p, sc, k = dr.payload, dr.scales, dr.k_cache
    total = pb.cache_nbytes(dr.k_cache, dr.v_cache)
    assert total == 2 * s_.cache_elems * 2
    good = (p.data_ptr(), nb(p), sc.data_ptr(), nb(sc), k.data_ptr(), k.data_ptr() + half, total, 0)
    assert pb.pkv_restore_status(dr.plan, *good) == pb.PKV_OK
    torch.cuda.synchronize()
    bad = [
        good[:5] + (k.data_ptr() + half + 16,) + good[6:],   # V not right after the page's K slots
        good[:5] + (k.data_ptr(),) + good[6:],               # V on top of K
        good[:6] + (total // 2, 0),                          # one half's size
        good[:4] + (p.data_ptr(), p.data_ptr() + half) + good[6:],  # cache over the payload
    ]
    for args in bad:
        assert pb.pkv_restore_status(dr.plan, *args) == pb.PKV_ERR_INVALID_ARGUMENT, args
    check_full(dr, ckpt)


def test_tiny_k4v4_reading(torch):
    check_both_orders(wl.make_case("tiny", int4_tag=wl.TAG_K4V4))


PROPERTY_CASES = [
    # (B, P, D, H, n_tokens, deltas, rho0s, tag_set, repair_frac, out)
    (8, 8, 64, 2, (61,), (3,), (0,), (0, 1, 2, 3), 0.2, wl.OUT_FP16),
    (16, 16, 128, 1, (200,), (-77,), (16,), (2,), 0.0, wl.OUT_BF16),
    (32, 16, 128, 4, (150,), (0,), (5,), (0, 1, 2), 0.3, wl.OUT_BF16),
    (64, 32, 64, 2, (130,), (9999,), (31,), (1, 3), 0.1, wl.OUT_FP16),
    (32, 8, 64, 8, (97, 33, 256), (1, -1, 8192), (3, 64, 1000), (0, 1, 2, 3), 0.25, wl.OUT_BF16),
    (16, 32, 256, 2, (45,), (-8192,), (17,), (0, 2), 0.0, wl.OUT_FP16),
    (32, 16, 128, 3, (70,), (12,), (9,), (0, 1, 2, 3), 0.0, wl.OUT_BF16),  # H*D/16 = 24 (idle lanes)
    (4, 16, 128, 8, (23,), (5,), (2,), (0, 1, 2, 3), 0.2, wl.OUT_FP16),
    # tensor-parallel shards of the 8B shape: one-wave workgroups, two and four tokens per thread
    (32, 16, 128, 1, (300, 77), (-1500, 0), (1507, 5), (0, 1, 2, 3), 0.15, wl.OUT_BF16),
    (32, 16, 128, 2, (190,), (-1500,), (1509,), (0, 1, 2, 3), 0.15, wl.OUT_BF16),
]


@pytest.mark.parametrize("layout", [wl.KV_SEPARATE, wl.KV_PAIRED], ids=["separate", "paired"])
@pytest.mark.parametrize("params", PROPERTY_CASES, ids=[f"case{i}" for i in range(len(PROPERTY_CASES))])
def test_property_cases(params, layout, torch):
    B, P, D, H, n, deltas, rho0s, tags, rep, out = params
    case = wl.make_custom(hash(params) & 0xFFFF, L=2, H=H, D=D, B=B, P=P, n_tokens=n, deltas=deltas, rho0s=rho0s,
                          tag_set=tags, mix=[1.0] * len(tags), repair_frac=rep, out_dtype=out, outlier_pairs=1)
    if layout == wl.KV_PAIRED:
        _paired(case)
    log(f"[gpu] property case {params} layout {layout}")
    check_both_orders(case)


@pytest.mark.parametrize("name", ["qwen3_32b_1l", "glm4_9b_1l", "llama33_70b_1l"])
def test_model_family_rope(name, torch):
    """The paper's model families with their own RoPE: Qwen3 (rotate-half,
    theta 1e6), GLM-4 (interleaved pairs on half the head), Llama-3.3
    (rotate-half with scaled frequencies)."""
    log(f"[gpu] {name}: full-cache parity with the model's RoPE")
    for order in ("early", "late"):
        st = check_full(*restore_small(wl.make_case(name), order=order))
        log(f"  {order} order: {st}")
        assert st.bit_exact_fraction > 0.9999


ROPE_CASES = [
    # (D, rotary_dim, style, scaled frequencies, tag set, out dtype)
    (128, 64, wl.ROPE_HALF, False, (0, 1, 2, 3), wl.OUT_BF16),
    (128, 32, wl.ROPE_INTERLEAVED, True, (0, 2), wl.OUT_FP16),
    (64, 64, wl.ROPE_INTERLEAVED, False, (1, 3), wl.OUT_BF16),
    (256, 96, wl.ROPE_HALF, True, (0, 1, 2), wl.OUT_FP16),
    (48, 16, wl.ROPE_INTERLEAVED, False, (0, 1, 2, 3), wl.OUT_BF16),
]


@pytest.mark.parametrize("params", ROPE_CASES, ids=[f"rope{i}" for i in range(len(ROPE_CASES))])
def test_rope_variant_cases(params, torch):
    import dataclasses
    D, R, style, scaled, tags, out = params
    case = wl.make_custom(50 + len(tags), L=2, H=3, D=D, B=16, P=16, n_tokens=(70, 33), deltas=(-2049, 5),
                          rho0s=(2100, 9), tag_set=tags, mix=[1.0] * len(tags), repair_frac=0.2, out_dtype=out,
                          outlier_pairs=1)
    case.shape = dataclasses.replace(case.shape, rope_style=style, rotary_dim=0 if R == D else R,
                                     inv_freq=wl.llama3_inv_freq(5e5, R) if scaled else None)
    log(f"[gpu] rope variant {params}")
    check_both_orders(case)


def test_all_repair_writes_nothing(torch):
    case = wl.make_custom(21, L=2, n_tokens=(64, 20), deltas=(4, 2), repair_all=True)
    dr, _ = restore_small(case)
    assert dr.info["num_units"] == 0
    k, v = dr.host_caches()
    assert np.array_equal(k, case.host_prefill(0)) and np.array_equal(v, case.host_prefill(1))


def test_fp16_tag_zero_shift_is_bit_copy(torch):
    case = wl.make_custom(22, H=8, D=128, B=32, P=16, n_tokens=(300,), deltas=(0,), rho0s=(13,),
                          tag_set=(wl.TAG_FP16,), mix=(1.0,), repair_frac=0.1, out_dtype=wl.OUT_FP16)
    for order in ("early", "late"):
        st = check_full(*restore_small(case, order=order))
        assert st.n_bit_exact == st.n


def test_restore_is_repeatable_and_plan_reusable(torch):
    from paper_2609_26219_amd.device import DeviceRestore
    case = wl.make_case("tiny")
    ckpt = oracle_checkpoint(case)
    dr = DeviceRestore(case, checkpoint=ckpt)
    dr.run()
    dr.run()
    torch.cuda.synchronize()
    k1, v1 = dr.host_caches()
    # same plan, a second pair of caches
    k2 = torch.zeros_like(dr.k_cache)
    v2 = torch.zeros_like(dr.v_cache)
    pb.restore_tensors(dr.plan, dr.payload, dr.scales, k2, v2)
    torch.cuda.synchronize()
    written = oracle.written_slots(case.shape, case.requests)
    s = case.shape
    a = k2.cpu().numpy().view(np.uint16).reshape(s.num_layers, s.pool_slots, -1)
    b = k1.reshape(a.shape)
    assert np.array_equal(a[:, written], b[:, written])
    assert (a[:, ~written] == 0).all()
    check_full(dr, ckpt)


def test_restore_argument_errors(torch):
    from paper_2609_26219_amd.device import DeviceRestore
    case = wl.make_case("tiny")
    ckpt = oracle_checkpoint(case)
    dr = DeviceRestore(case, checkpoint=ckpt)
    nb = lambda t: t.numel() * t.element_size()
    p, s, k, v = dr.payload, dr.scales, dr.k_cache, dr.v_cache
    good = (p.data_ptr(), nb(p), s.data_ptr(), nb(s), k.data_ptr(), v.data_ptr(), nb(k), 0)
    assert pb.pkv_restore_status(dr.plan, *good) == pb.PKV_OK
    torch.cuda.synchronize()
    bad = [
        (p.data_ptr(), nb(p) - 16) + good[2:],                     # payload too small
        good[:3] + (nb(s) - 2,) + good[4:],                        # scales too small
        good[:6] + (nb(k) - 2, 0),                                 # cache too small
        good[:4] + (k.data_ptr(), k.data_ptr()) + good[6:],        # K and V alias
        (p.data_ptr() + 1,) + good[1:],                            # misaligned payload
        good[:4] + (k.data_ptr() + 2,) + good[5:],                 # misaligned cache
        good[:4] + (p.data_ptr(),) + good[5:],                     # cache overlaps payload
        (0,) + good[1:],                                           # null payload
    ]
    for args in bad:
        assert pb.pkv_restore_status(dr.plan, *args) == pb.PKV_ERR_INVALID_ARGUMENT, args
    check_full(dr, ckpt)  # nothing above wrote anything


def test_streams(torch):
    from paper_2609_26219_amd.device import DeviceRestore
    case = wl.make_case("llama8b_1l")
    ckpt = oracle_checkpoint(case)
    dr = DeviceRestore(case, checkpoint=ckpt)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        dr.run()
    s.synchronize()
    check_full(dr, ckpt)


# ---------------------------------------------------------------------------
# Full-size workloads: the checkpoint is written on the GPU by
# pkv_quantize_gather from the drawn old caches (layer by layer), compared
# bit for bit with the oracle's on the sampled (request, layer) pairs, then
# repair blocks are poisoned and the restore is compared with the oracle's
# restore of the oracle's checkpoint on those pairs.
# ---------------------------------------------------------------------------

def _full_size(case, samples, torch, order="auto"):
    from paper_2609_26219_amd.device import DeviceRestore
    dr = DeviceRestore(case)
    refs = {key: oracle_layer_checkpoint(case, *key) for key in samples}
    check_device_checkpoint(case, dr.payload, dr.scales, refs)
    poison_device(case, dr.payload, dr.scales)
    with restore_order(order):
        dr.run()
        torch.cuda.synchronize()
    return check_sampled(dr, refs)


def test_llama8b_32l_full_size(torch):
    log("[gpu] llama8b_32l: full-size checkpoint + restore, 3 sampled layers + untouched check")
    st = _full_size(wl.make_case("llama8b_32l"), [(0, 0), (0, 17), (0, 31)], torch)
    log(f"  {st}")


def test_llama8b_32l_full_size_late_order(torch):
    """The late start order (chosen by size for launches that fit on the
    device at once) forced on the full 32-layer launch."""
    log("[gpu] llama8b_32l, late order forced: full-size checkpoint + restore, 2 sampled layers + untouched check")
    st = _full_size(_paired(wl.make_case("llama8b_32l")), [(0, 1), (0, 29)], torch, order="late")
    log(f"  {st}")


def test_llama8b_32l_full_size_paired_pages(torch):
    log("[gpu] llama8b_32l, paired K/V pages: full-size checkpoint + restore, 2 sampled layers + untouched check")
    st = _full_size(_paired(wl.make_case("llama8b_32l")), [(0, 3), (0, 30)], torch)
    log(f"  {st}")


@pytest.mark.parametrize("heads", [1, 2])
def test_tensor_parallel_share_full_size(heads, torch):
    """One GPU's share of the 8B-shaped workload under tensor parallelism over
    KV heads (1 or 2 heads per GPU: one-wave workgroups), at full length."""
    log(f"[gpu] 8B-shaped share with {heads} KV head(s): full-size checkpoint + restore, 2 sampled layers")
    case = wl.make_custom(41, L=32, H=heads, D=128, B=32, P=16, n_tokens=(32768,), deltas=(-1500,), rho0s=(5007,),
                          mix=(0.7, 0.2, 0.1), tag_set=(wl.TAG_K8V4, wl.TAG_K8V8, wl.TAG_FP16), repair_frac=0.15,
                          out_dtype=wl.OUT_BF16, theta=5e5, outlier_pairs=1)
    st = _full_size(_paired(case), [(0, 0), (0, 31)], torch)
    log(f"  {st}")


def test_llama70b_full_size(torch):
    log("[gpu] llama70b: full-size checkpoint + restore, 2 sampled layers + untouched check")
    _full_size(wl.make_case("llama70b", distinct_layers=2), [(0, 1), (0, 78)], torch)


def test_batched16_full_size(torch):
    log("[gpu] batched16: 16 requests on a 2^20-slot pool, 4 sampled (request, layer) + untouched check")
    _full_size(wl.make_case("batched16", distinct_layers=1), [(0, 0), (5, 13), (11, 31), (15, 7)], torch)


def test_plan_payload_bytes_per_request(torch):
    """pkv_plan_payload_bytes: each request's checkpoint size, for restore and
    checkpoint plans alike, equal to the oracle's layout walk; requests
    outside the plan are argument errors."""
    import ctypes

    case = wl.make_custom(21, L=2, H=3, D=32, B=8, P=4, n_tokens=(37, 5, 16), deltas=(3, 0, -2),
                          rho0s=(9, 4, 30), tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1))
    plans = (pb.pkv_restore_plan(case.shape, case.requests), pb.pkv_checkpoint_plan(case.src_shape, case.requests))
    for plan in plans:
        for ri, req in enumerate(case.requests):
            assert pb.pkv_plan_payload_bytes(plan, ri) == oracle.request_payload_bytes(case.shape, req)
        out = ctypes.c_uint64(7)
        for bad in (-1, len(case.requests)):
            assert pb.pkv_plan_payload_bytes_status(plan.handle, bad, ctypes.byref(out)) == pb.PKV_ERR_INVALID_ARGUMENT
        assert pb.pkv_plan_payload_bytes_status(plan.handle, 0, None) == pb.PKV_ERR_INVALID_ARGUMENT
        assert out.value == 7
