"""GPU parity of the checkpoint write (quantize-and-gather) against the CPU
oracle, bit for bit, and of the full write -> restore cycle."""
import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

from parity import Stats, check_checkpoint_write, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    pb.load()
    return _t


@pytest.mark.parametrize("name,int4", [("tiny", wl.TAG_K8V4), ("tiny", wl.TAG_K4V4), ("llama8b_1l", wl.TAG_K8V4)])
def test_checkpoint_bit_exact_named(name, int4, torch):
    log(f"[gpu] checkpoint write {name}")
    check_checkpoint_write(wl.make_case(name, int4_tag=int4), torch)


@pytest.mark.parametrize("params", [
    dict(L=2, H=2, D=64, B=16, P=16, n_tokens=(100, 40), deltas=(5, -3), rho0s=(20, 7), out_dtype=wl.OUT_BF16),
    dict(L=1, H=4, D=128, B=64, P=32, n_tokens=(130,), deltas=(9,), rho0s=(31,), out_dtype=wl.OUT_BF16),
    dict(L=2, H=3, D=128, B=32, P=8, n_tokens=(70, 1, 33), deltas=(0, 2, -4), rho0s=(5, 9, 60), out_dtype=wl.OUT_FP16),
    dict(L=1, H=8, D=256, B=8, P=16, n_tokens=(41,), deltas=(3,), rho0s=(5,), out_dtype=wl.OUT_BF16),
    dict(L=1, H=2, D=512, B=64, P=16, n_tokens=(150,), deltas=(2,), rho0s=(9,), out_dtype=wl.OUT_BF16),
    dict(L=2, H=20, D=16, B=8, P=8, n_tokens=(21, 50), deltas=(1, 0), rho0s=(3, 8), out_dtype=wl.OUT_FP16),
    dict(L=1, H=3, D=48, B=16, P=16, n_tokens=(37,), deltas=(2,), rho0s=(5,), out_dtype=wl.OUT_FP16),
    # blocks spanning more than three pages: the general kernel with 4 and 2 loads per lane
    dict(L=1, H=4, D=64, B=32, P=8, n_tokens=(77,), deltas=(1,), rho0s=(6,), out_dtype=wl.OUT_BF16),
    dict(L=2, H=2, D=32, B=16, P=4, n_tokens=(45, 16), deltas=(0, 3), rho0s=(2, 9), out_dtype=wl.OUT_FP16),
    # 70B-shaped blocks (64 tokens, 32-token pages): 16 loads per lane in the tile kernel with 8 waves;
    # with 12 heads the workgroup is too large for it and the general kernel takes 16 loads in one pass
    dict(L=2, H=8, D=128, B=64, P=32, n_tokens=(150, 64), deltas=(4096, 0), rho0s=(31, 96), out_dtype=wl.OUT_BF16),
    dict(L=1, H=12, D=128, B=64, P=32, n_tokens=(130,), deltas=(-7,), rho0s=(17,), out_dtype=wl.OUT_BF16),
], ids=["bf16_two_requests", "b64_bf16", "h3_three_requests_fp16", "d256_b8", "d512_b64_streamed_twice",
        "h20_d16", "d48_idle_lanes", "general_nl4", "general_nl2", "h8_b64_p32_tile16", "h12_b64_general16"])
def test_checkpoint_bit_exact_custom(params, torch):
    case = wl.make_custom(11, tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), outlier_pairs=1, **params)
    check_checkpoint_write(case, torch)


@pytest.mark.parametrize("params", [
    dict(L=2, H=2, D=64, B=16, P=16, n_tokens=(100, 40), deltas=(5, -3), rho0s=(20, 7), out_dtype=wl.OUT_BF16),
    dict(L=2, H=8, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,), out_dtype=wl.OUT_BF16),
    dict(L=1, H=4, D=64, B=32, P=8, n_tokens=(77,), deltas=(1,), rho0s=(6,), out_dtype=wl.OUT_FP16),
    dict(L=1, H=8, D=128, B=64, P=32, n_tokens=(150,), deltas=(4096,), rho0s=(31,), out_dtype=wl.OUT_BF16),
], ids=["two_requests", "h8_d128", "general_kernel", "h8_b64_p32_tile16"])
def test_checkpoint_bit_exact_paired_pages(params, torch):
    import dataclasses
    case = wl.make_custom(12, tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), outlier_pairs=1, **params)
    case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    check_checkpoint_write(case, torch)


@pytest.mark.parametrize("out", [wl.OUT_FP16, wl.OUT_BF16])
def test_checkpoint_exact_and_near_ties(out, torch):
    """Rows on a grid of half-integer multiples of the scale (exact ties, which
    round to even) and one cache ulp either side of them: the codes must
    equal the oracle's correctly rounded double-precision ones."""
    case = wl.make_custom(31 + out, L=2, H=4, D=64, B=16, P=16, n_tokens=(90, 37), deltas=(3, -1), rho0s=(5, 40),
                          tag_set=(1, 2, 3), mix=(1, 1, 1), out_dtype=out)
    s = case.src_shape
    kc, vc = case.host_old_caches()
    rng = np.random.default_rng(5)
    for cache in (kc, vc):
        for layer in range(s.num_layers):
            flat = cache[layer].reshape(-1, s.num_kv_heads, s.head_dim)
            for ri in range(len(case.requests)):
                slots = case.suffix_bits(ri, layer)[0]
                step = 2.0 ** -int(rng.integers(2, 6))  # a binary16 scale
                grid = (rng.integers(0, 15, size=(len(slots), s.num_kv_heads, s.head_dim)) + 0.5) * step
                ulp = rng.choice([-1, 0, 1], size=grid.shape)
                bits = wl.to_cache_bits(grid, out).astype(np.int32) + ulp
                bits[:, :, 0] = wl.to_cache_bits(np.zeros(1), out)[0]   # min 0: zero 0
                bits[:, :, 1] = wl.to_cache_bits(np.full(1, 15 * step), out)[0]  # max 15 * step
                flat[slots] = bits.astype(np.uint16)
    check_checkpoint_write(case, torch, (kc, vc))


def test_write_then_restore_cycle(torch):
    """Checkpoint written on the GPU, restored on the GPU into the new pages
    with the key phase shift, compared element by element with the oracle's
    restore of the oracle's own checkpoint."""
    case = wl.make_case("llama8b_1l")
    payload, scales, ref_p, ref_s = check_checkpoint_write(case, torch)
    s = case.shape
    dpay = torch.from_numpy(payload).cuda()
    dsc = torch.from_numpy(scales.view(np.int16)).cuda()
    k = torch.zeros((s.num_layers, s.pool_pages, s.page_size, s.num_kv_heads, s.head_dim), dtype=torch.int16,
                    device="cuda")
    v = torch.zeros_like(k)
    plan = pb.pkv_restore_plan(s, case.requests)
    pb.restore_tensors(plan, dpay, dsc, k, v)
    torch.cuda.synchronize()
    kh = k.cpu().numpy().view(np.uint16).reshape(s.num_layers, s.pool_slots, s.num_kv_heads, s.head_dim)
    vh = v.cpu().numpy().view(np.uint16).reshape(kh.shape)
    st = Stats()
    req = case.requests[0]
    layout = oracle.block_layout(req.tags, s.block_tokens, s.num_kv_heads, s.head_dim)
    for b in oracle.reused_blocks(req):
        slots, kk, vv = oracle.restore_block(ref_p, ref_s, s, req, 0, b, layout)  # oracle reads its own checkpoint
        st.add(kh[0, slots], kk, s.out_dtype, int(req.delta))
        st.add(vh[0, slots], vv, s.out_dtype)
    st.assert_ok(s.out_dtype)
    log(f"  cycle: {st}")


def test_plan_kinds_are_checked(torch):
    case = wl.make_case("tiny")
    ck = pb.pkv_checkpoint_plan(case.src_shape, case.requests)
    rs = pb.pkv_restore_plan(case.shape, case.requests)
    buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    p = buf.data_ptr()
    assert pb.pkv_restore_status(ck, p, 1 << 16, p + (1 << 16), 1 << 16, p + (2 << 16), p + (3 << 16), 1 << 16,
                                 0) == pb.PKV_ERR_INVALID_ARGUMENT
    assert pb.load().pkv_quantize_gather(rs.handle, p, p, 0, p, 0, p, 0, None) == pb.PKV_ERR_INVALID_ARGUMENT


def _old_device_caches(case, torch):
    from paper_2609_26219_amd.device import alloc_caches

    kc, vc = case.host_old_caches()
    dk, dv = alloc_caches(case.src_shape, "cuda")
    dk.copy_(torch.from_numpy(kc.view(np.int16)))
    dv.copy_(torch.from_numpy(vc.view(np.int16)))
    return kc, vc, dk, dv


def test_checkpoint_buffers_checked_before_launch(torch):
    """Pageable host memory for the caches, the payload or the scales is
    refused before any launch, and nothing is written anywhere."""
    from parity import FILL

    case = wl.make_case("tiny")
    s = case.src_shape
    assert s.kv_layout == wl.KV_SEPARATE
    kc, vc, dk, dv = _old_device_caches(case, torch)
    payload = torch.full((case.payload_nbytes,), FILL, dtype=torch.uint8, device="cuda")
    scales = torch.full((case.scale_elems,), 0x5A5A, dtype=torch.int16, device="cuda")
    host_p = np.full(case.payload_nbytes, FILL, np.uint8)
    host_s = np.full(case.scale_elems, 0x5A5A, np.uint16)
    host_k, host_v = np.ascontiguousarray(kc), np.ascontiguousarray(vc)
    plan = pb.pkv_checkpoint_plan(s, case.requests)
    q = pb.load().pkv_quantize_gather
    nb = lambda t: t.numel() * t.element_size()
    cb = pb.cache_nbytes(dk, dv)
    P, S = payload.data_ptr(), scales.data_ptr()
    bad = [
        (dk.data_ptr(), dv.data_ptr(), cb, host_p.ctypes.data, host_p.nbytes, S, nb(scales)),
        (dk.data_ptr(), dv.data_ptr(), cb, P, nb(payload), host_s.ctypes.data, host_s.nbytes),
        (host_k.ctypes.data, dv.data_ptr(), host_k.nbytes, P, nb(payload), S, nb(scales)),
        (dk.data_ptr(), host_v.ctypes.data, host_v.nbytes, P, nb(payload), S, nb(scales)),
    ]
    for args in bad:
        assert q(plan.handle, *args, None) == pb.PKV_ERR_INVALID_ARGUMENT
    torch.cuda.synchronize()
    assert (host_p == FILL).all() and (host_s == 0x5A5A).all()
    assert (payload.cpu().numpy() == FILL).all() and (scales.cpu().numpy() == 0x5A5A).all()
    assert np.array_equal(host_k, kc) and np.array_equal(host_v, vc)
    # the same call on device buffers writes the oracle's checkpoint
    assert q(plan.handle, dk.data_ptr(), dv.data_ptr(), cb, P, nb(payload), S, nb(scales), None) == pb.PKV_OK
    torch.cuda.synchronize()
    assert not (payload.cpu().numpy() == FILL).all()


@pytest.mark.parametrize("name", ["tiny", "llama8b_1l"])
def test_checkpoint_into_pinned_host_memory(name, torch):
    """The checkpoint written straight into pinned host memory (the kernel
    stores over the host link) is the oracle's, bit for bit."""
    from oracle import quantize as oq
    from parity import FILL

    case = wl.make_case(name)
    log(f"[gpu] checkpoint write into pinned host memory: {name}")
    kc, vc, dk, dv = _old_device_caches(case, torch)
    hp = torch.full((case.payload_nbytes,), FILL, dtype=torch.uint8, pin_memory=True)
    hs = torch.full((case.scale_elems,), 0x5A5A, dtype=torch.int16, pin_memory=True)
    plan = pb.pkv_checkpoint_plan(case.src_shape, case.requests)
    pb.quantize_gather_tensors(plan, dk, dv, hp, hs)
    torch.cuda.synchronize()
    ref_p, ref_s = oq.quantize_gather(case.src_shape, case.requests, kc, vc, case.payload_nbytes, case.scale_elems)
    assert pb.pkv_plan_payload_bytes(plan, 0) == oracle.request_payload_bytes(case.shape, case.requests[0])
    assert np.array_equal(hp.numpy(), ref_p)
    assert np.array_equal(hs.numpy().view(np.uint16), ref_s)
