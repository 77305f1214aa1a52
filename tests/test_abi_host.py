"""Host-side tests of the C ABI: runs without a GPU.

The library must load and export every function ``include/pkv.h`` declares;
``pkv_payload_size`` must agree with the oracle's and the generator's own
layout walks; every argument error of ``pkv_restore_plan`` must be reported
before any HIP call (so here, on a machine without a GPU)."""
import copy
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pkv.h")


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return False


VALID = pb.PKV_OK if _gpu_present() else pb.PKV_ERR_DEVICE


@pytest.fixture(scope="module")
def lib():
    return pb.load()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pkv_[a-z_]+)\s*\(", text)))


def test_header_declares_what_binding_lists():
    assert _declared_functions() == sorted(pb.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", pb.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (pkv_\w+)", out))
    for name in _declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_plan_payload_bytes_rejects_null(lib):
    import ctypes
    out = ctypes.c_uint64(5)
    assert pb.pkv_plan_payload_bytes_status(None, 0, ctypes.byref(out)) == pb.PKV_ERR_INVALID_ARGUMENT
    assert out.value == 5


def test_status_strings(lib):
    for code in range(-7, 1):
        assert pb.pkv_status_string(code) != "unknown status"
    assert pb.pkv_status_string(5) == "unknown status"


@pytest.mark.parametrize("name", ["tiny", "llama8b_1l"])
def test_payload_size_three_ways(name):
    case = wl.make_case(name)
    for tag_map in (None, wl.TAG_K4V4):
        r = case.requests[0]
        if tag_map is not None:
            r = copy.copy(r)
            r.tags = np.where(r.tags == wl.TAG_K8V4, tag_map, r.tags).astype(np.uint8)
        lib_bytes, lib_scales = pb.pkv_payload_size(case.shape, r)
        gen_bytes, gen_scales = wl.encoded_request_nbytes(case.shape, r)
        assert lib_bytes == gen_bytes == oracle.request_payload_bytes(case.shape, r)
        assert lib_scales == gen_scales


# ---------------------------------------------------------------------------
# Plan validation
# ---------------------------------------------------------------------------

def _base():
    case = wl.make_custom(3, L=2, H=2, D=64, B=16, P=16, n_tokens=(100, 40), deltas=(5, -3), rho0s=(20, 7),
                          repair_frac=0.0)
    return case.shape, [copy.copy(r) for r in case.requests]


def _status(shape, reqs):
    return pb.pkv_restore_plan_status(shape, reqs)


def test_valid_plan_passes_validation():
    shape, reqs = _base()
    assert _status(shape, reqs) == VALID
    assert _status(shape, []) == VALID


@pytest.mark.parametrize("field,value", [
    ("head_dim", 72), ("head_dim", 8), ("head_dim", 1024), ("num_kv_heads", 0), ("num_layers", 0),
    ("page_size", 12), ("page_size", 0), ("pool_pages", 0), ("rope_theta", 0.0), ("rope_theta", float("nan")),
    ("out_dtype", 2), ("block_tokens", 0), ("block_tokens", 2048), ("num_kv_heads", 65),
    ("kv_layout", 2), ("kv_layout", -1),
])
def test_bad_model(field, value):
    shape, reqs = _base()
    import dataclasses
    shape = dataclasses.replace(shape, **{field: value})
    assert _status(shape, reqs) == pb.PKV_ERR_INVALID_ARGUMENT


def test_page_of_one_cache_at_most_2gib():
    """The kernels address inside a page with 32-bit offsets: a page of
    P * H * D * 2 bytes above 2 GiB is refused, exactly 2 GiB is accepted."""
    import dataclasses
    shape, reqs = _base()
    big = dataclasses.replace(shape, page_size=1 << 20, num_kv_heads=8, head_dim=128, pool_pages=1)
    assert _status(big, []) == VALID  # 2^20 * 1024 * 2 = 2 GiB
    assert _status(dataclasses.replace(big, num_kv_heads=16), []) == pb.PKV_ERR_INVALID_ARGUMENT


def test_tile_alignment_rule():
    import dataclasses
    shape, reqs = _base()
    # B*H*D % 32 != 0 -> rejected (B=1, H=1, D=16)
    shape = dataclasses.replace(shape, block_tokens=1, num_kv_heads=1, head_dim=16)
    for r in reqs:
        nb = wl.num_blocks(r.suffix_tokens, 1)
        r.tags = np.zeros(nb, np.uint8)
        r.repair = np.zeros(nb, np.uint8)
    assert _status(shape, reqs) == pb.PKV_ERR_INVALID_ARGUMENT


def test_bad_tag():
    shape, reqs = _base()
    reqs[1].tags = reqs[1].tags.copy()
    reqs[1].tags[1] = 4
    assert _status(shape, reqs) == pb.PKV_ERR_BAD_TAG


def test_bad_tag_in_repair_block_still_rejected():
    shape, reqs = _base()
    reqs[0].tags = reqs[0].tags.copy()
    reqs[0].repair = reqs[0].repair.copy()
    reqs[0].tags[2] = 9
    reqs[0].repair[2] = 1
    assert _status(shape, reqs) == pb.PKV_ERR_BAD_TAG


@pytest.mark.parametrize("field,value", [
    ("reserved", 1), ("payload_offset", 8), ("scale_offset", 2), ("suffix_tokens", -1), ("dst_row0", -5),
])
def test_bad_request_fields(field, value):
    shape, reqs = _base()
    setattr(reqs[0], field, value)
    assert _status(shape, reqs) == pb.PKV_ERR_INVALID_ARGUMENT


def _first_f_page(shape, req):
    b = int(np.nonzero(req.repair == 0)[0][0])
    return (req.dst_row0 + b * shape.block_tokens) // shape.page_size


def test_page_out_of_range():
    shape, reqs = _base()
    reqs[0].page_table = reqs[0].page_table.copy()
    reqs[0].page_table[_first_f_page(shape, reqs[0])] = shape.pool_pages
    assert _status(shape, reqs) == pb.PKV_ERR_PAGE_OUT_OF_RANGE
    reqs[0].page_table[_first_f_page(shape, reqs[0])] = -2
    assert _status(shape, reqs) == pb.PKV_ERR_PAGE_OUT_OF_RANGE


def test_rows_past_page_table():
    shape, reqs = _base()
    reqs[1].page_table = reqs[1].page_table[:1].copy()
    assert _status(shape, reqs) == pb.PKV_ERR_PAGE_OUT_OF_RANGE


def test_page_unmapped():
    shape, reqs = _base()
    reqs[0].page_table = reqs[0].page_table.copy()
    last_row = reqs[0].dst_row0 + reqs[0].suffix_tokens - 1
    reqs[0].page_table[last_row // shape.page_size] = -1
    assert _status(shape, reqs) == pb.PKV_ERR_PAGE_UNMAPPED


def test_unmapped_pages_of_repair_blocks_and_prefix_are_fine():
    shape, reqs = _base()
    r = reqs[0]
    r.repair = np.zeros_like(r.repair)
    r.repair[0] = 1
    r.page_table = r.page_table.copy()
    # Pages holding only prefix rows or rows of repair block 0: unmap them.
    first_f_row = r.dst_row0 + shape.block_tokens
    for lp in range(first_f_row // shape.page_size):
        r.page_table[lp] = -1
    assert _status(shape, reqs) == VALID


def test_page_alias_within_request():
    shape, reqs = _base()
    r = reqs[0]
    r.page_table = r.page_table.copy()
    lp = _first_f_page(shape, r)
    r.page_table[lp + 1] = r.page_table[lp]
    assert _status(shape, reqs) == pb.PKV_ERR_PAGE_ALIAS


def test_page_alias_across_requests():
    shape, reqs = _base()
    reqs[1].page_table = reqs[1].page_table.copy()
    reqs[1].page_table[_first_f_page(shape, reqs[1])] = reqs[0].page_table[_first_f_page(shape, reqs[0])]
    assert _status(shape, reqs) == pb.PKV_ERR_PAGE_ALIAS


def test_null_pointers(lib):
    import ctypes
    shape, reqs = _base()
    m = pb.make_model(shape)
    arr = pb._Requests(reqs)
    out = ctypes.c_void_p()
    assert lib.pkv_restore_plan(None, arr.array, arr.count, ctypes.byref(out)) == pb.PKV_ERR_INVALID_ARGUMENT
    assert lib.pkv_restore_plan(ctypes.byref(m), None, 1, ctypes.byref(out)) == pb.PKV_ERR_INVALID_ARGUMENT
    assert lib.pkv_restore_plan(ctypes.byref(m), arr.array, arr.count, None) == pb.PKV_ERR_INVALID_ARGUMENT
    assert lib.pkv_restore_plan(ctypes.byref(m), arr.array, -1, ctypes.byref(out)) == pb.PKV_ERR_INVALID_ARGUMENT
    arr.array[0].tags = None
    assert lib.pkv_restore_plan(ctypes.byref(m), arr.array, arr.count, ctypes.byref(out)) == pb.PKV_ERR_INVALID_ARGUMENT
    assert out.value is None
    lib.pkv_free(None)  # no-op
    assert lib.pkv_restore(None, None, 0, None, 0, None, None, 0, None) == pb.PKV_ERR_INVALID_ARGUMENT


def test_empty_suffix_and_all_repair_are_valid():
    shape, reqs = _base()
    reqs[0].suffix_tokens = 0
    reqs[0].tags = np.zeros(0, np.uint8)
    reqs[0].repair = np.zeros(0, np.uint8)
    reqs[1].repair = np.ones_like(reqs[1].repair)
    reqs[1].page_table = np.full_like(reqs[1].page_table, -1)
    assert _status(shape, reqs) == VALID


# ---------------------------------------------------------------------------
# Checkpoint (quantize-and-gather) plan validation
# ---------------------------------------------------------------------------

def _ckpt_base():
    case = wl.make_custom(8, L=2, H=2, D=64, B=16, P=16, n_tokens=(100, 40), deltas=(5, -3), rho0s=(20, 7))
    return case.src_shape, [copy.copy(r) for r in case.requests]


def _ck_status(shape, reqs):
    return pb.pkv_checkpoint_plan_status(shape, reqs)


def test_checkpoint_plan_valid_and_empty():
    shape, reqs = _ckpt_base()
    assert _ck_status(shape, reqs) == VALID
    assert _ck_status(shape, []) == VALID


def test_checkpoint_plan_errors():
    shape, reqs = _ckpt_base()
    r = copy.copy(reqs[0])
    r.tags = r.tags.copy()
    r.tags[0] = 5
    assert _ck_status(shape, [r, reqs[1]]) == pb.PKV_ERR_BAD_TAG
    r = copy.copy(reqs[0])
    r.src_page_table = r.src_page_table.copy()
    r.src_page_table[r.src_row0 // shape.page_size] = -1
    assert _ck_status(shape, [r, reqs[1]]) == pb.PKV_ERR_PAGE_UNMAPPED
    r.src_page_table[r.src_row0 // shape.page_size] = shape.pool_pages
    assert _ck_status(shape, [r, reqs[1]]) == pb.PKV_ERR_PAGE_OUT_OF_RANGE
    r = copy.copy(reqs[0])
    r.src_page_table = r.src_page_table[:1].copy()
    assert _ck_status(shape, [r, reqs[1]]) == pb.PKV_ERR_PAGE_OUT_OF_RANGE
    r = copy.copy(reqs[1])
    r.payload_offset = reqs[0].payload_offset + 16  # overlaps request 0's payload
    assert _ck_status(shape, [reqs[0], r]) == pb.PKV_ERR_INVALID_ARGUMENT
    r = copy.copy(reqs[1])
    r.scale_offset = reqs[0].scale_offset + 4
    assert _ck_status(shape, [reqs[0], r]) == pb.PKV_ERR_INVALID_ARGUMENT
    for field, value in (("reserved", 1), ("reserved2", 1), ("payload_offset", 8), ("scale_offset", 2),
                         ("src_row0", -1), ("suffix_tokens", -1)):
        r = copy.copy(reqs[0])
        setattr(r, field, value)
        assert _ck_status(shape, [r, reqs[1]]) == pb.PKV_ERR_INVALID_ARGUMENT, field


@pytest.mark.parametrize("H,D,B", [(32, 128, 32), (2, 512, 1024), (8, 16, 4), (3, 48, 6)])
def test_checkpoint_plan_any_valid_model(H, D, B):
    """Every model pkv_restore_plan accepts is accepted; the workgroup is one
    wave per head, at most 16."""
    import dataclasses

    from test_gather_indexing import checkpoint_units
    shape, reqs = _ckpt_base()
    big = dataclasses.replace(shape, num_kv_heads=H, head_dim=D, block_tokens=B)
    for i, r in enumerate(reqs):
        r.tags = np.zeros(wl.num_blocks(r.suffix_tokens, B), np.uint8)
        r.payload_offset = i << 30
        r.scale_offset = i << 20
    assert _ck_status(big, reqs) == VALID
    units, wg = checkpoint_units(big, reqs)
    assert wg == 64 * min(H, 16) and len(units) == big.num_layers * sum(len(r.tags) for r in reqs)


def test_plan_kinds_are_not_interchangeable(lib):
    # without a GPU no plan can be built; the kind check itself is exercised on the GPU
    assert lib.pkv_quantize_gather(None, None, None, 0, None, 0, None, 0, None) == pb.PKV_ERR_INVALID_ARGUMENT


def test_missing_library_fails_loudly():
    """No fallback: without libpkv.so the binding raises instead of running
    anything else."""
    saved = pb._lib
    pb._lib = None
    try:
        with pytest.raises(ImportError):
            pb.load("/nonexistent/libpkv.so")
    finally:
        pb._lib = saved


def test_model_reserved_field_must_be_zero():
    import ctypes
    shape, reqs = _base()
    m = pb.make_model(shape)
    m.reserved = 1
    units_fn = pb.load().pkv_payload_size
    size, elems = ctypes.c_uint64(), ctypes.c_uint64()
    r = pb._Requests(reqs)
    assert units_fn(ctypes.byref(m), r.array, ctypes.byref(size), ctypes.byref(elems)) == pb.PKV_ERR_INVALID_ARGUMENT
    m.reserved = 0
    assert units_fn(ctypes.byref(m), r.array, ctypes.byref(size), ctypes.byref(elems)) == pb.PKV_OK


def test_paired_layout_is_a_valid_model():
    import dataclasses
    shape, reqs = _base()
    assert _status(dataclasses.replace(shape, kv_layout=wl.KV_PAIRED), reqs) == VALID
