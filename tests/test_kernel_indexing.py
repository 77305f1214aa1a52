"""CPU emulation of the kernel's address arithmetic (no GPU).

Takes the work list the host plan builds (through an internal test hook of
libpkv), replays the thread -> (token, head, piece) mapping and the address
formulas of ``restore.hip`` for every thread of every workgroup, and checks:
every read stays inside the payload/scales and inside the valid rows of a
reused block's tiles; each work item carries the one page its rows map to;
every write stays inside the caches; every element of every restored row is
written exactly once and nothing else is written.
Keep the constants below in step with the kernel's launch code.
"""
import ctypes
import os

import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

KBITS = (16, 8, 8, 4)
VBITS = (16, 8, 4, 4)
UNIT_ELEMS = 16384  # target output elements per unit
UNIT_DTYPE = np.dtype([("k_off", "<u8"), ("v_off", "<u8"), ("scale_off", "<u8"), ("row0", "<i8"), ("pt_off", "<i8"),
                       ("table_off", "<i4"), ("layer", "<i4"), ("tag", "<i4"), ("n_valid", "<i4"),
                       ("page1", "<i4"), ("page2", "<i4")])


def host_units(shape, requests):
    lib = pb.load()
    fn = lib.pkv_internal_host_units
    fn.argtypes = [ctypes.POINTER(pb.PkvModel), ctypes.POINTER(pb.PkvRequest), ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]
    fn.restype = ctypes.c_int32
    m = pb.make_model(shape)
    reqs = pb._Requests(requests)
    count = ctypes.c_int64()
    assert fn(ctypes.byref(m), reqs.array, reqs.count, None, 0, ctypes.byref(count)) == 0
    units = np.zeros(count.value, dtype=UNIT_DTYPE)
    assert fn(ctypes.byref(m), reqs.array, reqs.count, units.ctypes.data, count.value, ctypes.byref(count)) == 0
    return units


def restore_workgroup(shape) -> int:
    fn = pb.load().pkv_internal_restore_workgroup
    fn.argtypes = [ctypes.POINTER(pb.PkvModel), ctypes.POINTER(ctypes.c_int32)]
    fn.restype = ctypes.c_int32
    m = pb.make_model(shape)
    wg = ctypes.c_int32()
    assert fn(ctypes.byref(m), ctypes.byref(wg)) == 0
    return wg.value


def emulate(case):
    s = case.shape
    H, D, B, P = s.num_kv_heads, s.head_dim, s.block_tokens, s.page_size
    WG = restore_workgroup(s)
    cols = H * D // 16
    assert WG % 64 == 0 and 64 <= WG <= 256
    tpp = WG // cols
    dq = D // 16
    paired = s.kv_layout == wl.KV_PAIRED
    shift = int(np.log2(P)) + int(paired)  # slot rows from a layer's start to page p: p << shift
    layer_elems = (2 if paired else 1) * s.pool_pages * P * H * D
    cache_elems = s.num_layers * layer_elems  # of each cache, or of the one paired cache
    v_offset = P * H * D if paired else 0  # v_cache - k_cache in elements within one paired buffer
    units = host_units(s, case.requests)
    tid = np.arange(WG)
    t0 = tid // cols
    active = t0 < tpp
    c = tid % cols
    head = c // dq
    j = c % dq
    writes_k = np.zeros(cache_elems, dtype=np.int32)
    writes_v = np.zeros(cache_elems, dtype=np.int32)
    payload_read = np.zeros(case.payload_nbytes, dtype=bool)
    # allowed payload bytes: valid rows of reused blocks' tiles
    allowed = np.zeros(case.payload_nbytes, dtype=bool)
    for ri, r in enumerate(case.requests):
        offsets, layer_bytes = oracle.block_layout(r.tags, B, H, D)
        for layer in range(s.num_layers):
            for b in oracle.reused_blocks(r):
                n = oracle.valid_tokens(r, B, b)
                ko, vo = offsets[b]
                base = r.payload_offset + layer * layer_bytes
                t = int(r.tags[b])
                allowed[base + ko: base + ko + n * H * D * KBITS[t] // 8] = True
                allowed[base + vo: base + vo + n * H * D * VBITS[t] // 8] = True
    per_unit = max(1, min(B, UNIT_ELEMS // (H * D)))

    def pieces(r, b):  # a block's rows cut at page boundaries, each page's run into ceil(run / per_unit) parts
        t, n, count = 0, oracle.valid_tokens(r, B, b), 0
        while t < n:
            run = min(P - (r.dst_row0 + b * B + t) % P, n - t)
            count += -(-run // per_unit)
            t += run
        return count

    n_units = sum(pieces(r, b) for r in case.requests for b in oracle.reused_blocks(r))
    assert len(units) == n_units * s.num_layers
    pt_all = np.concatenate([r.page_table for r in case.requests]).astype(np.int64)
    pt_start = np.cumsum([0] + [len(r.page_table) for r in case.requests])
    for u in units:
        n_valid = int(u["n_valid"])
        assert 1 <= n_valid <= per_unit
        ri = int(np.searchsorted(pt_start, int(u["pt_off"]), side="right") - 1)
        assert pt_start[ri] == u["pt_off"]
        r = case.requests[ri]
        tag = int(u["tag"]) & 0xFF
        rot = (int(u["tag"]) >> 8) & 1
        assert rot == int(r.delta != 0)
        assert u["table_off"] == ri * D  # (cos, sin) table of this request, D doubles
        rows = u["row0"] + np.arange(n_valid)
        lp = rows >> int(np.log2(P))
        assert (lp == lp[0]).all(), "a unit crosses a page boundary"
        assert (lp < len(r.page_table)).all()
        page = pt_all[u["pt_off"] + lp]
        assert ((page >= 0) & (page < s.pool_pages)).all()
        assert (page == u["page1"]).all(), "the work item's page is not the rows' page"
        page = np.full(n_valid, int(u["page1"]), dtype=np.int64)  # what the kernel uses
        dst_row = int(u["layer"]) * layer_elems + ((page << shift) | (rows & (P - 1))) * H * D
        kb, vb = KBITS[tag], VBITS[tag]
        if tag != 0:
            sc = int(u["scale_off"]) + 4 * head[active]
            assert (sc >= 0).all() and (sc + 4 <= case.scale_elems).all()
        for tt in range(tpp):
            sel = active & (t0 == tt)
            for t in range(tt, n_valid, tpp):
                rr = t * H + head[sel]
                krow = int(u["k_off"]) + rr * (D * kb // 8)
                vrow = int(u["v_off"]) + rr * (D * vb // 8)
                for base, bits in ((krow, kb), (vrow, vb)):
                    for start in (base + 8 * j[sel] * bits // 8, base + (D // 2 + 8 * j[sel]) * bits // 8):
                        for st in start:
                            assert 0 <= st and st + bits <= case.payload_nbytes
                            payload_read[st: st + bits] = True
                dst = dst_row[t] + head[sel] * D
                for off in (8 * j[sel], D // 2 + 8 * j[sel]):
                    for d0 in dst + off:
                        assert 0 <= d0 and d0 + v_offset + 8 <= cache_elems
                        writes_k[d0: d0 + 8] += 1
                        writes_v[d0 + v_offset: d0 + v_offset + 8] += 1
    assert not (payload_read & ~allowed).any(), "read outside the valid rows of reused blocks"
    assert (payload_read == allowed).all(), "some restored payload byte is never read"
    written = oracle.written_slots(s, case.requests)  # [pool_slots], the same in every layer
    if paired:  # [L][pool_pages][2][P][H*D]: K rows in half 0, V rows in half 1
        rows_of = np.tile(written.reshape(s.pool_pages, 1, P), (s.num_layers, 1, 1))
        want_k = np.zeros((s.num_layers * s.pool_pages, 2, P), np.int32)
        want_v = np.zeros_like(want_k)
        want_k[:, 0, :] = rows_of.reshape(-1, P)
        want_v[:, 1, :] = rows_of.reshape(-1, P)
        want_k = np.repeat(want_k.reshape(-1), H * D)
        want_v = np.repeat(want_v.reshape(-1), H * D)
        assert not (writes_k + writes_v > 1).any(), "a cache element written twice"
    else:
        want_k = want_v = np.repeat(np.tile(written, s.num_layers), H * D).astype(np.int32)
    assert np.array_equal(writes_k, want_k), "K writes differ from the restored rows"
    assert np.array_equal(writes_v, want_v), "V writes differ from the restored rows"


@pytest.mark.parametrize("maker", [
    lambda: wl.make_case("tiny"),
    lambda: wl.make_case("tiny", int4_tag=wl.TAG_K4V4),
    lambda: wl.make_custom(1, L=2, H=3, D=128, B=32, P=16, n_tokens=(70,), deltas=(12,), rho0s=(9,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2),
    lambda: wl.make_custom(2, L=1, H=8, D=64, B=4, P=16, n_tokens=(23, 9), deltas=(5, 0), rho0s=(2, 40),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2),
    lambda: wl.make_custom(3, L=2, H=2, D=256, B=64, P=32, n_tokens=(130,), deltas=(-9,), rho0s=(31,),
                           tag_set=(0, 2), mix=(1, 1), repair_frac=0.1),
    lambda: wl.make_custom(4, L=1, H=32, D=128, B=8, P=8, n_tokens=(41,), deltas=(3,), rho0s=(5,),
                           tag_set=(1, 2), mix=(1, 1), repair_frac=0.0),
    lambda: wl.make_custom(5, L=2, H=8, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2),
    # tensor-parallel shards of the 8B shape: 1, 2 and 4 heads per GPU (64-, 64- and 128-thread workgroups)
    lambda: wl.make_custom(14, L=2, H=1, D=128, B=32, P=16, n_tokens=(75,), deltas=(-1500,), rho0s=(1507,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2),
    lambda: wl.make_custom(15, L=2, H=2, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2),
    lambda: wl.make_custom(16, L=1, H=4, D=128, B=32, P=16, n_tokens=(75,), deltas=(5,), rho0s=(13,),
                           tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2),
], ids=["tiny", "tiny_k4v4", "h3_d128", "h8_b4_two_requests", "d256_b64", "h32_b8", "h8_d128_split_units",
        "tp_h1", "tp_h2", "tp_h4"])
def test_kernel_addresses(maker):
    emulate(maker())


@pytest.mark.parametrize("H,D,B,P,want", [
    (8, 128, 32, 16, 256), (4, 128, 32, 16, 128), (2, 128, 32, 16, 64), (1, 128, 32, 16, 64),
    (1, 128, 64, 32, 64), (32, 128, 8, 8, 256), (8, 512, 4, 2, 256), (2, 64, 16, 16, 64), (3, 128, 32, 16, 128),
])
def test_restore_workgroup_size(H, D, B, P, want):
    """Each thread owns at most four tokens of the largest unit (units stop at
    page ends), in whole waves, 64 to 256 threads."""
    case = wl.make_custom(1, L=1, H=H, D=D, B=B, P=P, n_tokens=(B,), deltas=(0,), rho0s=(0,))
    wg = restore_workgroup(case.shape)
    assert wg == want
    cols = H * D // 16
    unit = min(max(1, min(B, UNIT_ELEMS // (H * D))), P)
    assert -(-unit // (wg // cols)) <= 4


def _paired(case):
    import dataclasses
    case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    return case


@pytest.mark.parametrize("maker", [
    lambda: _paired(wl.make_case("tiny")),
    lambda: _paired(wl.make_custom(1, L=2, H=3, D=128, B=32, P=16, n_tokens=(70,), deltas=(12,), rho0s=(9,),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2)),
    lambda: _paired(wl.make_custom(2, L=1, H=8, D=64, B=4, P=16, n_tokens=(23, 9), deltas=(5, 0), rho0s=(2, 40),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2)),
    lambda: _paired(wl.make_custom(5, L=2, H=8, D=128, B=32, P=16, n_tokens=(75,), deltas=(-3,), rho0s=(7,),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2)),
    lambda: _paired(wl.make_custom(6, L=1, H=2, D=64, B=64, P=4, n_tokens=(130,), deltas=(1,), rho0s=(3,),
                                   tag_set=(0, 2), mix=(1, 1), repair_frac=0.1)),
    lambda: _paired(wl.make_custom(14, L=2, H=1, D=128, B=32, P=16, n_tokens=(75,), deltas=(-1500,), rho0s=(1507,),
                                   tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2)),
], ids=["tiny", "h3_d128", "h8_b4_two_requests", "h8_d128_unaligned", "b64_p4", "tp_h1"])
def test_kernel_addresses_paired_pages(maker):
    emulate(maker())


_XCD_PROGRAM = r"""
#include <cstdio>
#include <vector>
#include "pkv_internal.h"
int main() {
  using pkv::xcd_grouped;
  const long long grids[] = {0, 1, 7, 8, 63, 64, 65, 127, 128, 129, 1000, 83520, 83521, 131072, 1331936};
  for (long long grid : grids) {
    std::vector<long long> phys(grid, -1);
    for (long long b = 0; b < grid; ++b) {
      const long long l = xcd_grouped(b, grid);
      if (l < 0 || l >= grid || phys[l] != -1) { printf("grid %lld: not a permutation at %lld\n", grid, b); return 1; }
      phys[l] = b;
    }
    const long long round = pkv::kXcdCount * pkv::kXcdGroup, full = grid / round * round;
    for (long long l = 0; l < grid; ++l) {
      const long long first = l / pkv::kXcdGroup * pkv::kXcdGroup;
      if (l < full && phys[l] % pkv::kXcdCount != phys[first] % pkv::kXcdCount) {
        printf("grid %lld: item %lld not on the XCD of item %lld\n", grid, l, first); return 1;
      }
      if (l >= full && phys[l] != l) { printf("grid %lld: tail item %lld moved\n", grid, l); return 1; }
    }
  }
  printf("ok\n");
  return 0;
}
"""


def test_xcd_grouping_is_a_permutation(tmp_path):
    """Work items are renumbered so that kXcdGroup consecutive ones share an
    XCD (workgroup b runs on XCD b % 8); every launch size must still see
    each work item exactly once."""
    import shutil
    import subprocess
    if shutil.which("g++") is None:
        pytest.skip("no host C++ compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = tmp_path / "xcd.cpp"
    src.write_text(_XCD_PROGRAM)
    exe = tmp_path / "xcd"
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", os.path.join(root, "include"), "-I",
                    os.path.join(root, "paper_2609_26219_amd", "csrc"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "ok", out.stdout + out.stderr
