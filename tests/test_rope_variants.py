"""Model-aware key phase correction: pins of the oracle's RoPE variants
(rotate-half and interleaved pairs, partial rotary, explicit frequency
tables), and a CPU check that the kernel's key-piece layout with the
planner's element-ordered (cos, sin) table rotates exactly the oracle's pairs."""
import ctypes
import math

import numpy as np
import pytest

import oracle
from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl

HALF, INTER = oracle.ROPE_HALF, oracle.ROPE_INTERLEAVED


def test_hand_worked_quarter_and_half_turns():
    """Frequencies (pi/2, pi), Delta = 1: pair 0 turns a quarter, pair 1 a half."""
    k = np.array([[1.0, 2.0, 3.0, 4.0]])
    f = [math.pi / 2, math.pi]
    inter = oracle.correct_key_phase(k, 1, 1e4, INTER, 4, f)[0]   # pairs (0,1), (2,3)
    half = oracle.correct_key_phase(k, 1, 1e4, HALF, 4, f)[0]     # pairs (0,2), (1,3)
    assert np.allclose(inter, [-2.0, 1.0, -3.0, -4.0], atol=1e-15, rtol=0)
    assert np.allclose(half, [-3.0, -2.0, 1.0, -4.0], atol=1e-15, rtol=0)


@pytest.mark.parametrize("style", [HALF, INTER])
def test_partial_rotary_passes_the_rest_through(style):
    rng = np.random.default_rng(1)
    k = rng.standard_normal((5, 128))
    k[:, 64:66] = -0.0
    out = oracle.correct_key_phase(k, 777, 1e4, style, 64)
    assert np.array_equal(out[:, 64:], k[:, 64:]) and np.array_equal(np.signbit(out[:, 64:]), np.signbit(k[:, 64:]))
    # the rotated part is the full rotary of a 64-channel head
    assert np.allclose(out[:, :64], oracle.correct_key_phase(k[:, :64], 777, 1e4, style), atol=1e-13, rtol=0)


def test_interleaved_is_rotate_half_of_permuted_channels():
    """Moving channel 2i to i and 2i+1 to i + R/2 turns interleaved pairs into
    rotate-half pairs; the two forms agree under that permutation."""
    rng = np.random.default_rng(2)
    R, D = 96, 128
    k = rng.standard_normal((7, D))
    perm = np.concatenate([np.arange(0, R, 2), np.arange(1, R, 2), np.arange(R, D)])  # new position -> old channel
    for delta in (1, -513, 40000):
        inter = oracle.correct_key_phase(k, delta, 5e5, INTER, R)
        half = oracle.correct_key_phase(k[:, perm], delta, 5e5, HALF, R)
        assert np.allclose(inter[:, perm], half, atol=1e-12, rtol=0)


@pytest.mark.parametrize("style,R", [(HALF, 128), (INTER, 128), (HALF, 64), (INTER, 32)])
def test_group_law_with_a_frequency_table(style, R):
    freq = wl.llama3_inv_freq(5e5, R)
    rng = np.random.default_rng(3)
    k = rng.standard_normal((4, 128))
    for p, d in ((100, 37), (30000, -8000)):
        stored = oracle.correct_key_phase(k, p, 5e5, style, R, freq)
        moved = oracle.correct_key_phase(stored, d, 5e5, style, R, freq)
        direct = oracle.correct_key_phase(k, p + d, 5e5, style, R, freq)
        assert np.allclose(moved, direct, atol=1e-9, rtol=0)


def test_default_table_is_theta_power():
    rng = np.random.default_rng(4)
    k = rng.standard_normal((3, 64))
    table = [1e4 ** (-2.0 * i / 64) for i in range(32)]
    assert np.allclose(oracle.correct_key_phase(k, 91, 1e4, HALF, 64, table),
                       oracle.correct_key_phase(k, 91, 1e4, HALF, 64, None), atol=1e-13, rtol=0)


def test_llama3_scaled_frequencies():
    theta, dim, factor = 5e5, 128, 8.0
    base = theta ** (-np.arange(0, dim, 2) / dim)
    f = np.array(wl.llama3_inv_freq(theta, dim, factor))
    wavelen = 2 * math.pi / base
    fast = wavelen < 8192 / 4.0
    slow = wavelen > 8192 / 1.0
    assert fast.any() and slow.any()
    assert np.array_equal(f[fast], base[fast]) and np.allclose(f[slow], base[slow] / factor, rtol=1e-15)
    mid = ~fast & ~slow
    assert ((f[mid] <= base[mid]) & (f[mid] >= base[mid] / factor)).all()
    assert (np.diff(f) < 0).all()  # still strictly decreasing


# ---------------------------------------------------------------------------
# Kernel layout: key piece j of a head = two 8-channel runs (lo, hi)
# ---------------------------------------------------------------------------

def key_piece(j, D, R, style):
    """The kernel's key piece j: (lo, hi, rotate lo, rotate hi)."""
    if style == HALF:
        if 8 * j < R // 2:
            return 8 * j, R // 2 + 8 * j, True, True
        q = j - R // 16
        return R + 8 * q, R + (D - R) // 2 + 8 * q, False, False
    lo, hi = 8 * j, D // 2 + 8 * j
    return lo, hi, lo + 8 <= R, hi + 8 <= R


def host_tables(shape, requests):
    lib = pb.load()
    fn = lib.pkv_internal_host_tables
    fn.argtypes = [ctypes.POINTER(pb.PkvModel), ctypes.POINTER(pb.PkvRequest), ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]
    fn.restype = ctypes.c_int32
    m = pb.make_model(shape)
    reqs = pb._Requests(requests)
    n = ctypes.c_int64()
    assert fn(ctypes.byref(m), reqs.array, reqs.count, None, 0, ctypes.byref(n)) == 0
    out = np.zeros(n.value, np.float64)
    assert fn(ctypes.byref(m), reqs.array, reqs.count, out.ctypes.data, n.value, ctypes.byref(n)) == 0
    return out.reshape(len(requests), shape.head_dim // 2, 2)


@pytest.mark.parametrize("D,R,style,scaled", [(128, 128, HALF, False), (128, 64, HALF, False), (64, 16, HALF, True),
                                              (128, 128, INTER, False), (128, 64, INTER, True), (48, 32, INTER, False),
                                              (256, 96, HALF, True)])
def test_kernel_pairs_and_table_match_the_oracle(D, R, style, scaled):
    inv = wl.llama3_inv_freq(5e5, R) if scaled else None
    case = wl.make_custom(3, L=1, H=2, D=D, B=16, P=16, n_tokens=(40, 20), deltas=(-301, 7), rho0s=(5, 90))
    shape = case.shape.__class__(**{**case.shape.__dict__, "rope_style": style, "rotary_dim": R if R != D else 0,
                                    "inv_freq": inv})
    tables = host_tables(shape, case.requests)
    a, b = oracle.rope_pairs(D, R, style)
    pair_of = {(int(x), int(y)): i for i, (x, y) in enumerate(zip(a, b))}
    freq = oracle.rope_frequencies(shape.rope_theta, R, inv)
    written = np.zeros(D, int)
    rotated = np.zeros(D, int)
    for j in range(D // 16):
        lo, hi, rlo, rhi = key_piece(j, D, R, style)
        written[lo:lo + 8] += 1
        written[hi:hi + 8] += 1
        for e in range(8):
            if style == HALF:
                pair = (lo + e, hi + e) if rlo else None
            else:
                run, k = (lo, e) if e < 4 else (hi, e - 4)
                pair = (run + 2 * k, run + 2 * k + 1) if (rlo if e < 4 else rhi) else None
            for ri, req in enumerate(case.requests):
                c, s = tables[ri, 8 * j + e]
                if pair is None:
                    assert (c, s) == (1.0, 0.0)
                    continue
                i = pair_of[pair]
                ang = req.delta * freq[i]
                assert abs(c - math.cos(ang)) < 1e-12 and abs(s - math.sin(ang)) < 1e-12
            if pair is not None:
                rotated[list(pair)] += 1
    assert (written == 1).all()                       # every key channel in exactly one run
    assert (rotated[:R] == 1).all() and (rotated[R:] == 0).all()  # exactly the first R channels rotate


def test_rope_fields_are_validated():
    case = wl.make_case("tiny")
    s = case.shape
    bad = [dict(rope_style=2), dict(rotary_dim=8), dict(rotary_dim=72), dict(rotary_dim=24),
           dict(inv_freq=(float("nan"),) * 32)]
    for kw in bad:
        shape = s.__class__(**{**s.__dict__, **kw})
        assert pb.pkv_restore_plan_status(shape, case.requests) == pb.PKV_ERR_INVALID_ARGUMENT, kw
