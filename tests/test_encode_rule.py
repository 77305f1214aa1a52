"""CPU model of the checkpoint kernel's float code path, checked against the
oracle quantizer's codes and ranges.

The kernel forms t = (x - zero) * (1/scale) in float32: the subtraction, the
reciprocal and the product each round by at most 2^-24 relative, so on a
quotient of at most 255 t is within 5e-5 of the exact quotient.  It rounds t
to the nearest integer (the hardware's float -> byte conversion, ties to
even), and recomputes in double, with a true division, every packed word that
holds a value whose t lies within 1e-4 of a half-integer.  So its codes equal
the definition's rint((x - zero) / scale) everywhere.  The range pass compares
the high bf16 value of each 32-bit word as the raw word and clears the low
half of the result.

This model replays both rules with numpy float32 arithmetic (IEEE single,
round to nearest even, like the kernel's v_sub_f32 / v_mul_f32) on tiles built
to sit on and next to ties, and on bf16 and fp16 values over many magnitudes.
Keep it in step with gather.hip."""
import numpy as np
import pytest

from oracle import quantize as oq

TIE_WINDOW = np.float32(1e-4)


def f16_value(bits):
    return float(np.array(bits, np.uint16).view(np.float16))


def to_bf16(x32):
    b = x32.view(np.uint32)
    b = ((b + (((b >> 16) & 1) + 0x7FFF)) >> 16 << 16).astype(np.uint32)
    return b.view(np.float32)


def kernel_codes(x32, zero, scale, bits):
    """Codes of the kernel's rule and the number of values sent to double."""
    zf = np.float32(zero)
    invf = np.float32(1.0 / scale)
    t = (x32 - zf) * invf  # float32 subtract, then float32 multiply
    fast = np.rint(t)  # ties to even, like the conversion
    near = np.abs((t - np.floor(t)) - np.float32(0.5)) < TIE_WINDOW
    exact = np.clip(np.rint((x32.astype(np.float64) - zero) / scale), 0, (1 << bits) - 1)
    codes = np.where(near, exact, fast)
    assert fast.max() <= (1 << bits) - 1 and fast.min() >= 0  # no clip needed on the fast path
    return codes.astype(np.uint8), int(near.sum())


def tiles(rng, trial, bits):
    n = int(rng.integers(8, 256))
    mode = trial % 5
    if mode == 0:
        x = rng.standard_normal(n) * 10 ** rng.uniform(-6, 4)
    elif mode == 1:  # narrow span far from zero
        x = rng.uniform(-1, 1, n) * 10 ** rng.uniform(-3, 1) + rng.uniform(-100, 100)
    elif mode == 2:  # tiny values next to unit ones
        x = np.concatenate([rng.standard_normal(n // 2) * 1e-30, rng.standard_normal(n - n // 2)])
    else:  # values on and within 1e-6 steps of half-integer multiples of a first tile's scale
        base = rng.standard_normal(n) * 10 ** rng.uniform(-2, 2)
        _, sb, zb = oq.quantize_tile(base.astype(np.float32).astype(np.float64), bits)
        s, z = f16_value(sb), f16_value(zb)
        k = rng.integers(0, (1 << bits) - 1, n)
        x = z + (k + 0.5) * s + rng.choice([-1, 0, 1], n) * rng.uniform(0, 1e-6, n) * s
        x[0], x[1] = base.min(), base.max()
    x32 = x.astype(np.float32)
    x32 = to_bf16(x32) if trial % 3 == 0 else x32.astype(np.float16).astype(np.float32)
    return x32[np.isfinite(x32) & (np.abs(x32) <= 65504)]


@pytest.mark.parametrize("bits", [8, 4])
def test_float_rule_matches_the_definition(bits):
    rng = np.random.default_rng(26219 + bits)
    total = fallbacks = 0
    for trial in range(1500):
        x32 = tiles(rng, trial, bits)
        if x32.size == 0:
            continue
        codes, sb, zb = oq.quantize_tile(x32.astype(np.float64), bits)
        scale, zero = f16_value(sb), f16_value(zb)
        if scale == 0.0:
            continue
        got, nf = kernel_codes(x32, zero, scale, bits)
        np.testing.assert_array_equal(got, codes)
        total += x32.size
        fallbacks += nf
    assert total > 100_000
    assert 0 < fallbacks < total // 10  # the tie tiles do reach the double path


def test_raw_word_range_of_bf16_pairs():
    """min / max over (low value, raw word) per word, low half cleared, equal
    the min / max over both bf16 values of every word."""
    rng = np.random.default_rng(7)
    for trial in range(400):
        n = int(rng.integers(1, 64))
        scale = 10 ** rng.uniform(-30, 30)
        pairs = to_bf16((rng.standard_normal(2 * n) * scale).astype(np.float32)).view(np.uint32) >> 16
        if trial % 4 == 0:  # signed zeros and equal neighbours
            pairs[rng.integers(0, 2 * n, n)] = rng.choice([0x0000, 0x8000, pairs[0]], n)
        lo, hi = pairs[0::2].astype(np.uint32), pairs[1::2].astype(np.uint32)
        words = lo | (hi << 16)
        lo_f = (words << 16).view(np.float32)
        raw_f = words.view(np.float32)
        both = np.concatenate([lo_f, (hi << 16).view(np.float32)])
        mn = np.float32(min(lo_f.min(), raw_f.min())).view(np.uint32) & 0xFFFF0000
        mx = np.float32(max(lo_f.max(), raw_f.max())).view(np.uint32) & 0xFFFF0000
        assert np.uint32(mn).view(np.float32) == both.min()
        assert np.uint32(mx).view(np.float32) == both.max()
