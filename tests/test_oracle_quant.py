"""Pins of the oracle's fp16 conversions and group quantizer (CPU only).

The quantizer follows DiffKV Sec. 2.2: s, z from the group's min and max,
Q = round((X - z) / s), X_hat = s * Q + z, s and z kept in fp16.  Pins:
library routines (numpy's IEEE binary16 casts), closed forms, a grid-exact
round trip, brute-force nearest code, and the rounding error bound.
"""
import numpy as np
import pytest


def test_half_to_float_exhaustive(orc):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    got = orc.half_to_float(bits)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_float_to_half_rne_matches_numpy(orc):
    rng = np.random.default_rng(123)
    # random bit patterns over the whole finite fp32 range, biased to fp16's
    u = rng.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    f = u.view(np.float32)
    f = f[np.isfinite(f)]
    e = rng.uniform(-30, 17, size=1 << 20)
    g = (rng.standard_normal(1 << 20) * np.exp2(e)).astype(np.float32)
    # exact ties between neighbouring fp16 values, incl. subnormal and overflow edges
    h = np.arange(0, 0x7c00, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    ties = ((lo + hi) / 2)[:-1].astype(np.float32)
    edges = np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 65536.0, 2.0 ** -24, 2.0 ** -25,
                      2.0 ** -25 * 1.0000001, 2.0 ** -26, 6.1035e-5, 1e-8, np.inf, -np.inf],
                     np.float32)
    allf = np.concatenate([f, g, -g, ties, -ties, edges])
    with np.errstate(over="ignore"):
        ref = allf.astype(np.float16).view(np.uint16)
    got = orc.float_to_half(allf)
    assert np.array_equal(got, ref)


def _deq(s16, z16, codes):
    s = np.uint16(s16).view(np.float16).astype(np.float64)
    z = np.uint16(z16).view(np.float16).astype(np.float64)
    return s * codes.astype(np.float64) + z


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantize_hand_example(orc, bits):
    # x = 0, 1, ..., Lb: s = 1, z = 0, codes = x exactly
    lb = (1 << bits) - 1
    x = np.arange(32) % (lb + 1)
    x[0], x[1] = 0, lb
    s, z, c = orc.quantize_group(x.astype(np.float16).view(np.uint16), bits)
    assert s == np.float16(1.0).view(np.uint16)
    assert z == 0
    assert np.array_equal(c, x.astype(np.uint8))


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantize_grid_exact_round_trip(orc, bits):
    """Values z + s*c with s a power of two and both end codes present come back exactly."""
    rng = np.random.default_rng(bits)
    lb = (1 << bits) - 1
    for _ in range(200):
        e = int(rng.integers(-8, 2))
        s = 2.0 ** e
        z = float(np.float16(rng.integers(-64, 64) * s))
        c = rng.integers(0, lb + 1, 32)
        i0, i1 = rng.choice(32, 2, replace=False)
        c[i0], c[i1] = 0, lb
        x = z + s * c
        assert np.array_equal(np.float16(x).astype(np.float64), x)  # representable
        s16, z16, codes = orc.quantize_group(x.astype(np.float16).view(np.uint16), bits)
        if z == 0.0:
            assert z16 == 0  # +0, never -0
        assert np.uint16(s16).view(np.float16) == s
        assert np.uint16(z16).view(np.float16) == z
        assert np.array_equal(codes, c.astype(np.uint8))
        assert np.array_equal(_deq(s16, z16, codes), x)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantize_nearest_code_and_bounds(orc, bits):
    rng = np.random.default_rng(100 + bits)
    lb = (1 << bits) - 1
    for trial in range(400):
        scale = 10.0 ** rng.uniform(-3, 2)
        x32 = (rng.standard_normal(32) * scale).astype(np.float32)
        if trial % 7 == 0:
            x32[rng.integers(0, 32, 3)] *= 10.0
        xb = x32.astype(np.float16).view(np.uint16)
        x = xb.view(np.float16).astype(np.float64)
        s16, z16, codes = orc.quantize_group(xb, bits)
        s = float(np.uint16(s16).view(np.float16))
        z = float(np.uint16(z16).view(np.float16))
        assert z == x.min()
        assert codes[np.argmin(x)] == 0
        assert codes[np.argmax(x)] == lb
        assert codes.max() <= lb
        xh = _deq(s16, z16, codes)
        # brute force: the chosen code is a nearest grid point (up to fp32 rounding of the ratio)
        grid = s * np.arange(lb + 1)[None, :] + z
        best = np.abs(x[:, None] - grid).min(axis=1)
        assert np.all(np.abs(x - xh) <= best + 1e-6 * s + 1e-12)
        # error bound: half a step plus the fp16 rounding of the scale, stretched over Lb steps
        s32 = (np.float32(x.max()) - np.float32(x.min())) / np.float32(lb)
        bound = s / 2 + lb * abs(float(s32) - s) + 1e-9
        assert np.all(np.abs(xh - x) <= bound)


def test_quantize_constant_and_signed_zero(orc):
    for val in [0.0, 1.5, -3.25, 65504.0]:
        x = np.full(32, val, np.float16).view(np.uint16)
        s16, z16, codes = orc.quantize_group(x, 4)
        assert s16 == 0 and np.all(codes == 0)
        assert np.uint16(z16).view(np.float16) == np.float16(val)
        assert np.all(_deq(s16, z16, codes) == val)
    neg0 = np.full(32, 0x8000, np.uint16)
    s16, z16, codes = orc.quantize_group(neg0, 8)
    assert z16 == 0 and s16 == 0  # -0 counts as +0
    mixed = np.full(32, 0x8000, np.uint16)
    mixed[5] = np.float16(2.0).view(np.uint16)
    s16, z16, codes = orc.quantize_group(mixed, 2)
    assert z16 == 0 and codes[5] == 3 and np.all(np.delete(codes, 5) == 0)


def test_quantize_scale_rounding_clamps(orc):
    """A subnormal scale can round far below (max-min)/Lb; the top codes are then clamped.

    x = k * 2^-24 for k in [0, 357]: s32 = 1.4 * 2^-24 rounds to the fp16 subnormal
    2^-24, so the exact ratio is k and every k > 255 must give code 255."""
    k = np.linspace(0, 357, 32).round().astype(np.int64)
    x = (k * 2.0 ** -24).astype(np.float16)
    assert np.array_equal(x.astype(np.float64) / 2.0 ** -24, k)
    s16, z16, codes = orc.quantize_group(x.view(np.uint16), 8)
    assert s16 == 1 and z16 == 0  # 2^-24 is the fp16 bit pattern 0x0001
    assert np.array_equal(codes, np.minimum(k, 255).astype(np.uint8))
