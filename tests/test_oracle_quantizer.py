"""Pins for the oracle's fp16 conversions and group quantizer (CPU only).

The quantizer is an encoding (affine 4-bit with per-group scale and offset,
the affine 4-bit format the paper's Introduction describes for weights);
these tests pin it to facts that do not come from the oracle itself:
numpy's binary16 conversion (an independent library routine), the definition
of directed rounding, and the error bound of affine quantization with the
scale rounded up and the bias rounded down.
"""
import numpy as np
import pytest

import oracle

F16 = np.float16


def _np_half_bits(f32):
    return int(np.float32(f32).astype(np.float16).view(np.uint16))


def test_half_to_double_exhaustive_matches_numpy():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    lib = oracle.lib()
    got = np.array([lib.jfo_half_to_double(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def _sample_floats(n, seed):
    rng = np.random.default_rng(seed)
    # random binary32 bit patterns restricted to the binary16 range and below
    e = rng.integers(127 - 30, 127 + 17, size=n)
    m = rng.integers(0, 1 << 23, size=n)
    s = rng.integers(0, 2, size=n)
    f = ((s << 31) | (e << 23) | m).astype(np.uint32).view(np.float32)
    # exact ties between binary16 neighbours and exactly representable values
    h = rng.integers(0, 0x7bff, size=n // 4).astype(np.uint16)
    hv = h.view(np.float16).astype(np.float32)
    nxt = (h + 1).astype(np.uint16).view(np.float16).astype(np.float32)
    ties = ((hv.astype(np.float64) + nxt.astype(np.float64)) / 2).astype(np.float32)
    specials = np.array([0.0, -0.0, 65504.0, 65519.0, 65520.0, 65536.0, 1e6, -1e6,
                         2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -26, 6.1e-5,
                         np.inf, -np.inf], np.float32)
    return np.concatenate([f, hv, ties, -ties, specials])


def test_float_to_half_nearest_matches_numpy():
    lib = oracle.lib()
    for f in _sample_floats(20000, 1):
        assert lib.jfo_float_to_half(float(f), 0) == _np_half_bits(f), f


@pytest.mark.parametrize("mode", [1, 2])
def test_float_to_half_directed_rounding_definition(mode):
    """toward -inf: largest fp16 <= f; toward +inf: smallest fp16 >= f
    (the definition of directed rounding, IEEE 754 clause 4.3.2)."""
    lib = oracle.lib()
    for f in _sample_floats(6000, 2 + mode):
        if not np.isfinite(f):
            continue
        hb = lib.jfo_float_to_half(float(f), mode)
        h = np.uint16(hb).view(np.float16)
        hv = float(h)
        fv = float(f)
        if mode == 1:
            assert hv <= fv or (np.isinf(hv) and hv < 0)
            up = np.nextafter(h, np.float16(np.inf))
            assert float(up) > fv
        else:
            assert hv >= fv or (np.isinf(hv) and hv > 0)
            dn = np.nextafter(h, np.float16(-np.inf))
            assert float(dn) < fv


def _groups(seed, n, G, dist="normal"):
    rng = np.random.default_rng(seed)
    if dist == "normal":
        x = rng.standard_normal((n, G)).astype(np.float32)
        x[:, rng.integers(0, G)] *= 8
    elif dist == "tiny":  # ranges below 15 * 2^-14: subnormal scales
        x = (rng.standard_normal((n, G)) * 2.0 ** -16).astype(np.float32)
    elif dist == "wide":
        x = (rng.standard_normal((n, G)) * 3000.0).astype(np.float32)
    elif dist == "few_levels":
        x = rng.integers(-3, 4, size=(n, G)).astype(np.float32) * 0.125
    else:
        raise ValueError(dist)
    return x.astype(np.float16)


@pytest.mark.parametrize("dist", ["normal", "tiny", "wide", "few_levels"])
@pytest.mark.parametrize("G", [32, 64, 128])
def test_quantizer_invariants(dist, G):
    xs = _groups(10 + G, 300, G, dist)
    for x in xs:
        codes, s, b = oracle.quantize_group(x)
        xd = x.astype(np.float64)
        mn, mx = xd.min(), xd.max()
        assert codes.max() <= 15
        # bias: fp16 rounded toward -inf from the (fp16-exact) minimum
        assert float(b) == mn
        rng32 = np.float32(np.float32(mx) - np.float32(mn))
        step = np.float32(rng32 / np.float32(15.0))
        if rng32 == 0:
            assert float(s) == 0.0 and not np.signbit(s)
            assert (codes == 0).all()
            continue
        # scale: the smallest fp16 >= step
        assert float(s) >= float(step)
        assert float(np.nextafter(s, F16(0))) < float(step)
        sd, bd = float(s), float(b)
        xhat = sd * codes.astype(np.float64) + bd
        # every element within half a step of its level (levels cover [mn, mx])
        assert np.all(np.abs(xd - xhat) <= sd * (0.5 + 2.0 ** -18))
        # the chosen level is a nearest one among all 16
        levels = sd * np.arange(16, dtype=np.float64) + bd
        best = np.min(np.abs(xd[:, None] - levels[None, :]), axis=1)
        assert np.all(np.abs(xd - xhat) <= best + sd * 2.0 ** -18)
        assert codes[np.argmin(xd)] == 0
        if sd >= 2.0 ** -14:  # normal scale: rounding up adds < 2^-10 relative
            assert codes[np.argmax(xd)] == 15


def test_constant_group_reconstructs_exactly():
    for v in [0.0, -0.0, 1.5, -3.25, 65504.0, 2.0 ** -24]:
        x = np.full(64, v, np.float16)
        codes, s, b = oracle.quantize_group(x)
        assert float(s) == 0.0 and (codes == 0).all()
        assert float(b) == float(np.float16(v))


def test_exact_grid_group_roundtrips():
    """x = bias + scale*c with a power-of-two scale quantizes to exactly c."""
    rng = np.random.default_rng(7)
    for _ in range(200):
        e = int(rng.integers(-8, 3))
        s = 2.0 ** e
        bias = float(rng.integers(-64, 64)) * s
        c = rng.integers(0, 16, size=64)
        c[rng.integers(0, 64)] = 0
        c[rng.integers(0, 64)] = 15
        if c.min() != 0 or c.max() != 15:
            continue
        x = (bias + s * c).astype(np.float16)
        assert np.array_equal(x.astype(np.float64), bias + s * c)
        codes, sc, b = oracle.quantize_group(x)
        assert float(sc) == s and float(b) == bias
        assert np.array_equal(codes, c)


def test_ties_round_half_even():
    """A value exactly halfway between two levels takes the even code: with
    scale 1 and bias 0, x = k + 0.5 -> code of the even neighbour."""
    x = np.zeros(64, np.float16)
    x[1] = 15.0  # min 0, max 15 -> step 1, scale 1, bias 0
    x[2:17] = np.arange(15) + 0.5
    codes, s, b = oracle.quantize_group(x)
    assert float(s) == 1.0 and float(b) == 0.0
    expect = [int(np.rint(k + 0.5)) for k in range(15)]  # numpy rint: half-even
    assert list(codes[2:17]) == expect
    assert expect[:4] == [0, 2, 2, 4]


def test_signed_zero_order_is_element_order_independent():
    """-0 orders below +0 for the minimum and above-zero ties go to +0 for the
    maximum, whatever the element order."""
    x = np.zeros(64, np.float16)
    x[5] = np.float16(-0.0)
    for perm_seed in range(5):
        xp = np.random.default_rng(perm_seed).permutation(x)
        codes, s, b = oracle.quantize_group(xp)
        assert np.signbit(b) and float(s) == 0.0 and not np.signbit(s)
    y = np.zeros(64, np.float16)
    y[:] = np.float16(-0.0)
    y[9] = np.float16(0.0)
    y[10] = np.float16(2.0)
    for perm_seed in range(5):
        yp = np.random.default_rng(perm_seed).permutation(y)
        codes, s, b = oracle.quantize_group(yp)
        assert np.signbit(b)
