"""The oracle's group quantizer against an independent NumPy float32 twin,
bit for bit, on about a million groups (CPU only).

The twin (``tests/quantizer_twin.py``) rounds to fp16 by integer arithmetic
on the binary32 significand and exponent, orders values by an integer key
(-0 below +0), and takes the encoding's binary32 steps in order: bias = the
group minimum rounded down, step = (max - min) / 15 rounded up to fp16,
code = round-half-even((x - bias) / scale) clamped to 0..15.  The oracle must
agree on every code, scale bit and bias bit.

The groups cover random Gaussian data over eleven decades of magnitude,
outlier channels, exact midpoint ties, subnormal scales, constant groups,
signed zeros and the fp16 extremes.  Planted mistakes in copies of the oracle
(the division done by a reciprocal, ties rounded up, the scale rounded to
nearest, -0 ordered equal to +0) must each be caught.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from quantizer_twin import quantize_groups as twin_quantize
from quantizer_twin import round_f32_to_f16

HERE = os.path.dirname(os.path.abspath(__file__))


def _f16(a):
    return np.asarray(a, np.float64).astype(np.float16)


def gaussian_groups(rng, n, G):
    mag = 10.0 ** rng.uniform(-6.0, 4.3, size=(n, 1))
    x = rng.standard_normal((n, G)) * mag
    return _f16(np.clip(x, -65504, 65504))


def outlier_groups(rng, n, G):
    x = rng.standard_normal((n, G))
    ch = rng.integers(0, G, size=n)
    x[np.arange(n), ch] *= 8.0
    return _f16(x)


def tie_groups(rng, n, G):
    """Elements bias + (c/2) * scale with bias, scale and every element exact
    in fp16 and binary32, so (x - bias) / scale is exactly c/2: odd c are
    midpoint ties.  c = 0 and c = 30 are present, so the quantizer's own
    bias and scale are exactly these."""
    e = rng.integers(-20, 3, size=(n, 1)).astype(np.float64)
    ms = rng.integers(1, 31, size=(n, 1)).astype(np.float64)
    mb = rng.integers(-500, 501, size=(n, 1)).astype(np.float64)
    c = rng.integers(0, 31, size=(n, G)).astype(np.float64)
    c[:, 0], c[:, 1] = 0, 30
    x = (2 * mb + c * ms) * np.exp2(e - 1)
    assert np.all(np.abs(2 * mb) + 30 * ms < 2048)
    h = _f16(x)
    assert np.array_equal(h.astype(np.float64), x)
    return h


def subnormal_scale_groups(rng, n, G):
    """Ranges below 15 * 2^-14, so the scale is an fp16 subnormal."""
    base = rng.choice([0.0, 2.0 ** -14, -2.0 ** -13, 1e-3, -0.5], size=(n, 1))
    k = rng.integers(0, 200, size=(n, G)).astype(np.float64)
    unit = np.exp2(-rng.integers(20, 25, size=(n, 1)).astype(np.float64))
    return _f16(base + k * unit)


def special_groups(G):
    rows = []
    for v in (0.0, -0.0, 1.0, -3.5, 65504.0, -65504.0, 2.0 ** -24, -2.0 ** -24, 6.1e-5):
        rows.append(np.full(G, v))
    z = np.zeros(G)
    z[::3] = -0.0
    rows.append(z)                      # signed zeros: -0 is the minimum
    z2 = np.full(G, -0.0)
    z2[5] = 0.0
    rows.append(z2)
    z3 = np.abs(np.linspace(0, 2, G))
    z3[4] = -0.0
    rows.append(z3)                     # +0 first, a later -0 is the minimum
    ext = np.linspace(-65504, 65504, G)
    rows.append(ext)                    # the widest range
    hi = np.full(G, 65504.0)
    hi[1] = 65472.0
    rows.append(hi)
    lo = np.zeros(G)
    lo[0] = 2.0 ** -24
    rows.append(lo)                     # one subnormal step
    mix = np.linspace(-1, 1, G)
    mix[7] = -0.0
    mix[9] = 0.0
    rows.append(mix)
    return _f16(np.array(rows))


def all_groups(G, n_each, seed):
    rng = np.random.default_rng(seed)
    return np.concatenate([gaussian_groups(rng, n_each, G), outlier_groups(rng, n_each // 4, G),
                           tie_groups(rng, n_each // 4, G),
                           subnormal_scale_groups(rng, n_each // 8, G), special_groups(G)])


def _compare(codes, scales, biases, tc, ts, tb):
    bad_c = np.any(codes != tc, axis=1)
    bad_s = scales.view(np.uint16) != ts.view(np.uint16)
    bad_b = biases.view(np.uint16) != tb.view(np.uint16)
    return bad_c | bad_s | bad_b


# ------------------------------------------------------- the twin's own pins
def test_twin_fp16_rounding_matches_numpy_nearest_and_directed_definition():
    """The twin's nearest rounding equals numpy's conversion; its directed
    roundings are the neighbours that bracket the value."""
    rng = np.random.default_rng(7)
    e = rng.integers(127 - 30, 127 + 17, size=200000)
    m = rng.integers(0, 1 << 23, size=200000)
    s = rng.integers(0, 2, size=200000)
    f = ((s << 31) | (e << 23) | m).astype(np.uint32).view(np.float32)
    h = rng.integers(0, 0x7BFF, size=50000).astype(np.uint16)
    ties = ((h.view(np.float16).astype(np.float64) +
             (h + 1).astype(np.uint16).view(np.float16).astype(np.float64)) / 2).astype(np.float32)
    f = np.concatenate([f, ties, -ties, np.float32([65519, 65520, 65504, 2 ** -25, 0.0, -0.0])])
    near = round_f32_to_f16(f, "even")
    with np.errstate(over="ignore"):
        ref = f.astype(np.float16)
    assert np.array_equal(near.view(np.uint16), ref.view(np.uint16))
    dn = round_f32_to_f16(f, "down").astype(np.float64)
    up = round_f32_to_f16(f, "up").astype(np.float64)
    fd = f.astype(np.float64)
    fin = np.abs(fd) <= 65504
    assert np.all(dn[fin] <= fd[fin]) and np.all(up[fin] >= fd[fin])
    # neighbours: no fp16 strictly between
    with np.errstate(over="ignore"):
        nxt_dn = np.nextafter(dn[fin].astype(np.float16), np.float16(np.inf)).astype(np.float64)
    assert np.all((dn[fin] == fd[fin]) | (nxt_dn > fd[fin]))
    nxt_up = np.nextafter(up[fin].astype(np.float16), np.float16(-np.inf)).astype(np.float64)
    assert np.all((up[fin] == fd[fin]) | (nxt_up < fd[fin]))


def test_twin_ties_round_half_even():
    x = _f16([[0, 15, 0.5, 1.5, 2.5, 3.5] + [0] * 58])
    codes, scale, bias = twin_quantize(x)
    assert float(scale[0]) == 1.0 and float(bias[0]) == 0.0
    assert list(codes[0, :6]) == [0, 15, 0, 2, 2, 4]


# ------------------------------------------------------- oracle == twin
@pytest.mark.parametrize("G,n_each", [(64, 800000), (32, 100000), (128, 50000)])
def test_oracle_quantizer_equals_twin_bitwise(G, n_each):
    x = all_groups(G, n_each, seed=G)
    codes, scales, biases = oracle.quantize_groups(x)
    tc, ts, tb = twin_quantize(x)
    bad = _compare(codes, scales, biases, tc, ts, tb)
    assert not bad.any(), "%d of %d groups differ, first %d: %r" % (
        bad.sum(), len(bad), np.argmax(bad), x[np.argmax(bad)])
    # the data really exercised the cases it claims to
    assert np.any(scales.view(np.uint16) == 0)                               # constant groups
    assert np.any((scales.view(np.uint16) > 0) & (scales.view(np.uint16) < 0x0400))  # subnormal
    assert np.any(biases.view(np.uint16) == 0x8000)                          # -0 bias


# ------------------------------------------------------- planted mistakes
MUTANTS = {
    "reciprocal": (r"volatile float r = diff / sf;", "volatile float r = diff * (1.0f / sf);"),
    "ties_up": (r"float q = rintf\(r\);", "float q = floorf(r + 0.5f);"),
    "scale_nearest": (r"jfo_float_to_half\(step, 2\)", "jfo_float_to_half(step, 0)"),
    "signed_zero": (r"\(v == mn && signbit\(v\) && !signbit\(mn\)\)", "0"),
}


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("oracle_mutants")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, mutant_dir):
    pat, rep = MUTANTS[name]
    src = open(os.path.join(os.path.dirname(HERE), "oracle", "jf_oracle.c")).read()
    assert len(re.findall(pat, src)) == 1, "mutation site not found: " + name
    mutated = re.sub(pat, lambda _: rep, src)
    cdir = mutant_dir / name
    cdir.mkdir()
    (cdir / "jf_oracle.c").write_text(mutated)
    import shutil
    shutil.copy(os.path.join(os.path.dirname(HERE), "oracle", "jf_oracle.h"), cdir / "jf_oracle.h")
    so = str(cdir / "libmutant.so")
    subprocess.run(["gcc", *oracle.CFLAGS, str(cdir / "jf_oracle.c"), "-o", so, "-lm"], check=True)
    lib = ctypes.CDLL(so)
    lib.jfo_quantize_groups.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    x = all_groups(64, 100000, seed=11)
    n, G = x.shape
    codes = np.zeros((n, G), np.uint8)
    s = np.zeros(n, np.uint16)
    b = np.zeros(n, np.uint16)
    xu = np.ascontiguousarray(x).view(np.uint16)
    lib.jfo_quantize_groups(xu.ctypes.data, n, G, codes.ctypes.data, s.ctypes.data, b.ctypes.data)
    tc, ts, tb = twin_quantize(x)
    bad = _compare(codes, s.view(np.float16), b.view(np.float16), tc, ts, tb)
    assert bad.sum() > 0, "planted mistake %r not detected" % name
