"""Pins of the TQ4 oracle (oracle/tq4.py) against facts other than itself.

Codebook: an independent continuous Lloyd-Max solver (closed-form cell masses
and first moments of the sphere-coordinate density through the regularised
incomplete beta function, no grid) is checked against Max's printed 16-level
Gaussian table in the large-d limit; the grid construction's start and
update are then checked against it (within one grid spacing, shrinking with
the spacing) and its codebooks against its distortion.  Rotation: the library Hadamard
matrix and orthogonality.  Quantization: brute-force nearest centroid.
Round trip: the expected distortion of a uniform point on the sphere equals d
times the codebook's integrated distortion.  Storage: the paper's printed
payload figures.  Attention: closed-form special cases and the rotate-the-
query-once identity that a page-native kernel relies on.
"""
import json
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.special
import scipy.stats

from oracle import tq4

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tq4_payload.json")


# ---- independent continuous Lloyd-Max solvers (no grid) ----------------------

def _sphere_moments(a, b, d):
    """Mass and first moment over [a, b] of (1 - x^2)^k, k = (d - 3)/2, in
    closed form: mass via the regularised incomplete beta function of x^2,
    first moment via the antiderivative -(1 - x^2)^(k + 1) / (2 (k + 1))."""
    k = (d - 3) / 2.0

    def cum(x):  # integral from 0 to x, odd in x
        return np.sign(x) * 0.5 * scipy.special.beta(0.5, k + 1) * scipy.special.betainc(0.5, k + 1, x * x)

    mass = cum(b) - cum(a)
    first = (-(1 - b * b) ** (k + 1) + (1 - a * a) ** (k + 1)) / (2 * (k + 1))
    return mass, first


def _sphere_lloyd(d, iters=20000):
    """Fixed point of Lloyd's conditions for the sphere-coordinate density."""
    c = scipy.stats.norm.ppf((np.arange(16) + 0.5) / 16) / np.sqrt(d)
    for _ in range(iters):
        e = np.concatenate([[-1.0], 0.5 * (c[:-1] + c[1:]), [1.0]])
        mass, first = _sphere_moments(e[:-1], e[1:], d)
        new = first / mass
        if np.max(np.abs(new - c)) < 1e-15:
            break
        c = new
    return c


def _gauss_lloyd(iters=20000):
    """Fixed point of Lloyd's conditions for N(0, 1): the centroid of a cell
    (a, b) is (phi(a) - phi(b)) / (Phi(b) - Phi(a))."""
    c = scipy.stats.norm.ppf((np.arange(16) + 0.5) / 16)
    for _ in range(iters):
        e = np.concatenate([[-np.inf], 0.5 * (c[:-1] + c[1:]), [np.inf]])
        new = (scipy.stats.norm.pdf(e[:-1]) - scipy.stats.norm.pdf(e[1:])) / (
            scipy.stats.norm.cdf(e[1:]) - scipy.stats.norm.cdf(e[:-1]))
        if np.max(np.abs(new - c)) < 1e-14:
            break
        c = new
    return c


def _sphere_distortion(c, d):
    """d x the mean squared error of quantizing one sphere coordinate with
    centroids c and midpoint cells, integrated in closed form (second
    moment through the beta function as well)."""
    c = np.asarray(c, np.float64)
    e = np.concatenate([[-1.0], 0.5 * (c[:-1] + c[1:]), [1.0]])
    mass, first = _sphere_moments(e[:-1], e[1:], d)
    # second moment: x^2 (1 - x^2)^k = (1 - x^2)^k - (1 - x^2)^(k + 1), and
    # (1 - x^2)^(k + 1) is the density for d + 2
    m_k1, _ = _sphere_moments(e[:-1], e[1:], d + 2)
    second = mass - m_k1
    total, _ = _sphere_moments(-1.0, 1.0, d)
    return d * np.sum(second - 2 * c * first + c * c * mass) / total


# ---- codebook ------------------------------------------------------------------

def test_gaussian_solver_matches_max_table():
    # J. Max, "Quantizing for minimum distortion", IRE Trans. Inf. Theory
    # (1960), Table I, N = 16: the positive output levels of the MSE-optimal
    # quantizer for a unit normal input.
    printed = [0.1284, 0.3881, 0.6568, 0.9424, 1.2562, 1.6180, 2.0690, 2.7326]
    g = _gauss_lloyd()
    np.testing.assert_allclose(g[8:], printed, atol=1.5e-4)
    np.testing.assert_allclose(g[:8], -g[8:][::-1], atol=1e-12)


def test_sphere_solver_tends_to_gaussian():
    # a coordinate of a uniform point on the sphere in d dimensions times
    # sqrt(d) tends to N(0, 1)
    g = _gauss_lloyd()
    s = _sphere_lloyd(1 << 22) * np.sqrt(1 << 22)
    np.testing.assert_allclose(s, g, atol=2e-5)


def _lloyd_step(c, d):
    """One continuous Lloyd update: each centroid to the mean of its cell."""
    e = np.concatenate([[-1.0], 0.5 * (c[:-1] + c[1:]), [1.0]])
    mass, first = _sphere_moments(e[:-1], e[1:], d)
    return first / mass


def _quantiles(d):
    """Continuous (i + 1/2)/16 quantiles of the density, by inverting the
    regularised incomplete beta function."""
    k = (d - 3) / 2.0
    p = (np.arange(16) + 0.5) / 16
    return np.sign(p - 0.5) * np.sqrt(scipy.special.betaincinv(0.5, k + 1, np.abs(2 * p - 1)))


@pytest.mark.parametrize("d", [64, 128, 256])
def test_grid_start_and_update_follow_the_density(d):
    # the start is a grid point next to each continuous quantile, and one
    # grid update is the continuous Lloyd update up to the grid: both within
    # one grid spacing h, and the update error shrinks with h (8x finer grid)
    h = 2.0 / (tq4.GRID_POINTS - 1)
    c0, n0 = tq4.codebook(d, max_updates=0)
    assert n0 == 0
    assert np.max(np.abs(c0 - _quantiles(d))) <= h
    c1, _ = tq4.codebook(d, max_updates=1, stop=0.0)
    assert np.max(np.abs(c1 - _lloyd_step(c0.astype(np.float64), d))) <= h
    fine = 8 * tq4.GRID_POINTS
    f0, _ = tq4.codebook(d, grid=fine, max_updates=0)
    f1, _ = tq4.codebook(d, grid=fine, max_updates=1, stop=0.0)
    assert np.max(np.abs(f1 - _lloyd_step(f0.astype(np.float64), d))) <= h / 8


@pytest.mark.parametrize("d", [64, 128, 256])
def test_grid_fixed_point_distortion(d):
    # run to convergence, the grid construction reaches the continuous
    # Lloyd-Max distortion: its O(h) bias per update moves the fixed point by
    # ~1-2 % (Lloyd contracts slowly here, ~0.965 per update), which costs
    # distortion only to second order
    c, _ = tq4.codebook(d, max_updates=5000, stop=0.0)
    ref = _sphere_lloyd(d)
    assert _sphere_distortion(c, d) <= _sphere_distortion(ref, d) * 1.0005


@pytest.mark.parametrize("d", [64, 128, 256])
def test_paper_codebook_near_optimal(d):
    c, n = tq4.codebook(d)
    assert c.dtype == np.float32 and c.shape == (16,)
    assert 1 <= n <= tq4.MAX_UPDATES
    assert np.all(np.diff(c) > 0) and np.all(np.abs(c) < 1)
    np.testing.assert_array_equal(c, -c[::-1])  # symmetric grid and start keep it symmetric
    ref = _sphere_lloyd(d)
    # 100 updates from the quantile start: within 3 % of the optimum's
    # centroids and 0.1 % of its distortion
    assert np.max(np.abs(c - ref) / np.abs(ref)) < 3e-2
    assert _sphere_distortion(c, d) <= _sphere_distortion(ref, d) * 1.001


def test_stop_rule_ends_early_when_change_is_small():
    # a loose stop threshold ends the updates early; a zero one never does
    _, n_loose = tq4.codebook(256, stop=1e-3)
    _, n_none = tq4.codebook(256, max_updates=7, stop=0.0)
    assert n_loose < tq4.MAX_UPDATES and n_none == 7


# ---- rotation and signs --------------------------------------------------------

@pytest.mark.parametrize("d", [2, 8, 64, 256])
def test_hadamard_is_sylvester(d):
    np.testing.assert_array_equal(tq4.hadamard(d), scipy.linalg.hadamard(d))
    h = tq4.hadamard(d)
    np.testing.assert_array_equal(h @ h.T, d * np.eye(d))


def test_rotation_orthogonal_and_norm_preserving():
    d = 256
    s = tq4.signs(d, tq4.K_SEED)
    r = tq4.rotation(d, s)
    np.testing.assert_allclose(r @ r.T, np.eye(d), atol=1e-12)
    x = np.random.default_rng(7).standard_normal((5, d))
    np.testing.assert_allclose(np.linalg.norm(x @ r.T, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)
    # a coordinate spike spreads to equal magnitudes 1/sqrt(d)
    e = np.zeros((1, d)); e[0, 37] = 1.0
    np.testing.assert_allclose(np.abs(e @ r.T), np.full((1, d), 1 / 16), atol=1e-15)


def test_signs():
    for d in (64, 256):
        sk, sv = tq4.signs(d, tq4.K_SEED), tq4.signs(d, tq4.V_SEED)
        assert sk.shape == (d,) and set(np.unique(sk)) <= {-1.0, 1.0}
        assert not np.array_equal(sk, sv)
        np.testing.assert_array_equal(sk, tq4.signs(d, tq4.K_SEED))
    assert not np.array_equal(tq4.signs(64, 0)[:64], tq4.signs(256, 0)[:64])


# ---- encoding -------------------------------------------------------------------

def _brute_nearest(y, c):
    """Index of the nearest centroid by scanning all 16 (the lower index on a
    tie, which is what a strict comparison with the midpoint gives)."""
    dist = np.abs(y[..., None] - c.astype(np.float64)[None, None, :])
    return np.argmin(dist, axis=-1)


def test_indices_are_nearest_centroids():
    d = 256
    c, _ = tq4.codebook(d)
    s = tq4.signs(d, tq4.K_SEED)
    x = np.random.default_rng(1).standard_normal((300, d)).astype(np.float16)
    x[0] = 0
    x[1, :] = 0; x[1, 5] = -3.0
    idx, norm16, y = tq4.encode(x, s, c)
    assert idx.dtype == np.uint8 and idx.max() <= 15
    np.testing.assert_array_equal(idx[2:], _brute_nearest(y[2:], c))
    # unit rotated vectors, except the zero vector
    np.testing.assert_allclose(np.linalg.norm(y[1:], axis=1), 1.0, rtol=1e-6)
    assert norm16[0] == 0 and np.all(y[0] == 0)
    # the fp16 norm is the float32 norm rounded
    ref = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=1)).astype(np.float32).astype(np.float16)
    np.testing.assert_array_equal(norm16, ref)


def test_norm_is_rounded_through_float32():
    # a norm just above an fp16 midpoint that float32 rounds onto the midpoint:
    # from the float32 norm the tie goes to even (1.0); rounding the exact
    # norm directly would give 1 + 2^-10
    a = 1.0 + 2.0 ** -11 + 2.0 ** -30
    c, _ = tq4.codebook(2)
    _, n16, _ = tq4.encode(np.array([[a, 0.0], [0.0, -a]]), tq4.signs(2, 0), c)
    assert n16.tolist() == [1.0, 1.0]
    assert np.float16(a) == np.float16(1.0 + 2.0 ** -10)


def test_threshold_ties_go_down():
    c, _ = tq4.codebook(256)
    t = tq4.thresholds(c)
    # a coordinate exactly on a threshold keeps the lower index, a hair above it
    # takes the upper one; the centroids themselves map to their own index
    for j in (0, 7, 14):
        y = np.array([[t[j], np.nextafter(t[j], 2.0)]])
        assert list(tq4.quantize(y, c)[0]) == [j, j + 1]
    np.testing.assert_array_equal(tq4.quantize(c.astype(np.float64)[None], c)[0], np.arange(16))
    assert tq4.quantize(np.array([[-1.0, 1.0]]), c).tolist() == [[0, 15]]


def test_pack_bit_order():
    idx = np.tile(np.arange(16, dtype=np.uint8), 2)[None, :]  # 0..15, 0..15
    w = tq4.pack(idx)
    assert list(w[0]) == [0x76543210, 0xFEDCBA98, 0x76543210, 0xFEDCBA98]
    r = np.random.default_rng(3).integers(0, 16, (4, 256)).astype(np.uint8)
    np.testing.assert_array_equal(tq4.unpack(tq4.pack(r)), r)


def test_round_trip_distortion_matches_codebook():
    # for x Gaussian, x / |x| is uniform on the sphere and so is its rotation:
    # E |x - x_hat|^2 / |x|^2 = d x the per-coordinate distortion (plus the
    # fp16 norm rounding, < 1e-6 here)
    d = 256
    c, _ = tq4.codebook(d)
    s = tq4.signs(d, tq4.V_SEED)
    x = np.random.default_rng(11).standard_normal((4000, d))
    idx, norm16, _ = tq4.encode(x, s, c)
    xh = tq4.reconstruct(idx, norm16, s, c)
    rel = np.sum((x - xh) ** 2, axis=1) / np.sum(x * x, axis=1)
    expect = _sphere_distortion(c, d)
    assert abs(rel.mean() - expect) < 0.02 * expect, (rel.mean(), expect)


def test_payload_matches_paper():
    g = json.load(open(GOLDEN))
    d = g["head_dim"]
    assert tq4.vector_bytes(d) == g["bytes_per_vector"]
    per_pos = g["layers"] * 2 * g["kv_heads"] * tq4.vector_bytes(d)
    assert per_pos == g["bytes_per_position"]
    for n, mib in g["history_mib"].items():
        assert int(n) * per_pos == mib * 2 ** 20
    assert round(100 * tq4.vector_bytes(d) / (2 * d), 1) == g["percent_of_fp16"]


# ---- attention over TQ4 vectors -------------------------------------------------

def _random_cache(L, hkv, d, seed, c):
    rng = np.random.default_rng(seed)
    sk, sv = tq4.signs(d, tq4.K_SEED), tq4.signs(d, tq4.V_SEED)
    out = []
    for s in (sk, sv):
        x = rng.standard_normal((L * hkv, d)).astype(np.float16)
        idx, n16, _ = tq4.encode(x, s, c)
        out += [tq4.pack(idx).reshape(L, hkv, d // 8), n16.reshape(L, hkv)]
    return out, sk, sv


def test_attention_special_cases():
    d, hkv, hq = 256, 4, 24
    c, _ = tq4.codebook(d)
    (kw, kn, vw, vn), sk, sv = _random_cache(6, hkv, d, 5, c)
    q = np.random.default_rng(6).standard_normal((hq, d)) / 16
    # one position: the output is that position's reconstructed value
    o = tq4.decode_attention(q, kw[:1], kn[:1], vw[:1], vn[:1], sk, sv, c, 1.0)
    for h in range(hq):
        v0 = tq4.reconstruct(tq4.unpack(vw[0, h // 6][None]), vn[0, h // 6][None], sv, c)[0]
        np.testing.assert_allclose(o[h], v0, rtol=0, atol=1e-12)
    # identical keys: the mean of the values
    kw2, kn2 = np.repeat(kw[:1], 6, axis=0), np.repeat(kn[:1], 6, axis=0)
    o = tq4.decode_attention(q, kw2, kn2, vw, vn, sk, sv, c, 1.0)
    for h in range(hq):
        vh = tq4.reconstruct(tq4.unpack(vw[:, h // 6]), vn[:, h // 6], sv, c)
        np.testing.assert_allclose(o[h], vh.mean(axis=0), rtol=0, atol=1e-12)


def test_rotated_query_identity():
    # q . x_hat = rho_hat (R q) . c[z]: a kernel may rotate the query once
    # and sum centroid values, and likewise rotate the summed values once
    d = 256
    c, _ = tq4.codebook(d)
    s = tq4.signs(d, tq4.K_SEED)
    x = np.random.default_rng(8).standard_normal((50, d))
    idx, n16, _ = tq4.encode(x, s, c)
    q = np.random.default_rng(9).standard_normal(d)
    direct = tq4.reconstruct(idx, n16, s, c) @ q
    rq = tq4.rotation(d, s) @ q
    via = n16.astype(np.float64) * (c.astype(np.float64)[idx] @ rq)
    np.testing.assert_allclose(direct, via, rtol=1e-12, atol=1e-12)
    p = np.random.default_rng(10).random(50)
    np.testing.assert_allclose(p @ tq4.reconstruct(idx, n16, s, c),
                               tq4.rotation(d, s).T @ ((p * n16.astype(np.float64)) @ c.astype(np.float64)[idx]),
                               rtol=1e-12, atol=1e-12)


def test_gather_follows_table():
    NP, hkv, P, d = 5, 2, 4, 64
    rng = np.random.default_rng(12)
    words = rng.integers(0, 2 ** 32, (NP, hkv, P, d // 8), dtype=np.uint64).astype(np.uint32)
    norms = rng.standard_normal((NP, hkv, P)).astype(np.float16)
    table = np.array([3, 0, 4])
    w, n = tq4.gather(words, norms, table, 10)
    for t in range(10):
        np.testing.assert_array_equal(w[t], words[table[t // P], :, t % P])
        np.testing.assert_array_equal(n[t], norms[table[t // P], :, t % P])
