"""Pins of the oracle's page -> operand reconstruction (oracle.reconstruct)
and of its binary64 -> binary16 rounding (oracle.double_to_half).

Independent checks: numpy's float64 -> float16 conversion (its own
implementation of round-to-nearest-even) and the dequantized vectors of
oracle.dequant_vector (pinned in test_oracle_layout / test_oracle_attention).
Crafted meta words put s * q + b just off a binary16 midpoint, where rounding
through binary32 first (the plain fp32 FMA path) gives the other neighbour:
the oracle must match the exact rounding there, and the test checks that the
double-rounding variant would fail it."""
import numpy as np
import pytest

import oracle
from paper_2609_17475_amd import workloads


def _f16_values():
    bits = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
    v = bits.view(np.float16).astype(np.float64)
    return v[np.isfinite(v)]


def test_double_to_half_matches_numpy():
    rng = np.random.default_rng(0)
    fin = np.unique(_f16_values())
    pos = fin[fin >= 0]
    mids = (pos[:-1] + pos[1:]) / 2                      # exact ties
    near = np.concatenate([np.nextafter(mids, np.inf), np.nextafter(mids, -np.inf)])
    rand = np.concatenate([rng.uniform(-70000, 70000, 20000),
                           rng.uniform(-1e-4, 1e-4, 20000),
                           rng.standard_normal(20000) * 10])
    edge = np.array([65504.0, 65519.99999, 65520.0, 65520.00001, 1e6, -65520.0,
                     2.0 ** -25, 2.0 ** -25 * 3, 2.0 ** -26, 0.0, -0.0])
    xs = np.concatenate([fin, mids, -mids, near, -near, rand, edge])
    got = np.array([oracle.double_to_half(float(x)) for x in xs], np.uint16)
    want = xs.astype(np.float16).view(np.uint16)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "first mismatch x=%r got %04x want %04x" % (
        xs[bad[0]], got[bad[0]], want[bad[0]])


def _pool(P, hkv, d, G, L, seed, NP=None):
    NP = NP or -(-L // P) + 2
    pool = oracle.Pool(oracle.layout(P, hkv, d, G, NP))
    perm = np.random.default_rng(seed).permutation(NP).astype(np.int32)
    table = perm[: -(-L // P)]
    k, v = workloads.gen_kv(seed, L, hkv, d, 2)
    oracle.quantize_append(pool, k, v, [0, L], [0], table[None])
    return pool, table


@pytest.mark.parametrize("P,hkv,d,G,L,kv0,g", [(32, 4, 128, 64, 100, 0, 2), (32, 4, 128, 64, 100, 2, 2),
                                               (64, 2, 64, 32, 65, 1, 1), (16, 3, 256, 128, 40, 0, 3)])
def test_reconstruct_is_rounded_dequant(P, hkv, d, G, L, kv0, g):
    pool, table = _pool(P, hkv, d, G, L, seed=L + d)
    k16, v16 = oracle.reconstruct(pool, table, L, kv0, g)
    for j in range(g):
        for t in range(L):
            page, slot = int(table[t // P]), t % P
            for is_v, out in ((False, k16), (True, v16)):
                x = oracle.dequant_vector(pool, is_v, page, kv0 + j, slot)
                assert np.array_equal(out[j, t].view(np.uint16), x.astype(np.float16).view(np.uint16))


def test_reconstruct_invalid_page_gives_zeros():
    pool, table = _pool(32, 1, 64, 32, 96, seed=3)
    t2 = table.copy()
    t2[1] = -1
    k16, v16 = oracle.reconstruct(pool, t2, 96, 0, 1)
    assert not np.any(k16[0, 32:64].view(np.uint16)) and not np.any(v16[0, 32:64].view(np.uint16))
    k_ref, _ = oracle.reconstruct(pool, table, 96, 0, 1)
    assert np.array_equal(k16[0, :32], k_ref[0, :32]) and np.array_equal(k16[0, 64:], k_ref[0, 64:])


def double_rounding_cases(n, seed=0):
    """(scale bits, code, bias bits) with finite fp16 scale >= 0 and bias,
    where rounding s*q + b through float32 first differs from rounding the
    exact value (found by a seeded search; numpy evaluates both)."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        s = rng.integers(0x0400, 0x7800, 200000).astype(np.uint16)
        c = rng.integers(1, 16, 200000)
        # tiny or small biases make the float32 sum inexact
        b = rng.choice(np.array([0x0001, 0x8001, 0x0002, 0x8002, 0x0003, 0x8003, 0x03ff, 0x83ff,
                                 0x0401, 0x8401, 0x2001, 0xa001], np.uint16), 200000)
        sv = s.view(np.float16).astype(np.float64)
        bv = b.view(np.float16).astype(np.float64)
        ex = sv * c + bv
        ok = np.isfinite(ex) & (np.abs(ex) < 65504)
        direct = ex.astype(np.float16).view(np.uint16)
        via32 = ex.astype(np.float32).astype(np.float16).view(np.uint16)
        hit = np.nonzero(ok & (direct != via32))[0]
        out += [(int(s[i]), int(c[i]), int(b[i])) for i in hit[: n - len(out)]]
    return out


def write_crafted(pool, table, cases, kv=0):
    """Put case i at group 0 of logical position i (page table[i // P],
    slot i % P): meta (scale, bias) and every code of the group = q."""
    lay = pool.layout
    P, d, G, hkv = lay.page_size, lay.head_dim, lay.group_size, lay.num_kv_heads
    meta = pool.k_meta.reshape(lay.num_pages, hkv, P, d // G, 2)
    codes = pool.k_codes.reshape(lay.num_pages, hkv, P, d // 2)
    for i, (sb, q, bb) in enumerate(cases):
        page, slot = int(table[i // P]), i % P
        meta[page, kv, slot, 0] = (sb, bb)
        codes[page, kv, slot, : G // 2] = q | (q << 4)


def test_reconstruct_exact_rounding_near_midpoints():
    pool, table = _pool(32, 1, 64, 32, 96, seed=4)
    cases = double_rounding_cases(96)
    write_crafted(pool, table, cases)
    k16, _ = oracle.reconstruct(pool, table, 96, 0, 1)
    via32 = []
    for i, (sb, q, bb) in enumerate(cases):
        s = float(np.uint16(sb).view(np.float16))
        b = float(np.uint16(bb).view(np.float16))
        exact = s * q + b
        got = k16[0, i, :32].view(np.uint16)
        assert np.all(got == np.float16(exact).view(np.uint16)), i
        via32.append(np.float16(np.float32(exact)).view(np.uint16))
    # the float32-first variant fails this test on every case
    assert all(v != k16[0, i, 0].view(np.uint16) for i, v in enumerate(via32))
