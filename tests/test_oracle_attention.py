"""Pins for the oracle's decode and prefill attention (CPU only).

Attention over the dequantized cache is plain softmax attention (Sec. 3.1,
"Decode and prefill need different kernels"; heads are independent,
eq. groupattention), so it is pinned to torch's float64 scaled-dot-product
attention (an independent library routine) on inputs whose quantization is
exact, to closed-form special cases, and to invariants (page order, head
independence, ragged batches, causality).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_17475_amd import workloads

torch.set_num_threads(4)


def exact_grid_rows(rng, n, hkv, d, G):
    """fp16 rows whose groups are bias + s*c with a power-of-two s and codes
    containing 0 and 15, so the 4-bit round trip reproduces them exactly."""
    x = np.empty((n, hkv, d), np.float64)
    for r in range(n):
        for h in range(hkv):
            for g in range(d // G):
                s = 2.0 ** int(rng.integers(-5, 0))
                b = float(rng.integers(-40, 10)) * s
                c = rng.integers(0, 16, size=G)
                c[rng.permutation(G)[:2]] = (0, 15)
                x[r, h, g * G:(g + 1) * G] = b + s * c
    x16 = x.astype(np.float16)
    assert np.array_equal(x16.astype(np.float64), x)
    return x16


def sdpa_ref(q, K, V, alpha, mask=None):
    """q [Hq][d] (or [T][Hq][d]); K, V [n][Hkv][d]; float64 torch SDPA."""
    qt = torch.from_numpy(np.asarray(q, np.float64))
    if qt.dim() == 2:
        qt = qt[None]
    T, Hq, d = qt.shape
    Hkv = K.shape[1]
    gq = Hq // Hkv
    Kt = torch.from_numpy(np.asarray(K, np.float64)).permute(1, 0, 2)
    Vt = torch.from_numpy(np.asarray(V, np.float64)).permute(1, 0, 2)
    Kt = Kt.repeat_interleave(gq, dim=0)
    Vt = Vt.repeat_interleave(gq, dim=0)
    o = torch.nn.functional.scaled_dot_product_attention(
        qt.permute(1, 0, 2), Kt, Vt, attn_mask=mask, scale=alpha)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("P,hkv,hq,d,G,n", [(4, 1, 4, 64, 64, 13), (8, 2, 8, 64, 32, 40),
                                            (256, 1, 2, 128, 64, 300), (4, 2, 6, 32, 32, 9)])
def test_decode_matches_sdpa_on_exact_grid(P, hkv, hq, d, G, n):
    rng = np.random.default_rng(P * 100 + n)
    n_pages = -(-n // P)
    NP = n_pages + 3
    lay = oracle.layout(P, hkv, d, G, NP)
    k = exact_grid_rows(rng, n, hkv, d, G)
    v = exact_grid_rows(rng, n, hkv, d, G)
    table = rng.permutation(NP)[:n_pages].astype(np.int32)
    pool = oracle.Pool(lay)
    oracle.quantize_append(pool, k, v, [0, n], [0], table[None])
    q = (rng.standard_normal((1, hq, d)) * 0.3).astype(np.float16)
    out = oracle.decode(pool, q, table[None], [n], alpha=0.7)
    ref = sdpa_ref(q[0].astype(np.float64), k, v, 0.7)[0]
    np.testing.assert_allclose(out[0], ref, rtol=1e-12, atol=1e-12)


def test_decode_random_inputs_matches_sdpa_over_dequantized_rows():
    rng = np.random.default_rng(11)
    P, hkv, hq, d, G, n = 8, 2, 8, 128, 64, 61
    lay = oracle.layout(P, hkv, d, G, 10)
    k, v = workloads.gen_kv(5, n, hkv, d, 3)
    table = np.array([9, 3, 0, 7, 2, 5, 1, 8], np.int32)
    pool = oracle.Pool(lay)
    oracle.quantize_append(pool, k, v, [0, n], [0], table[None])
    Kd = np.array([[oracle.dequant_vector(pool, False, int(table[t // P]), h, t % P)
                    for h in range(hkv)] for t in range(n)])
    Vd = np.array([[oracle.dequant_vector(pool, True, int(table[t // P]), h, t % P)
                    for h in range(hkv)] for t in range(n)])
    # dequantized rows stay within half a scale of the fp16 inputs
    assert np.max(np.abs(Kd - k.astype(np.float64))) < 2.0
    q = (rng.standard_normal((1, hq, d)) / np.sqrt(d)).astype(np.float16)
    out = oracle.decode(pool, q, table[None], [n], alpha=1.0)
    ref = sdpa_ref(q[0].astype(np.float64), Kd, Vd, 1.0)[0]
    np.testing.assert_allclose(out[0], ref, rtol=1e-12, atol=1e-13)


def _pool_with(rng, P, hkv, d, G, k, v, NP=None):
    n = k.shape[0]
    n_pages = -(-n // P)
    NP = NP or n_pages + 2
    lay = oracle.layout(P, hkv, d, G, NP)
    table = rng.permutation(NP)[:n_pages].astype(np.int32)
    pool = oracle.Pool(lay)
    oracle.quantize_append(pool, k, v, [0, n], [0], table[None])
    return pool, table


def test_single_position_returns_its_value():
    rng = np.random.default_rng(12)
    k, v = workloads.gen_kv(6, 1, 1, 64, 2)
    pool, table = _pool_with(rng, 4, 1, 64, 32, k, v)
    q = (rng.standard_normal((1, 3, 64))).astype(np.float16)
    out = oracle.decode(pool, q, table[None], [1], alpha=1.0)
    vhat = oracle.dequant_vector(pool, True, int(table[0]), 0, 0)
    for h in range(3):
        assert np.array_equal(out[0, h], vhat)


def test_identical_keys_give_mean_of_values():
    rng = np.random.default_rng(13)
    n, d = 37, 64
    k = np.repeat(rng.standard_normal((1, 1, d)).astype(np.float16), n, axis=0)
    v = rng.standard_normal((n, 1, d)).astype(np.float16)
    pool, table = _pool_with(rng, 8, 1, d, 64, k, v)
    q = rng.standard_normal((1, 2, d)).astype(np.float16)
    out = oracle.decode(pool, q, table[None], [n], alpha=1.0)
    vhat = np.array([oracle.dequant_vector(pool, True, int(table[t // 8]), 0, t % 8)
                     for t in range(n)])
    np.testing.assert_allclose(out[0, 0], vhat.mean(0), rtol=0, atol=1e-14)
    np.testing.assert_allclose(out[0, 1], vhat.mean(0), rtol=0, atol=1e-14)


def test_dominant_logit_returns_needle_value():
    rng = np.random.default_rng(14)
    n, d = 50, 64
    k, v = workloads.gen_kv(7, n, 1, d, 0)
    t_star = 23
    pool, table = _pool_with(rng, 8, 1, d, 64, k, v)
    kh = oracle.dequant_vector(pool, False, int(table[t_star // 8]), 0, t_star % 8)
    q = (kh / np.linalg.norm(kh) * 8.0)[None, None, :].astype(np.float16)
    out = oracle.decode(pool, q, table[None], [n], alpha=10.0)
    vhat = oracle.dequant_vector(pool, True, int(table[t_star // 8]), 0, t_star % 8)
    np.testing.assert_allclose(out[0, 0], vhat, atol=1e-6)


def test_physical_page_permutation_is_bitwise_invariant():
    rng = np.random.default_rng(15)
    P, hkv, hq, d, G, n = 4, 2, 4, 64, 32, 22
    k, v = workloads.gen_kv(8, n, hkv, d, 2)
    q = rng.standard_normal((1, hq, d)).astype(np.float16)
    outs = []
    for seed in (1, 2, 3):
        pool, table = _pool_with(np.random.default_rng(seed), P, hkv, d, G, k, v, NP=12)
        outs.append(oracle.decode(pool, q, table[None], [n], alpha=0.5))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_query_heads_are_independent():
    rng = np.random.default_rng(16)
    P, hkv, hq, d, G, n = 8, 2, 8, 64, 64, 30
    k, v = workloads.gen_kv(9, n, hkv, d, 2)
    pool, table = _pool_with(rng, P, hkv, d, G, k, v)
    q = rng.standard_normal((1, hq, d)).astype(np.float16)
    perm = np.array([2, 0, 3, 1, 7, 5, 4, 6])  # permutes within each KV group
    o1 = oracle.decode(pool, q, table[None], [n], 1.0)
    o2 = oracle.decode(pool, q[:, perm], table[None], [n], 1.0)
    assert np.array_equal(o1[:, perm], o2)


def test_ragged_batch_equals_requests_alone_with_shared_prefix():
    rng = np.random.default_rng(17)
    P, hkv, hq, d, G = 4, 1, 2, 64, 32
    NP = 20
    lay = oracle.layout(P, hkv, d, G, NP)
    pool = oracle.Pool(lay)
    pre = 8  # two shared pages
    lens = [8 + 9, 8 + 3]
    k, v = workloads.gen_kv(10, 8 + 9 + 3, hkv, d, 1)
    tables = np.full((2, 5), -1, np.int32)
    tables[0, :5] = [6, 2, 11, 13, 4]
    tables[1, :3] = [6, 2, 9]
    oracle.quantize_append(pool, k[:pre], v[:pre], [0, pre], [0], tables[:1])
    oracle.quantize_append(pool, k[pre:], v[pre:], [0, 9, 12], [pre, pre], tables)
    q = rng.standard_normal((2, hq, d)).astype(np.float16)
    both = oracle.decode(pool, q, tables, lens, 1.0)
    a = oracle.decode(pool, q[:1], tables[:1], lens[:1], 1.0)
    b = oracle.decode(pool, q[1:], tables[1:], lens[1:], 1.0)
    assert np.array_equal(both[0], a[0]) and np.array_equal(both[1], b[0])


def test_decode_rejects_empty_sequence():
    rng = np.random.default_rng(18)
    k, v = workloads.gen_kv(11, 3, 1, 32, 0)
    pool, table = _pool_with(rng, 4, 1, 32, 32, k, v)
    with pytest.raises(ValueError):
        oracle.decode(pool, np.zeros((1, 1, 32), np.float16), table[None], [0], 1.0)


# ---------------------------------------------------------------- prefill
def _prefill_setup(seed, P, hkv, hq, d, G, p0, T):
    rng = np.random.default_rng(seed)
    kp = exact_grid_rows(rng, p0, hkv, d, G)
    vp = exact_grid_rows(rng, p0, hkv, d, G)
    n_pages = -(-(p0 + T) // P)
    NP = n_pages + 2
    lay = oracle.layout(P, hkv, d, G, NP)
    table = rng.permutation(NP)[:n_pages].astype(np.int32)
    pool = oracle.Pool(lay)
    if p0:
        oracle.quantize_append(pool, kp, vp, [0, p0], [0], table[None])
    kc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    vc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    q = (rng.standard_normal((T, hq, d)) / np.sqrt(d)).astype(np.float16)
    return pool, table, kp, vp, kc, vc, q


@pytest.mark.parametrize("P,hkv,hq,d,G,p0,T", [(4, 1, 4, 64, 64, 10, 7), (8, 2, 8, 64, 32, 16, 12),
                                                (8, 2, 4, 128, 64, 0, 9)])
def test_prefill_matches_causal_sdpa(P, hkv, hq, d, G, p0, T):
    pool, table, kp, vp, kc, vc, q = _prefill_setup(P + p0 + T, P, hkv, hq, d, G, p0, T)
    out = oracle.prefill(pool, q, kc, vc, table, p0, alpha=1.0)
    K = np.concatenate([kp.astype(np.float64), kc.astype(np.float64)])
    V = np.concatenate([vp.astype(np.float64), vc.astype(np.float64)])
    mask = torch.from_numpy(np.arange(p0 + T)[None, :] <= (p0 + np.arange(T))[:, None])
    ref = sdpa_ref(q.astype(np.float64), K, V, 1.0, mask=mask)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_prefill_row_subset_matches_full():
    pool, table, kp, vp, kc, vc, q = _prefill_setup(31, 8, 2, 4, 64, 32, 24, 11)
    full = oracle.prefill(pool, q, kc, vc, table, 24, 1.0)
    rows = [10, 0, 5]
    sub = oracle.prefill(pool, q, kc, vc, table, 24, 1.0, rows=rows)
    assert np.array_equal(full[rows], sub)


def test_prefill_is_causal():
    pool, table, kp, vp, kc, vc, q = _prefill_setup(32, 4, 1, 2, 64, 64, 8, 9)
    base = oracle.prefill(pool, q, kc, vc, table, 8, 1.0)
    j = 4
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[j] = -kc2[j]
    vc2[j] += np.float16(1.0)
    pert = oracle.prefill(pool, q, kc2, vc2, table, 8, 1.0)
    assert np.array_equal(base[:j], pert[:j])
    assert not np.any(np.all(base[j:] == pert[j:], axis=(1, 2)))


def test_prefill_single_row_quantized_equals_decode_after_append():
    pool, table, kp, vp, kc, vc, q = _prefill_setup(33, 8, 2, 8, 64, 32, 21, 1)
    out = oracle.prefill(pool, q, kc, vc, table, 21, 1.0, chunk_quantized=True)
    p2 = pool.copy()
    oracle.quantize_append(p2, kc, vc, [0, 1], [21], table[None])
    dec = oracle.decode(p2, q, table[None], [22], 1.0)
    assert np.array_equal(out, dec)
