"""Pins of oracle.verify (short packed verification: token k of the last Sq
cached positions attends to positions 0 .. L - Sq + k).

Independent check: torch's fp64 scaled_dot_product_attention with an
explicit boolean mask over the whole dequantized cache (keys and values
reconstructed one vector at a time by oracle.dequant_vector, whose pins are
elsewhere), so a mask aligned at the start of the cache, one position late
or early, or a token order reversed fails here."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_17475_amd import workloads


def _pool(P, hkv, d, G, L, seed):
    NP = -(-L // P) + 2
    pool = oracle.Pool(oracle.layout(P, hkv, d, G, NP))
    perm = np.random.default_rng(seed).permutation(NP).astype(np.int32)
    table = perm[: -(-L // P)][None]
    k, v = workloads.gen_kv(seed, L, hkv, d, 2)
    oracle.quantize_append(pool, k, v, [0, L], [0], table)
    return pool, table


def _dequant(pool, table, P, hkv, L, is_v):
    return np.array([[oracle.dequant_vector(pool, is_v, int(table[0][t // P]), h, t % P)
                      for h in range(hkv)] for t in range(L)])


@pytest.mark.parametrize("sq,L,hkv,hq", [(2, 70, 1, 4), (3, 130, 2, 8), (4, 33, 1, 2),
                                         (3, 2, 1, 4)])
def test_verify_equals_masked_sdpa(sq, L, hkv, hq):
    P, d, G = 32, 64, 32
    pool, table = _pool(P, hkv, d, G, L, seed=L + sq)
    rng = np.random.default_rng(sq)
    q = (rng.standard_normal((1, sq, hq, d)) / 8).astype(np.float16)
    alpha = 0.9
    got = oracle.verify(pool, q, table, [L], alpha)
    K = torch.from_numpy(_dequant(pool, table, P, hkv, L, False))  # [L][hkv][d]
    V = torch.from_numpy(_dequant(pool, table, P, hkv, L, True))
    gq = hq // hkv
    mask = torch.tensor([[t <= L - sq + k for t in range(L)] for k in range(sq)])
    for h in range(hq):
        qh = torch.from_numpy(q[0, :, h].astype(np.float64))          # [sq][d]
        kh, vh = K[:, h // gq], V[:, h // gq]
        ref = torch.nn.functional.scaled_dot_product_attention(
            qh[None], kh[None], vh[None], attn_mask=mask[None], scale=alpha)[0].numpy()
        for k in range(sq):
            if L - sq + 1 + k <= 0:  # a token that sees nothing: zero row
                assert not np.any(got[0, k, h])
            else:
                np.testing.assert_allclose(got[0, k, h], ref[k], rtol=1e-12, atol=1e-12)


def test_verify_single_query_is_decode():
    pool, table = _pool(32, 1, 64, 32, 90, seed=3)
    q = (np.random.default_rng(1).standard_normal((1, 1, 4, 64)) / 8).astype(np.float16)
    a = oracle.verify(pool, q, table, [90], 1.0)[:, 0]
    b = oracle.decode(pool, q[:, 0], table, [90], 1.0)
    assert np.array_equal(a, b)
