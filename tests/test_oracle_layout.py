"""Pins for the oracle's pool byte layout and page placement (CPU only).

Paging follows the paper's Background paragraph "Compact histories need
reusable storage" (fixed pool, 256-token pages, a page table mapping token
order to pages); eq. kvbytes gives the per-position payload for its TQ4
records, and the affine-Q4 analog is checked in closed form here.
"""
import json
import os

import numpy as np

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def test_golden_layout_example():
    with open(os.path.join(HERE, "golden", "layout_example.json")) as f:
        g = json.load(f)
    L = g["layout"]
    lay = oracle.layout(L["page_size"], L["num_kv_heads"], L["head_dim"], L["group_size"],
                        L["num_pages"])
    pool = oracle.Pool(lay, fill=0xA5)
    k = np.array([[g["x"]], [g["y"]]], np.float16)  # [2 rows][1 head][8]
    oracle.quantize_append(pool, k, k.copy(), [0, 2], [0], np.array([g["block_table"]]))
    assert pool.k_codes.tobytes().hex() == g["k_codes_hex"]
    assert pool.v_codes.tobytes().hex() == g["v_codes_hex"]
    assert ["%04x" % m for m in pool.k_meta] == g["meta_hex_u16"]
    assert ["%04x" % m for m in pool.v_meta] == g["meta_hex_u16"]
    assert list(oracle.quantize_group(k[0, 0])[0]) == g["x_codes"]
    assert list(oracle.quantize_group(k[1, 0])[0]) == g["y_codes"]


def test_pool_bytes_closed_form():
    """Bytes per position per layer = 2*Hkv*(d/2 + 2*2*d/G): 4-bit codes plus
    an fp16 scale and bias per group, for K and V (the affine analog of
    eq. kvbytes).  1,152 B at Hkv=8, d=128, G=64; 144 B at Hkv=1."""
    for hkv, d, G, per_pos in [(8, 128, 64, 1152), (1, 128, 64, 144), (4, 256, 64, 2 * 4 * (128 + 16))]:
        lay = oracle.layout(256, hkv, d, G, 1024)
        pool = oracle.Pool(lay)
        total = pool.k_codes.nbytes + pool.v_codes.nbytes + pool.k_meta.nbytes + pool.v_meta.nbytes
        assert total == 1024 * 256 * per_pos
    # the 262,144-position window at 32/8 heads: 301,989,888 bytes of K+V
    assert 262144 * 1152 == 301989888


def test_paper_tq4_payload_formula():
    """eq. kvbytes: 16 layers * 2 (K,V) * 4 heads * (128 packed bytes + 2-byte
    norm) = 16,640 B/position; 4,160 MiB at 262,144 positions."""
    beta = 16 * 2 * 4 * (128 + 2)
    assert beta == 16640
    assert beta * 262144 / 2 ** 20 == 4160


def _fill_random(pool, rng, L, n_rows, table, hkv, d):
    k = rng.standard_normal((n_rows, hkv, d)).astype(np.float16)
    v = rng.standard_normal((n_rows, hkv, d)).astype(np.float16)
    oracle.quantize_append(pool, k, v, [0, n_rows], [0], table[None, :])
    return k, v


def test_untouched_bytes_keep_poison_and_pages_follow_table():
    rng = np.random.default_rng(3)
    P, hkv, d, G, NP = 8, 2, 64, 32, 6
    lay = oracle.layout(P, hkv, d, G, NP)
    table = np.array([4, 1, 3], np.int32)
    pool = oracle.Pool(lay, fill=0xA5)
    n = 19  # 2 full pages and 3 slots of the third
    _fill_random(pool, rng, lay, n, table, hkv, d)
    page_codes = P * hkv * d // 2
    for page in range(NP):
        blk = pool.k_codes[page * page_codes:(page + 1) * page_codes]
        vblk = pool.v_codes[page * page_codes:(page + 1) * page_codes]
        if page in (0, 2, 5):
            assert (blk == 0xA5).all() and (vblk == 0xA5).all()
    # third logical page (physical 3) holds slots 0..2 only
    blk = pool.k_codes[3 * page_codes:4 * page_codes].reshape(hkv, P, d // 2)
    assert not (blk[:, :3] == 0xA5).all()
    assert (blk[:, 3:] == 0xA5).all()


def test_permuted_pages_same_logical_content():
    """Dequantized logical rows do not depend on which physical pages hold them."""
    rng = np.random.default_rng(4)
    P, hkv, d, G, NP = 4, 1, 32, 32, 8
    lay = oracle.layout(P, hkv, d, G, NP)
    k = rng.standard_normal((14, hkv, d)).astype(np.float16)
    v = rng.standard_normal((14, hkv, d)).astype(np.float16)
    outs = []
    for table in (np.array([0, 1, 2, 3]), np.array([7, 2, 5, 0])):
        pool = oracle.Pool(lay)
        oracle.quantize_append(pool, k, v, [0, 14], [0], table[None, :])
        rows = [oracle.dequant_vector(pool, iv, int(table[t // P]), 0, t % P)
                for t in range(14) for iv in (False, True)]
        outs.append(np.array(rows))
    assert np.array_equal(outs[0], outs[1])


def test_append_in_pieces_equals_append_at_once():
    rng = np.random.default_rng(5)
    P, hkv, d, G, NP = 4, 2, 64, 64, 5
    lay = oracle.layout(P, hkv, d, G, NP)
    table = np.array([[3, 0, 4]], np.int32)
    k = rng.standard_normal((11, hkv, d)).astype(np.float16)
    v = rng.standard_normal((11, hkv, d)).astype(np.float16)
    a = oracle.Pool(lay)
    oracle.quantize_append(a, k, v, [0, 11], [0], table)
    b = oracle.Pool(lay)
    for lo, hi in [(0, 5), (5, 6), (6, 11)]:
        oracle.quantize_append(b, k[lo:hi], v[lo:hi], [0, hi - lo], [lo], table)
    for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
        assert np.array_equal(getattr(a, n), getattr(b, n))


def test_batched_append_equals_per_request():
    rng = np.random.default_rng(6)
    P, hkv, d, G, NP = 4, 1, 32, 32, 10
    lay = oracle.layout(P, hkv, d, G, NP)
    tables = np.array([[1, 2, 3], [7, 8, 9]], np.int32)
    k = rng.standard_normal((7, hkv, d)).astype(np.float16)
    v = rng.standard_normal((7, hkv, d)).astype(np.float16)
    a = oracle.Pool(lay)
    oracle.quantize_append(a, k, v, [0, 3, 7], [2, 5], tables)
    b = oracle.Pool(lay)
    oracle.quantize_append(b, k[:3], v[:3], [0, 3], [2], tables[:1])
    oracle.quantize_append(b, k[3:], v[3:], [0, 4], [5], tables[1:])
    for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
        assert np.array_equal(getattr(a, n), getattr(b, n))
