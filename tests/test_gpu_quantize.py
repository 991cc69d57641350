"""GPU quantize-append: the device pools must equal the oracle's byte for byte
(codes, scales, biases, page placement, untouched poison bytes)."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import POISON, Case, append_both, build, log, pool_bytes_equal  # noqa: E402

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv  # noqa: E402


@pytest.mark.parametrize("P,hkv,d,G,lens,prefix", [
    (256, 1, 128, 64, (4097,), 0),
    (64, 2, 64, 32, (300, 171), 128),
    (256, 8, 128, 64, (700, 513), 256),
    (128, 4, 256, 64, (390,), 0),
    (64, 3, 128, 128, (65, 64, 1), 0),
    (256, 2, 256, 32, (257, 300), 256),
    # more row tiles (938 x 2 x 3 of 64 rows) than waves in the persistent
    # grid (4 x 4 waves per CU), with a KV-head count that does not divide
    # the grid: waves move to another KV head between tiles, and each tile
    # must be stored under its own
    (64, 3, 64, 32, (60000,), 0),
])
def test_pool_bytes_bit_exact(P, hkv, d, G, lens, prefix):
    log("quantize P=%d hkv=%d d=%d G=%d lens=%s prefix=%d" % (P, hkv, d, G, lens, prefix))
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hkv, lens=lens, shared_prefix=prefix, n_out=3,
                 seed=P + d + G)
    assert pool_bytes_equal(case) == []


@pytest.mark.parametrize("dist", ["tiny", "wide", "special"])
@pytest.mark.parametrize("n", [130, 520])  # below / above the row-tiled kernel's threshold
def test_pool_bytes_bit_exact_edge_values(dist, n):
    log("quantize edge values %s n=%d" % (dist, n))
    P, hkv, d, G = 64, 2, 128, 64
    n_pages = -(-n // P)
    NP = n_pages + 2
    table = np.random.default_rng(n).permutation(NP)[:n_pages].astype(np.int32)[None]
    lay = jfkv.layout(P, hkv, d, G, NP)
    case = Case(lay, oracle.layout(P, hkv, d, G, NP), jfkv.KVPool(lay, fill=POISON),
                oracle.Pool(oracle.layout(P, hkv, d, G, NP), fill=POISON),
                table, [n], hkv, [], [])
    rng = np.random.default_rng(42)
    if dist == "tiny":  # ranges below 15*2^-14: subnormal fp16 scales
        k = (rng.standard_normal((n, hkv, d)) * 2.0 ** -17).astype(np.float16)
        v = (rng.standard_normal((n, hkv, d)) * 2.0 ** -12).astype(np.float16)
    elif dist == "wide":  # near the fp16 range: scales up to ~8.7e3
        k = np.clip(rng.standard_normal((n, hkv, d)) * 30000, -65504, 65504).astype(np.float16)
        v = (rng.standard_normal((n, hkv, d)) * 1000).astype(np.float16)
    else:
        k = rng.standard_normal((n, hkv, d)).astype(np.float16)
        v = rng.standard_normal((n, hkv, d)).astype(np.float16)
        k[0] = 0.0                       # constant group (+0)
        k[1] = np.float16(-0.0)          # constant group (-0)
        k[2, :, :64] = 1.5               # one constant group of two
        k[3, :, ::2] = np.float16(-0.0)  # mixed signed zeros
        k[3, :, 1::2] = 0.0
        v[4] = np.float16(65504.0)
        v[4, :, 5] = np.float16(-65504.0)
        v[5] = np.float16(2.0 ** -24)    # smallest subnormal
        v[5, :, 0] = 0.0
        k[6, :, :] = np.arange(d, dtype=np.float16) % 16  # exact grid, scale 1
        v[7, :, :] = (np.arange(d) % 16 + 0.5).astype(np.float16)  # ties at midpoints
    append_both(case, k, v, [0, n], [0], case.tables)
    torch.cuda.synchronize()
    assert pool_bytes_equal(case) == []


def test_single_row_appends_equal_bulk_and_skip_invalid_pages():
    log("quantize single-row appends + invalid page entries")
    P, hkv, d, G = 64, 2, 128, 64
    NP = 6
    rng = np.random.default_rng(3)
    n = 150
    k = rng.standard_normal((n, hkv, d)).astype(np.float16)
    v = rng.standard_normal((n, hkv, d)).astype(np.float16)
    tables = np.array([[4, 1, 5]], np.int32)
    lay = jfkv.layout(P, hkv, d, G, NP)
    gpu = jfkv.KVPool(lay, fill=POISON)
    host = oracle.Pool(oracle.layout(P, hkv, d, G, NP), fill=POISON)
    case = Case(lay, None, gpu, host, tables, [n], hkv, [], [])
    for t in range(n):  # one decode-style append per row
        append_both(case, k[t:t + 1], v[t:t + 1], [0, 1], [t], tables)
    torch.cuda.synchronize()
    assert pool_bytes_equal(case) == []
    # entries -1 and out of range are skipped, other rows still land (a bulk
    # append of 150 rows: the small-append kernel; test_invalid_pages_tiled
    # covers the row-tiled one)
    bad_tables = np.array([[-1, 3, NP + 7]], np.int32)
    dev = "cuda"
    jfkv.jf_kv_quantize_append(gpu, torch.from_numpy(k).to(dev), torch.from_numpy(v).to(dev),
                               torch.tensor([0, n], dtype=torch.int32, device=dev),
                               torch.tensor([0], dtype=torch.int32, device=dev),
                               torch.from_numpy(bad_tables).to(dev))
    oracle.quantize_append(host, k[P:2 * P], v[P:2 * P], [0, P], [P], np.array([[0, 3]], np.int32))
    torch.cuda.synchronize()
    assert pool_bytes_equal(case) == []


def test_invalid_pages_and_odd_start_tiled():
    """Row-tiled kernel (>= 256 rows): page entries -1 / out of range are
    skipped; an odd start position makes every V position pair straddle two
    rows of different tiles; a second request starts mid-page."""
    log("quantize tiled: invalid pages, odd start, two requests")
    P, hkv, d, G = 64, 2, 128, 64
    NP = 16
    rng = np.random.default_rng(5)
    n0, n1 = 301, 260
    k = rng.standard_normal((n0 + n1, hkv, d)).astype(np.float16)
    v = rng.standard_normal((n0 + n1, hkv, d)).astype(np.float16)
    tables = np.array([[7, -1, 3, 12, NP + 2, 0, 9, 1],
                       [2, 4, 5, 6, 8, 10, 11, 13]], np.int32)
    lay = jfkv.layout(P, hkv, d, G, NP)
    case = Case(lay, None, jfkv.KVPool(lay, fill=POISON),
                oracle.Pool(oracle.layout(P, hkv, d, G, NP), fill=POISON), tables, [], hkv, [],
                [])
    dev = "cuda"
    jfkv.jf_kv_quantize_append(case.gpu, torch.from_numpy(k).to(dev), torch.from_numpy(v).to(dev),
                               torch.tensor([0, n0, n0 + n1], dtype=torch.int32, device=dev),
                               torch.tensor([3, 37], dtype=torch.int32, device=dev),
                               torch.from_numpy(tables).to(dev))
    # the oracle writes only rows on valid pages: request 0's positions 3..63
    # (rows 0..60) and 128..255 (rows 125..252); request 1 entirely
    host = case.host
    oracle.quantize_append(host, k[0:61], v[0:61], [0, 61], [3], tables[:1])
    oracle.quantize_append(host, k[125:253], v[125:253], [0, 128], [128], tables[:1])
    oracle.quantize_append(host, k[n0:], v[n0:], [0, n1], [37], tables[1:])
    torch.cuda.synchronize()
    assert pool_bytes_equal(case) == []
