"""GPU split-K decode over paged 4-bit KV against the CPU oracle.

Tolerance: |o_gpu - o_ref| <= 2e-3 absolute (fp16 output, fp32 accumulation),
plus relative L2 <= 2e-3 on flat data (three fp16 roundings per position, see
gpu_cases.check_tol); the needle variants (|o| up to ~30) allow
2e-3 + 2^-11 |o_ref| (fp16 output rounding is 2^-11 relative).
Invariants: page order and head independence bitwise, split count within
tolerance, ragged batch equal to each request alone (bitwise), determinism.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import (Case, POISON, append_both, build, check_tol, decode_gpu,  # noqa: E402
                       decode_oracle, log)

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402


def _q(seed, B, hq, d, scale=None):
    rng = np.random.default_rng(seed)
    s = (1.0 / np.sqrt(d)) if scale is None else scale
    return (rng.standard_normal((B, hq, d)) * s).astype(np.float16)


@pytest.mark.parametrize("P,hkv,hq,d,G,lens", [
    (256, 1, 4, 128, 64, (1,)),
    (256, 1, 4, 128, 64, (37,)),
    (256, 1, 4, 128, 64, (4097,)),
    (64, 1, 4, 128, 64, (1000,)),
    (256, 2, 8, 64, 32, (777,)),
    (64, 8, 32, 128, 128, (130, 65)),
    (256, 4, 24, 256, 64, (600,)),   # the paper's 24 q / 4 KV heads, d = 256
    (128, 2, 2, 128, 64, (300,)),    # one query head per KV head
    (64, 2, 6, 128, 32, (500,)),     # three per KV head
    (64, 1, 8, 128, 64, (333,)),     # eight per KV head (one column set of eight)
    (64, 1, 16, 128, 64, (333,)),    # sixteen per KV head (one chunk of two sets of eight)
    (64, 2, 20, 128, 128, (400,)),   # ten per KV head, one group per half (second set: 2)
    (64, 1, 12, 64, 64, (500,)),     # d = 64, twelve per KV head (sets of 8 + 4)
    (64, 1, 20, 128, 64, (450,)),    # twenty per KV head (chunks of 16 + 4)
    (64, 1, 12, 128, 32, (350,)),    # 32-dim groups, twelve (chunks of 2 x 4 + 4)
    (64, 1, 40, 256, 64, (300,)),    # d = 256: one set per chunk (chunks of 4)
])
def test_decode_matches_oracle(P, hkv, hq, d, G, lens):
    log("decode P=%d hkv=%d hq=%d d=%d G=%d lens=%s" % (P, hkv, hq, d, G, lens))
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=lens, n_out=max(1, d // 50), seed=sum(lens))
    q = _q(7, len(lens), hq, d)
    got = decode_gpu(case, q)
    ref = decode_oracle(case, q)
    check_tol(got, ref, what="decode")


@pytest.mark.parametrize("lens,prefix", [((4096 + 300, 2048 + 5), 2048), ((513, 512), 512)])
def test_ragged_batch_with_shared_prefix(lens, prefix):
    log("decode ragged lens=%s prefix=%d" % (lens, prefix))
    case = build(P=256, hkv=8, d=128, G=64, hq=32, lens=lens, shared_prefix=prefix, seed=11)
    q = _q(8, len(lens), 32, 128)
    got = decode_gpu(case, q)
    check_tol(got, decode_oracle(case, q), what="ragged")
    for b in range(len(lens)):
        alone = decode_gpu(case, q[b:b + 1], lens=[lens[b]], tables=case.tables[b:b + 1])
        assert np.array_equal(alone[0], got[b])


def test_needle_variant():
    log("decode needle")
    L = 3000
    case = build(P=256, hkv=2, d=128, G=64, hq=8, lens=(L,), n_out=3, seed=21)
    qn, t_star = workloads.needle_queries(case.k_rows[0], 8, seed=5)
    q = qn[None]
    got = decode_gpu(case, q)
    ref = decode_oracle(case, q)
    assert np.abs(ref).max() > 1.0
    check_tol(got, ref, atol=2e-3, rel_elem=2.0 ** -11, rel_l2=2e-3, what="needle")


def test_single_position_and_identical_keys():
    log("decode special cases")
    P, hkv, d, G = 64, 1, 128, 64
    rng = np.random.default_rng(9)
    n = 200
    k = np.repeat(rng.standard_normal((1, hkv, d)).astype(np.float16), n, axis=0)
    v = rng.standard_normal((n, hkv, d)).astype(np.float16)
    lay = jfkv.layout(P, hkv, d, G, 5)
    case = Case(lay, None, jfkv.KVPool(lay, fill=POISON),
                oracle.Pool(oracle.layout(P, hkv, d, G, 5), fill=POISON),
                np.array([[3, 0, 4, 1]], np.int32), [n], 4, [], [])
    append_both(case, k, v, [0, n], [0], case.tables)
    q = _q(10, 1, 4, d, scale=0.5)
    # identical keys: output is the mean of the dequantized values
    vhat = np.array([oracle.dequant_vector(case.host, True, int(case.tables[0, t // P]), 0, t % P)
                     for t in range(n)])
    got = decode_gpu(case, q)
    check_tol(got, np.broadcast_to(vhat.mean(0), got.shape).astype(np.float64), what="identical")
    # one position: output is that position's value
    got1 = decode_gpu(case, q, lens=[1])
    check_tol(got1, np.broadcast_to(vhat[0], got.shape).astype(np.float64), atol=1e-3,
              what="L=1")


def test_page_permutation_and_determinism_bitwise():
    log("decode page permutation")
    outs = []
    for shuffle in (1, 2, 3):
        case = build(P=64, hkv=2, d=128, G=64, hq=8, lens=(1500,), seed=31, shuffle_seed=shuffle)
        q = _q(11, 1, 8, 128)
        outs.append(decode_gpu(case, q))
        outs.append(decode_gpu(case, q))
    for o in outs[1:]:
        assert np.array_equal(outs[0], o)


def test_split_count_changes_only_rounding():
    log("decode split counts")
    case = build(P=64, hkv=2, d=128, G=64, hq=8, lens=(64 * 40 + 7,), seed=41)
    q = _q(12, 1, 8, 128)
    ref = decode_oracle(case, q)
    outs = {s: decode_gpu(case, q, max_splits=s) for s in (1, 2, 3, 7, 41, 64, 1024)}
    for s, o in outs.items():
        check_tol(o, ref, what="splits=%d" % s)
    assert np.max(np.abs(outs[1].astype(np.float64) - outs[64].astype(np.float64))) <= 2e-3


def test_query_heads_are_independent():
    log("decode head independence")
    case = build(P=64, hkv=2, d=128, G=64, hq=8, lens=(700,), seed=51)
    q = _q(13, 1, 8, 128)
    perm = np.array([1, 3, 0, 2, 6, 4, 7, 5])
    a = decode_gpu(case, q)
    b = decode_gpu(case, np.ascontiguousarray(q[:, perm]))
    assert np.array_equal(a[:, perm], b)


def test_empty_and_clamped_lengths():
    log("decode empty/clamped lengths")
    case = build(P=64, hkv=1, d=128, G=64, hq=4, lens=(128, 100), seed=61)
    q = _q(14, 2, 4, 128)
    got = decode_gpu(case, q, lens=[0, 100])
    assert np.all(got[0] == 0)
    check_tol(got[1:], decode_oracle(case, q[1:], lens=[100], tables=case.tables[1:]),
              what="after empty row")
    # a length beyond the table capacity is clamped to max_pages * page_size
    got2 = decode_gpu(case, q[:1], lens=[10 ** 6], tables=case.tables[:1])
    check_tol(got2, decode_oracle(case, q[:1], lens=[128], tables=case.tables[:1]), what="clamp")


def test_invalid_page_entries_are_skipped():
    """A page-table entry outside [0, num_pages) is never read and its
    positions do not contribute; attention is order-free over positions, so the
    reference is the same request with that page's positions removed."""
    log("decode invalid page entries")
    case = build(P=64, hkv=2, d=128, G=64, hq=8, lens=(64 * 12,), seed=71)
    q = _q(15, 1, 8, 128)
    bad = case.tables.copy()
    bad[0, 0] = -1                       # first page: no valid position seen before it
    bad[0, 5] = case.lay.num_pages + 3   # out of range
    got = decode_gpu(case, q, tables=bad)
    keep = [p for i, p in enumerate(case.tables[0]) if i not in (0, 5)]
    ref = decode_oracle(case, q, lens=[64 * 10], tables=np.array([keep], np.int32))
    check_tol(got, ref, what="invalid pages")


def test_workspace_reuse_across_calls():
    """One zero-filled workspace serves consecutive calls with different
    lengths, split counts and batch sizes: the completion counters return to
    zero after every call."""
    log("decode workspace reuse")
    case = build(P=64, hkv=2, d=128, G=64, hq=8, lens=(64 * 30 + 5, 900), seed=81)
    q = _q(16, 2, 8, 128)
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(2, 8, 128, 64), dtype=torch.uint8,
                     device="cuda")
    for lens, splits in [((64 * 30 + 5, 900), 64), ((100, 900), 7), ((64 * 30 + 5, 1), 64),
                         ((0, 900), 3), ((64 * 30 + 5, 900), 1), ((64 * 30 + 5, 900), 64)]:
        got = decode_gpu(case, q, max_splits=splits, lens=list(lens), ws=ws)
        for b in range(2):
            if lens[b] == 0:
                assert np.all(got[b] == 0)
                continue
            ref = decode_oracle(case, q[b:b + 1], lens=[lens[b]], tables=case.tables[b:b + 1])
            check_tol(got[b:b + 1], ref, what="reuse lens=%s splits=%d" % (lens, splits))
    counters = ws[:262144].cpu().numpy()
    assert np.all(counters == 0), "completion counters not reset"
