"""GPU chunked prefill (fp16 matrix cores) against the CPU oracle.

Tolerance: |o_gpu - o_ref| <= 2e-3 + 2^-11 |o_ref| elementwise, relative L2
<= 1e-3 (PREFILL_TOL).  Error analysis of the kernel's arithmetic:
  * key codes, scales, biases and the fp16 queries enter the scores exactly
    (fp32 accumulation; the bias part carries the query group sums as an
    fp16 high and low part, ~2^-22 relative);
  * reconstructed values enter as an fp16 high part plus an fp16 low part
    of value / 2 (~2^-21 relative), the chunk's own fp16 rows exactly;
  * p is rounded to fp16, and the same rounded p enter the numerator and the
    denominator, so the rounding perturbs each weight by at most 2^-11
    relative: the output moves by at most 2^-11 times the weighted mean of
    |v - o|, which averages out over many keys (flat data) and is small when
    one key dominates by a wide logit gap (needle data, gap 16 here);
  * the output is rounded to fp16 once: 2^-11 |o| relative.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import (POISON, Case, append_both, build, check_tol, log,  # noqa: E402
                       pool_bytes_equal)

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402

PREFILL_TOL = dict(atol=2e-3, rel_elem=2.0 ** -11, rel_l2=1e-3)


def prefill_gpu(case, q, kc, vc, prefix_len, scale=1.0):
    dev = "cuda"
    out = torch.empty(q.shape, dtype=torch.float16, device=dev)
    jfkv.jf_prefill_attn_q4(case.gpu, torch.from_numpy(q).to(dev), torch.from_numpy(kc).to(dev),
                            torch.from_numpy(vc).to(dev),
                            torch.from_numpy(np.ascontiguousarray(case.tables[0])).to(dev),
                            prefix_len, scale, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("P,hkv,hq,d,G,p0,T", [
    (256, 2, 8, 128, 64, 300, 37),
    (64, 1, 4, 128, 64, 0, 70),
    (64, 2, 8, 128, 64, 64, 1),
    (256, 4, 24, 256, 64, 512, 33),  # the paper's head geometry
    (64, 2, 4, 64, 32, 200, 90),
    (256, 8, 32, 128, 64, 1024, 160),
])
def test_prefill_matches_oracle(P, hkv, hq, d, G, p0, T):
    log("prefill P=%d hkv=%d hq=%d d=%d G=%d p0=%d T=%d" % (P, hkv, hq, d, G, p0, T))
    # reserve room for the chunk too, then attend prefix + chunk
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=(p0 + T,), n_out=2, seed=p0 + T)
    rng = np.random.default_rng(p0 * 7 + T)
    # the pool holds p0 + T rows; only the first p0 are the prefix here
    kc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    vc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    q = (rng.standard_normal((T, hq, d)) / np.sqrt(d)).astype(np.float16)
    got = prefill_gpu(case, q, kc, vc, p0)
    ref = oracle.prefill(case.host, q, kc, vc, case.tables[0], p0, 1.0)
    log("  max err %.3e rel L2 %.3e" % check_tol(got, ref, what="prefill", **PREFILL_TOL))


def test_prefill_then_append_chunk_bit_exact():
    log("prefill + chunk append")
    P, hkv, hq, d, G, p0, T = 64, 2, 8, 128, 64, 192, 100
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=(p0,), seed=5, extra_pages=2)
    # grow the table by hand: two free pages follow the used ones in this pool
    used = set(case.tables[0].tolist())
    free = [p for p in range(case.lay.num_pages) if p not in used]
    table = np.array([list(case.tables[0]) + free[:2]], np.int32)
    case.tables = table
    rng = np.random.default_rng(77)
    kc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    vc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    q = (rng.standard_normal((T, hq, d)) / np.sqrt(d)).astype(np.float16)
    got = prefill_gpu(case, q, kc, vc, p0)
    ref = oracle.prefill(case.host, q, kc, vc, table[0], p0, 1.0)
    check_tol(got, ref, what="prefill", **PREFILL_TOL)
    append_both(case, kc, vc, [0, T], [p0], table)
    torch.cuda.synchronize()
    assert pool_bytes_equal(case) == []


def test_prefill_is_causal_on_gpu():
    log("prefill causality")
    P, hkv, hq, d, G, p0, T = 64, 1, 4, 128, 64, 128, 80
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=(p0,), seed=6)
    rng = np.random.default_rng(78)
    kc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    vc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    q = (rng.standard_normal((T, hq, d)) / np.sqrt(d)).astype(np.float16)
    base = prefill_gpu(case, q, kc, vc, p0)
    j = 50
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[j] *= -1
    vc2[j] += np.float16(3.0)
    pert = prefill_gpu(case, q, kc2, vc2, p0)
    assert np.array_equal(base[:j], pert[:j])
    assert np.all(np.any(base[j:] != pert[j:], axis=(1, 2)))


def test_prefill_needle_prefix_and_chunk_keys():
    """Each query row points at one key (logit gap 16): even rows at a prefix
    key, odd rows at a chunk key at or before their own position, so the
    output is that key's (reconstructed, or fp16) value, |o| up to ~30 on
    outlier channels."""
    log("prefill needle")
    P, hkv, hq, d, G, p0, T = 256, 2, 8, 128, 64, 1024, 64
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=(p0 + T,), n_out=3, seed=31)
    rng = np.random.default_rng(32)
    kc = rng.standard_normal((T, hkv, d)).astype(np.float16)
    vc = (rng.standard_normal((T, hkv, d)) * 4).astype(np.float16)
    keys = np.concatenate([case.k_rows[0][:p0], kc]).astype(np.float64)
    gq = hq // hkv
    q = np.zeros((T, hq, d), np.float16)
    for i in range(T):
        n_vis = p0 + i + 1
        # even rows: a prefix key; odd rows: a chunk key at or before row i
        lo, hi = (0, p0) if i % 2 == 0 else (p0, n_vis)
        t_star = rng.integers(lo, hi, size=hq)
        for h in range(hq):
            kstar = keys[t_star[h], h // gq]
            norm = np.linalg.norm(kstar)
            # the other visible keys project onto k* / |k*| as ~N(0, 1): their
            # maximum is about sqrt(2 ln n_vis)
            gamma = 16.0 / max(norm - np.sqrt(2.0 * np.log(n_vis)), 1.0)
            q[i, h] = (gamma * kstar / norm).astype(np.float16)
    got = prefill_gpu(case, q, kc, vc, p0)
    ref = oracle.prefill(case.host, q, kc, vc, case.tables[0], p0, 1.0)
    assert np.abs(ref).max() > 8.0
    log("  max err %.3e rel L2 %.3e (max |o| %.1f)" % (
        check_tol(got, ref, what="needle", **PREFILL_TOL) + (np.abs(ref).max(),)))


def test_prefill_value_groups_reaching_fp16_max():
    """V groups whose range spans 0 .. 65504: the quantizer rounds the scale
    up, so scale * 15 + bias exceeds the fp16 maximum (65,520 here); the
    output must stay finite and match the oracle.  The query is zero, so
    every weight is exactly 1 and the output is the mean of the values."""
    log("prefill extreme value groups")
    P, hkv, hq, d, G, p0, T = 64, 1, 4, 128, 64, 128, 16
    rng = np.random.default_rng(41)
    n = p0 + T
    k = rng.standard_normal((n, hkv, d)).astype(np.float16)
    v = rng.uniform(0.0, 1.0, (n, hkv, d))
    v[::2, :, 0] = 65504.0          # group 0 spans [0, 65504] at even positions
    v[1::4, :, 64] = -65504.0       # group 1 spans [-65504, 1] at some odd ones
    v = v.astype(np.float16)
    lay = jfkv.layout(P, hkv, d, G, 4)
    case = Case(lay, None, jfkv.KVPool(lay, fill=POISON),
                oracle.Pool(oracle.layout(P, hkv, d, G, 4), fill=POISON),
                np.array([[2, 0, 3]], np.int32), [p0], hq, [], [])
    append_both(case, k[:p0], v[:p0], [0, p0], [0], case.tables)
    smeta = case.host.v_meta.view(np.float16).reshape(4, hkv, P, d // G, 2)[2, 0, 0, 0, 0]
    assert float(smeta) * 15 > 65504  # the reconstructed maximum is beyond fp16
    q = np.zeros((T, hq, d), np.float16)
    got = prefill_gpu(case, q, k[p0:], v[p0:], p0)
    ref = oracle.prefill(case.host, q, k[p0:], v[p0:], case.tables[0], p0, 1.0)
    assert np.all(np.isfinite(got))
    log("  max err %.3e rel L2 %.3e" % check_tol(got, ref, what="extreme", **PREFILL_TOL))
