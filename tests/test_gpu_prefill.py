"""GPU chunked prefill (fp16 matrix cores) against the CPU oracle.

Tolerance: |o_gpu - o_ref| <= 2e-3 + 2^-8 |o_ref|, relative L2 <= 4e-3.  The
operands that are rounded are p (fp16) and the reconstructed values
(scale * code + bias, rounded once to fp16); key codes, scales and biases
enter the scores exactly, with fp32 accumulation.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import append_both, build, check_tol, log, pool_bytes_equal  # noqa: E402

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv  # noqa: E402


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
    log("  max err %.3e rel L2 %.3e" % check_tol(got, ref, atol=2e-3, rel_elem=2.0 ** -8,
                                                 rel_l2=4e-3, what="prefill"))


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
    check_tol(got, ref, atol=2e-3, rel_elem=2.0 ** -8, rel_l2=4e-3, what="prefill")
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
