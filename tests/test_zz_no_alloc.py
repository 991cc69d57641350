"""The allocation-free decode step (jf_decode_step_q4_static: counters and
split records in the library's static device array) against the workspace
decode step (jf_decode_step_q4) on copies of the same pool: pool bytes and
outputs bitwise equal, and both within tolerance of the oracle.  Two calls in
a row, the second smaller (fewer requests, fewer heads, a shorter context),
so the second call runs on the array the first one left behind.  A request
beyond the array's size is refused before any launch."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import POISON, check_tol, log  # noqa: E402

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402

DEV = "cuda"


def _pools(P, hkv, d, G, lens, n_step, seed):
    B = len(lens)
    max_pages = -(-(max(lens) + n_step) // P)
    NP = B * max_pages + 1
    lay = jfkv.layout(P, hkv, d, G, NP)
    a = jfkv.KVPool(lay, fill=POISON)
    host = oracle.Pool(oracle.layout(P, hkv, d, G, NP), fill=POISON)
    pp = jfkv.PagePool(NP, P, shuffle_seed=seed)
    seqs = [pp.create() for _ in range(B)]
    for s, L in zip(seqs, lens):
        pp.reserve(s, L + n_step)
    tables = np.array(pp.export(seqs, max_pages)[0], np.int32)
    k, v = workloads.gen_kv(seed, sum(lens) + B, hkv, d, 2)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    jfkv.jf_kv_quantize_append(a, torch.from_numpy(k[:cu[-1]]).to(DEV),
                               torch.from_numpy(v[:cu[-1]]).to(DEV),
                               torch.tensor(cu, dtype=torch.int32, device=DEV),
                               torch.zeros(B, dtype=torch.int32, device=DEV),
                               torch.from_numpy(tables).to(DEV))
    oracle.quantize_append(host, k[:cu[-1]], v[:cu[-1]], list(cu), [0] * B, tables)
    b = jfkv.KVPool(lay, device=DEV)
    for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
        getattr(b, n).copy_(getattr(a, n))
    new_k = k[cu[-1]:].reshape(B, hkv, d)
    new_v = v[cu[-1]:].reshape(B, hkv, d)
    return a, b, host, tables, new_k, new_v


@pytest.mark.parametrize("case", [
    # (P, hkv, hq, d, G, lens, max_splits): the second call is smaller
    [(256, 8, 32, 128, 64, (5000, 1300, 700), 64), (256, 8, 32, 128, 64, (900,), 64)],
    [(64, 2, 8, 128, 64, (3000, 2500), 16), (64, 1, 4, 64, 32, (130,), 4)],
])
def test_static_step_equals_workspace_step(case):
    for call, (P, hkv, hq, d, G, lens, ms) in enumerate(case):
        log("static step call %d: P=%d hkv=%d hq=%d d=%d G=%d lens=%s max_splits=%d" % (
            call, P, hkv, hq, d, G, lens, ms))
        B = len(lens)
        a, b, host, tables, kn, vn = _pools(P, hkv, d, G, lens, 1, seed=40 + call)
        q = (np.random.default_rng(50 + call).standard_normal((B, hq, d)) /
             np.sqrt(d)).astype(np.float16)
        steps_lens = [L + 1 for L in lens]
        gt = torch.from_numpy(tables).to(DEV)
        lt = torch.tensor(steps_lens, dtype=torch.int32, device=DEV)
        kt, vt, qt = (torch.from_numpy(np.ascontiguousarray(x)).to(DEV) for x in (kn, vn, q))
        out_s = torch.empty((B, hq, d), dtype=torch.float16, device=DEV)
        jfkv.jf_decode_step_q4_static(a, kt, vt, qt, gt, lt, 1.0, ms, out_s)
        ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, hq, d, ms), dtype=torch.uint8,
                         device=DEV)
        out_w = torch.empty_like(out_s)
        jfkv.jf_decode_step_q4(b, kt, vt, qt, gt, lt, 1.0, ms, ws, out_w)
        torch.cuda.synchronize()
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            assert torch.equal(getattr(a, n), getattr(b, n)), "pool %s differs" % n
        got = out_s.cpu().numpy()
        assert np.array_equal(got, out_w.cpu().numpy()), "static != workspace step"
        for bb in range(B):
            oracle.quantize_append(host, kn[bb][None], vn[bb][None], [0, 1], [lens[bb]],
                                   tables[bb:bb + 1])
        ref = oracle.decode(host, q, tables, steps_lens, 1.0)
        err, rel = check_tol(got, ref, what="static step call %d" % call)
        log("  max err %.2e rel L2 %.2e" % (err, rel))


def test_static_step_refuses_oversized_requests():
    lay = jfkv.layout(256, 8, 128, 64, 4)
    pool = jfkv.KVPool(lay, device=DEV)
    B, hq, d = 64, 32, 128
    z16 = torch.zeros((B, 8, d), dtype=torch.float16, device=DEV)
    q = torch.zeros((B, hq, d), dtype=torch.float16, device=DEV)
    bt = torch.zeros((B, 1), dtype=torch.int32, device=DEV)
    lens = torch.ones(B, dtype=torch.int32, device=DEV)
    out = torch.empty_like(q)
    with pytest.raises(jfkv.JfError) as e:
        # 64 x 32 x 64 x 132 x 4 bytes of records: beyond the 8 MiB array
        jfkv.jf_decode_step_q4_static(pool, z16, z16, q, bt, lens, 1.0, 64, out)
    assert e.value.status == jfkv.JF_ERR_INVALID and "static scratch" in str(e.value)
