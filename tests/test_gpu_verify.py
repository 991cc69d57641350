"""GPU short packed verifier (jf_verify_attn_q4) against the CPU oracle.

The last Sq cached positions of a request are its Sq query tokens (2 to 4 in
the paper's eligible tiles; MTP width 3 in its 32K+6K study); token k sees
positions 0 .. L - Sq + k.  The oracle (oracle.verify) is the plain decode
definition over the first L - Sq + k + 1 positions of each token.

Tolerance: |o - o_ref| <= 2e-3 + 2^-11 |o_ref| elementwise and relative L2
<= 1e-3 (gpu_cases.check_tol).  2e-3 is the bound on the fp32-accumulated
attention; 2^-11 |o_ref| is the half-ulp of the fp16 output itself, which
short windows need: a token that sees a few dozen positions averages few
values, so an outlier channel (x8) gives |o| up to ~8, where one fp16
half-ulp is already 2^-9 ~ 2e-3.  The verifier runs the decode kernel's
arithmetic with a per-token causal limit, nothing else.
Cases: Sq = 1..4, one and several head chunks, d = 64/128/256, G = 32/64/128,
ragged batches with a shared prefix, lengths shorter than Sq (tokens that see
nothing give zero rows), split caps, a needle at the last position that
only the last token may see, and Sq = 1 equal to decode bitwise.  The
262,144-position window is in test_gpu_fullsize."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import build, check_tol, decode_gpu, log  # noqa: E402

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv  # noqa: E402

DEV = "cuda"
TOL_REL = 2.0 ** -11  # fp16 output rounding, relative


def _q(seed, B, sq, hq, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((B, sq, hq, d)) / np.sqrt(d)).astype(np.float16)


def verify_gpu(case, q, max_splits=64, scale=1.0, lens=None, ws=None):
    B, sq, hq, d = q.shape
    lens = case.lens if lens is None else lens
    if ws is None:
        ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, hq * sq, d, max_splits),
                         dtype=torch.uint8, device=DEV)
    out = torch.empty(q.shape, dtype=torch.float16, device=DEV)
    jfkv.jf_verify_attn_q4(case.gpu, torch.from_numpy(q).to(DEV),
                           torch.from_numpy(np.ascontiguousarray(case.tables)).to(DEV),
                           torch.tensor(lens, dtype=torch.int32, device=DEV), scale, max_splits,
                           ws, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("P,hkv,hq,d,G,lens,sq", [
    (256, 1, 4, 128, 64, (3,), 3),
    (256, 1, 4, 128, 64, (37,), 2),
    (256, 1, 4, 128, 64, (4097,), 3),
    (256, 1, 4, 128, 64, (4097,), 4),
    (64, 8, 32, 128, 64, (1000, 259), 3),  # the bench geometry, ragged
    (256, 2, 8, 64, 32, (777,), 2),
    (64, 4, 24, 256, 64, (600,), 3),       # 24 q / 4 KV heads, d = 256
    (128, 2, 2, 128, 128, (300,), 4),      # one query head per KV head
    (64, 2, 6, 128, 32, (500, 2), 3),      # a request shorter than Sq
    (64, 1, 8, 128, 64, (700,), 3),        # 24 (head, token) pairs: chunks of 16 + 8
    (64, 2, 8, 64, 64, (650,), 3),         # d = 64, 12 pairs: one block, two column sets
])
def test_verify_matches_oracle(P, hkv, hq, d, G, lens, sq):
    log("verify P=%d hkv=%d hq=%d d=%d G=%d lens=%s sq=%d" % (P, hkv, hq, d, G, lens, sq))
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=lens, seed=sum(lens) + sq)
    q = _q(7 + sq, len(lens), sq, hq, d)
    got = verify_gpu(case, q)
    ref = oracle.verify(case.host, q, case.tables, case.lens, 1.0)
    err, rel = check_tol(got, ref, rel_elem=TOL_REL, what="verify")
    log("  max err %.2e rel L2 %.2e" % (err, rel))
    for b, L in enumerate(lens):  # tokens that see no position: zero rows
        for k in range(sq):
            if L - sq + 1 + k <= 0:
                assert not np.any(got[b, k])


def test_verify_one_query_is_decode_bitwise():
    log("verify Sq=1 vs decode")
    case = build(P=64, hkv=2, hq=8, lens=(900, 333), seed=3)
    q = _q(4, 2, 1, 8, 128)
    a = verify_gpu(case, q)
    b = decode_gpu(case, np.ascontiguousarray(q[:, 0]))
    assert np.array_equal(a[:, 0], b)


def test_verify_split_caps_and_shared_prefix():
    log("verify split caps, shared prefix")
    case = build(P=64, hkv=2, hq=8, lens=(2048 + 301, 1024 + 7), shared_prefix=1024, seed=5)
    q = _q(6, 2, 3, 8, 128)
    ref = oracle.verify(case.host, q, case.tables, case.lens, 1.0)
    for s in (1, 5, 64):
        check_tol(verify_gpu(case, q, max_splits=s), ref, rel_elem=TOL_REL,
                  what="verify splits=%d" % s)
    check_tol(verify_gpu(case, q, scale=-0.7), oracle.verify(case.host, q, case.tables,
                                                             case.lens, -0.7),
              rel_elem=TOL_REL, what="scale")
    assert np.array_equal(verify_gpu(case, q), verify_gpu(case, q))


def test_verify_needle_at_the_last_position():
    """Every token's query points at the key of the request's last position,
    scaled so that its logit exceeds every other key's by 12: only the last
    token may attend to it; a mask aligned one position late, or at the
    start of the cache, moves the earlier tokens' outputs by O(|v|)."""
    log("verify needle")
    sq, hq, hkv, d = 4, 8, 2, 128
    case = build(P=64, hkv=hkv, d=d, hq=hq, lens=(1500,), n_out=0, seed=9)
    L = case.lens[0]
    q = np.zeros((1, sq, hq, d), np.float16)
    for h in range(hq):
        keys = case.k_rows[0][:, h // (hq // hkv)].astype(np.float64)
        u = keys[L - 1]
        dots = keys @ u
        assert dots[L - 1] > dots[:L - 1].max()
        s = 12.0 / (dots[L - 1] - dots[:L - 1].max())
        q[0, :, h] = (s * u).astype(np.float16)
    got = verify_gpu(case, q)
    ref = oracle.verify(case.host, q, case.tables, case.lens, 1.0)
    err, rel = check_tol(got, ref, rel_elem=TOL_REL, what="verify needle")
    log("  max err %.2e rel L2 %.2e" % (err, rel))
    # the last token follows the needle, the others do not see it
    vlast = oracle.dequant_vector(case.host, True, int(case.tables[0][(L - 1) // 64]), 0,
                                  (L - 1) % 64)
    assert np.linalg.norm(ref[0, sq - 1, 0] - vlast) < 0.1 * np.linalg.norm(vlast)
    for k in range(sq - 1):
        assert np.linalg.norm(ref[0, k, 0] - vlast) > 0.3 * np.linalg.norm(vlast)
