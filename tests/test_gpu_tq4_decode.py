"""GPU decode attention over TQ4 pages (jf_tq4_decode_attn) against the TQ4
oracle (oracle/tq4.py: decode_attention reconstructs every vector by
eq. codec and takes the plain softmax in float64).

Both sides read the same pool bytes: K and V rows are encoded by the oracle
(tq4.encode, tq4.pack) on the host, written into a poison-filled pool at their
pages and copied to the device, so the expected values come from the oracle
alone.

Tolerance: |o - o_ref| <= 2e-3 + 2^-10 |o_ref| elementwise and relative L2
<= 1.5e-3.  Error budget of the kernel's arithmetic:
  * the 16 centroids are rounded to fp16 once (relative <= 2^-11, the same
    error for every index of one centroid): ~4-5e-4 relative L2 on the
    outputs of this data (a float64 simulation of that rounding alone);
  * q' = H S q / 16 is exact in fp32 and enters as fp16 high + low parts;
  * p and the value weights p * norm are fp16 (2^-11 relative per weight,
    averaged over positions), the output is rounded to fp16 once (~2.8e-4);
  * accumulation in fp32.
Cases: the paper's geometry (24 query heads over 4 KV heads, d = 256,
256-position pages) from one position to the full 262,144-position window,
ragged batches, 1 and 16 query heads per KV head, split caps 1..64,
an invalid page entry, a negative scale; bitwise determinism."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import check_tol, log  # noqa: E402

from oracle import tq4  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402

DEV = "cuda"
D = 256
POISON = 0xA5
TOL = dict(atol=2e-3, rel_elem=2.0 ** -10, rel_l2=1.5e-3)
_CB = {}


def codebook():
    if "c" not in _CB:
        _CB["c"] = tq4.codebook(D)[0]
    return _CB["c"]


class Case:
    """TQ4 K and V pools built by the oracle, on the host and on the device."""

    def __init__(self, P, hkv, lens, seed, NP=None, n_out=3):
        self.P, self.hkv, self.lens = P, hkv, list(lens)
        B = len(lens)
        need = [-(-L // P) for L in lens]
        self.max_pages = max(need)
        self.NP = NP or sum(need) + 3
        rng = np.random.default_rng(seed)
        perm = rng.permutation(self.NP).astype(np.int32)
        self.tables = np.full((B, self.max_pages), -1, np.int32)
        off = 0
        for b, k in enumerate(need):
            self.tables[b, :k] = perm[off:off + k]
            off += k
        self.c = codebook()
        self.sk, self.sv = tq4.signs(D, tq4.K_SEED), tq4.signs(D, tq4.V_SEED)
        shape = (self.NP, hkv, P)
        self.kw = np.full(shape + (D // 8,), POISON * 0x01010101, np.uint32)
        self.vw = self.kw.copy()
        self.kn = np.full(shape, POISON * 0x0101, np.uint16).view(np.float16)
        self.vn = self.kn.copy()
        k, v = workloads.gen_kv(seed, sum(lens), hkv, D, n_out)
        r0 = 0
        for b, L in enumerate(lens):
            t = np.arange(L)
            pages, slots = self.tables[b][t // P], t % P
            for h in range(hkv):
                for src, words, norms, s in ((k, self.kw, self.kn, self.sk),
                                             (v, self.vw, self.vn, self.sv)):
                    idx, nrm, _ = tq4.encode(src[r0:r0 + L, h], s, self.c)
                    words[pages, h, slots] = tq4.pack(idx)
                    norms[pages, h, slots] = nrm
            r0 += L
        lay = jfkv.layout(P, hkv, D, 64, self.NP)
        self.k_pool = jfkv.TQ4Pool(lay, device=DEV)
        self.v_pool = jfkv.TQ4Pool(lay, device=DEV)
        for pool, w, n in ((self.k_pool, self.kw, self.kn), (self.v_pool, self.vw, self.vn)):
            pool.words.copy_(torch.from_numpy(w.view(np.int32)))
            pool.norms.copy_(torch.from_numpy(n))
        self.dev = {n: torch.from_numpy(a.astype(np.float32)).to(DEV)
                    for n, a in (("sk", self.sk), ("sv", self.sv), ("c", self.c))}

    def gpu(self, q, scale=1.0, max_splits=64, tables=None, lens=None, ws=None):
        tables = self.tables if tables is None else tables
        lens = self.lens if lens is None else lens
        B, hq, _ = q.shape
        if ws is None:
            ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, hq, D, max_splits),
                             dtype=torch.uint8, device=DEV)
        out = torch.empty((B, hq, D), dtype=torch.float16, device=DEV)
        jfkv.jf_tq4_decode_attn(self.k_pool, self.v_pool, self.dev["sk"], self.dev["sv"],
                                self.dev["c"], torch.from_numpy(q).to(DEV),
                                torch.from_numpy(np.ascontiguousarray(tables)).to(DEV),
                                torch.tensor(lens, dtype=torch.int32, device=DEV), scale,
                                max_splits, ws, out)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    def oracle(self, q, scale=1.0, tables=None, lens=None):
        tables = self.tables if tables is None else tables
        lens = self.lens if lens is None else lens
        out = []
        for b, L in enumerate(lens):
            kw, kn = tq4.gather(self.kw, self.kn, tables[b], L)
            vw, vn = tq4.gather(self.vw, self.vn, tables[b], L)
            out.append(tq4.decode_attention(q[b], kw, kn, vw, vn, self.sk, self.sv, self.c,
                                            scale))
        return np.array(out)


def _q(seed, B, hq):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((B, hq, D)) / np.sqrt(D)).astype(np.float16)


@pytest.mark.parametrize("P,hkv,hq,lens", [
    (256, 4, 24, (1,)),
    (256, 4, 24, (37,)),
    (256, 4, 24, (1000,)),
    (256, 4, 24, (5000,)),
    (256, 4, 24, (3000, 700)),      # ragged batch
    (64, 2, 2, (900,)),             # one query head per KV head
    (64, 2, 32, (513, 64)),         # sixteen per KV head
    (32, 1, 6, (333,)),             # 32-position pages
])
def test_tq4_decode_matches_oracle(P, hkv, hq, lens):
    log("tq4 decode P=%d hkv=%d hq=%d lens=%s" % (P, hkv, hq, lens))
    case = Case(P, hkv, lens, seed=sum(lens) + P)
    q = _q(3, len(lens), hq)
    got = case.gpu(q)
    ref = case.oracle(q)
    err, rel = check_tol(got, ref, what="tq4 decode", **TOL)
    log("  max err %.2e rel L2 %.2e" % (err, rel))


def test_tq4_split_counts_negative_scale_and_determinism():
    log("tq4 decode splits / scale / determinism")
    case = Case(256, 4, (6000,), seed=7)
    q = _q(4, 1, 24)
    ref = case.oracle(q)
    for s in (1, 3, 17, 64):
        check_tol(case.gpu(q, max_splits=s), ref, what="splits=%d" % s, **TOL)
    check_tol(case.gpu(q, scale=-0.5), case.oracle(q, scale=-0.5), what="scale -0.5", **TOL)
    a, b = case.gpu(q), case.gpu(q)
    assert np.array_equal(a, b)


def test_tq4_invalid_page_entry_is_skipped():
    log("tq4 decode invalid page")
    case = Case(64, 2, (400,), seed=8)
    q = _q(5, 1, 12)
    tab = case.tables.copy()
    tab[0, 2] = -1  # positions 128..191 are not read
    got = case.gpu(q, tables=tab)
    keep = [int(p) for i, p in enumerate(tab[0]) if i != 2]
    assert len(keep) == 6
    # drop the page: the oracle reads the remaining positions in logical order
    n = 400 - 64

    def cat(pool):
        parts = [pool[p] for p in keep]                 # [hkv][P][...] each
        return np.concatenate([np.swapaxes(x, 0, 1) for x in parts])[:n]

    ref = tq4.decode_attention(q[0], cat(case.kw), cat(case.kn), cat(case.vw), cat(case.vn),
                               case.sk, case.sv, case.c, 1.0)[None]
    check_tol(got, ref, what="invalid page", **TOL)


def test_tq4_decode_full_window():
    """The paper's full native window: 262,144 positions in 1,024 shuffled
    256-position pages, 24 query heads over 4 KV heads, d = 256."""
    log("tq4 decode full window")
    L = 262144
    case = Case(256, 4, (L,), seed=11, n_out=5)
    q = _q(6, 1, 24)
    got = case.gpu(q)
    log("  decoded; oracle")
    ref = case.oracle(q)
    err, rel = check_tol(got, ref, what="tq4 full window", **TOL)
    log("  max err %.2e rel L2 %.2e" % (err, rel))


def test_workspace_shared_with_affine_decode_and_verifier():
    """One workspace serves, in turn, affine decode, the short verifier, TQ4
    decode and affine decode again, with different head counts and split
    caps: every call leaves the completion counters zero, and every output
    equals the output of the same call on a fresh workspace bitwise."""
    from gpu_cases import build, decode_gpu
    log("workspace shared by decode, verifier and TQ4 decode")
    tq = Case(256, 4, (1500,), seed=91)
    aff = build(P=64, hkv=2, d=128, G=64, hq=8, lens=(64 * 20 + 3,), seed=92)
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, 24, D, 64), dtype=torch.uint8,
                     device=DEV)
    qa = _q(93, 1, 8)[:, :, :128].copy()
    qv = (np.random.default_rng(94).standard_normal((1, 3, 8, 128)) / 16).astype(np.float16)
    qt = _q(95, 1, 24)

    def verify(w):
        out = torch.empty((1, 3, 8, 128), dtype=torch.float16, device=DEV)
        jfkv.jf_verify_attn_q4(aff.gpu, torch.from_numpy(qv).to(DEV),
                               torch.from_numpy(aff.tables).to(DEV),
                               torch.tensor(aff.lens, dtype=torch.int32, device=DEV), 1.0, 16,
                               w, out)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    calls = [lambda w: decode_gpu(aff, qa, max_splits=64, ws=w), verify,
             lambda w: tq.gpu(qt, max_splits=64, ws=w),
             lambda w: decode_gpu(aff, qa, max_splits=5, ws=w), lambda w: tq.gpu(qt, max_splits=3, ws=w)]
    for i, call in enumerate(calls):
        got = call(ws)
        assert torch.count_nonzero(ws[:262144]).item() == 0, "call %d left a counter set" % i
        fresh = call(torch.zeros_like(ws))
        assert np.array_equal(got, fresh), "call %d differs from a fresh workspace" % i
