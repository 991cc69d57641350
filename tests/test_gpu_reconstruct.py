"""GPU page -> operand reconstruction (jf_reconstruct_q4, jf_tq4_reconstruct)
against the CPU oracles.

Affine pages: bit-exact.  Every fp16 element equals oracle.reconstruct's, the
exact s * q + b rounded once to fp16; crafted (scale, code, bias) words
put the exact value just off an fp16 midpoint, where rounding an fp32
intermediate would give the other neighbour.
TQ4 pages: the kernel computes x_hat = norm * S H c[z] / 16 in fp32 (eight
butterfly stages of sums, then two products) and rounds to fp16 once; the
oracle (oracle/tq4.reconstruct) in fp64.  Bound per element: one fp16 ulp of
the reference plus the fp32 error, which is absolute on the scale of the
vector: every butterfly output is at most sum_i |c[z_i]| in magnitude, so
each of the 8 stages and 2 products adds at most 2^-24 of that (times
norm / 16): E = 10 * 2^-24 * (norm / 16) * sum_i |c[z_i]|.  At least 99% of
the elements equal the reference's own fp16 rounding.
Also: head-group offsets, group-by-group equals all heads at once (the
paper's two-head grouping, eq. groupattention), invalid pages give zeros,
tails of every size class, n_pos = 0, and an SDPA consumer over the
reconstructed operands against the oracle's prefill."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import build, log  # noqa: E402

import oracle  # noqa: E402
from oracle import tq4  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402

DEV = "cuda"
NAN16 = 0x7E00


def recon_gpu(case, n, kv0, g, table=None):
    table = case.tables[0] if table is None else table
    d = case.lay.head_dim
    k = torch.full((g, n, d), float("nan"), dtype=torch.float16, device=DEV)
    v = torch.full_like(k, float("nan"))
    jfkv.jf_reconstruct_q4(case.gpu, torch.from_numpy(np.ascontiguousarray(table)).to(DEV), n,
                           kv0, g, k, v)
    torch.cuda.synchronize()
    return k.cpu().numpy(), v.cpu().numpy()


def bits(a):
    return np.ascontiguousarray(a).view(np.uint16)


@pytest.mark.parametrize("P,hkv,d,G,L,n,kv0,g", [
    (256, 8, 128, 64, 3000, 3000, 0, 2),     # the paper's grouping: two KV heads at a time
    (256, 8, 128, 64, 3000, 3000, 6, 2),
    (256, 8, 128, 64, 3000, 1, 3, 1),
    (64, 4, 128, 32, 777, 777, 1, 3),        # ragged tail
    (64, 2, 64, 64, 100, 65, 0, 2),
    (64, 4, 256, 64, 500, 500, 0, 4),
    (128, 1, 256, 128, 129, 129, 0, 1),
])
def test_reconstruct_bit_exact(P, hkv, d, G, L, n, kv0, g):
    log("reconstruct P=%d hkv=%d d=%d G=%d n=%d kv0=%d g=%d" % (P, hkv, d, G, n, kv0, g))
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hkv, lens=(L,), seed=L + d + G)
    k, v = recon_gpu(case, n, kv0, g)
    rk, rv = oracle.reconstruct(case.host, case.tables[0], n, kv0, g)
    for what, a, b in (("K", k, rk), ("V", v, rv)):
        bad = np.nonzero(bits(a) != bits(b))
        assert bad[0].size == 0, "%s: %d elements differ, first %s gpu %04x oracle %04x" % (
            what, bad[0].size, tuple(x[0] for x in bad), bits(a)[tuple(x[0] for x in bad)],
            bits(b)[tuple(x[0] for x in bad)])


def test_groups_concatenate_to_all_heads_and_zero_length():
    case = build(P=64, hkv=4, d=128, G=64, hq=4, lens=(1000,), seed=5)
    k_all, v_all = recon_gpu(case, 1000, 0, 4)
    parts = [recon_gpu(case, 1000, 2 * j, 2) for j in range(2)]
    assert np.array_equal(bits(k_all), bits(np.concatenate([p[0] for p in parts])))
    assert np.array_equal(bits(v_all), bits(np.concatenate([p[1] for p in parts])))
    k0, v0 = recon_gpu(case, 0, 0, 4)
    assert k0.size == 0 and v0.size == 0


def test_invalid_page_gives_zeros():
    case = build(P=64, hkv=2, d=128, G=64, hq=2, lens=(300,), seed=6)
    table = case.tables[0].copy()
    table[1] = -1
    table[3] = case.lay.num_pages  # one past the pool
    k, v = recon_gpu(case, 300, 0, 2, table=table)
    rk, rv = oracle.reconstruct(case.host, table, 300, 0, 2)
    assert np.array_equal(bits(k), bits(rk)) and np.array_equal(bits(v), bits(rv))
    assert not np.any(bits(k)[:, 64:128]) and not np.any(bits(v)[:, 192:256])


def test_exact_rounding_near_fp16_midpoints():
    """Crafted (scale, code, bias) words where the fp32 FMA lands on an fp16
    midpoint (or its rounding through fp32 differs from the exact value's),
    written into both pools at the same bytes."""
    from test_oracle_reconstruct import double_rounding_cases, write_crafted
    case = build(P=64, hkv=1, d=64, G=32, hq=1, lens=(512,), seed=7)
    cases = double_rounding_cases(512, seed=1)
    write_crafted(case.host, case.tables[0], cases)
    for n in ("k_codes", "k_meta"):
        getattr(case.gpu, n).copy_(torch.from_numpy(getattr(case.host, n).view(np.uint8)).to(DEV)
                                   .view(getattr(case.gpu, n).dtype))
    k, _ = recon_gpu(case, 512, 0, 1)
    rk, _ = oracle.reconstruct(case.host, case.tables[0], 512, 0, 1)
    bad = np.nonzero(bits(k) != bits(rk))[1]
    assert bad.size == 0, "%d crafted positions differ, first %d (case %r)" % (
        bad.size, bad[0], cases[bad[0]])


# ---------------------------------------------------------------- TQ4
def _tq4_case(P, hkv, L, seed, NP=None):
    from test_gpu_tq4_decode import Case
    return Case(P, hkv, (L,), seed, NP=NP)


@pytest.mark.parametrize("P,hkv,L,n,kv0,g", [(256, 4, 1500, 1500, 0, 2), (256, 4, 1500, 1500, 2, 2),
                                             (64, 2, 333, 333, 0, 2), (32, 1, 40, 7, 0, 1)])
def test_tq4_reconstruct_matches_oracle(P, hkv, L, n, kv0, g):
    log("tq4 reconstruct P=%d hkv=%d n=%d kv0=%d g=%d" % (P, hkv, n, kv0, g))
    c = _tq4_case(P, hkv, L, seed=L + P)
    table = c.tables[0]
    k = torch.full((g, n, 256), float("nan"), dtype=torch.float16, device=DEV)
    v = torch.full_like(k, float("nan"))
    jfkv.jf_tq4_reconstruct(c.k_pool, c.v_pool, c.dev["sk"], c.dev["sv"], c.dev["c"],
                            torch.from_numpy(table).to(DEV), n, kv0, g, k, v)
    torch.cuda.synchronize()
    for what, out, words, norms, s in (("K", k, c.kw, c.kn, c.sk), ("V", v, c.vw, c.vn, c.sv)):
        got = out.cpu().numpy()
        for j in range(g):
            w, nr = tq4.gather(words[:, kv0 + j:kv0 + j + 1], norms[:, kv0 + j:kv0 + j + 1],
                               table, n)
            idx = tq4.unpack(w[:, 0])
            ref = tq4.reconstruct(idx, nr[:, 0], s, c.c)  # fp64 [n][256]
            r16 = ref.astype(np.float16)
            ulp16 = np.maximum(np.abs(np.nextafter(r16, np.float16(np.inf)).astype(np.float64)
                                      - r16.astype(np.float64)), 2.0 ** -24)
            l1 = np.abs(c.c.astype(np.float64)[idx]).sum(1)
            e32 = 10 * 2.0 ** -24 * np.abs(nr[:, 0].astype(np.float64)) / 16 * l1
            lim = ulp16 + e32[:, None]
            err = np.abs(got[j].astype(np.float64) - ref)
            assert np.all(err <= lim), "%s head %d: max err / bound %.2f" % (
                what, kv0 + j, (err / lim).max())
            same = np.mean(bits(got[j]) == bits(r16))
            assert same >= 0.99, "%s head %d: only %.4f equal to the fp16 rounding" % (
                what, kv0 + j, same)


def test_tq4_reconstruct_invalid_page():
    c = _tq4_case(64, 1, 200, seed=9)
    table = c.tables[0].copy()
    table[1] = -1
    k = torch.full((1, 200, 256), float("nan"), dtype=torch.float16, device=DEV)
    v = torch.full_like(k, float("nan"))
    jfkv.jf_tq4_reconstruct(c.k_pool, c.v_pool, c.dev["sk"], c.dev["sv"], c.dev["c"],
                            torch.from_numpy(table).to(DEV), 200, 0, 1, k, v)
    torch.cuda.synchronize()
    assert not torch.any(k[0, 64:128].view(torch.int16)).item()
    assert not torch.any(v[0, 64:128].view(torch.int16)).item()
    assert torch.isfinite(k.float()).all().item() and torch.isfinite(v.float()).all().item()


# ---------------------------------------------------------------- consumer
def test_grouped_sdpa_consumer_matches_oracle_prefill():
    """A grouped prefill as the paper runs it (eq. groupattention): for each
    two-KV-head group, reconstruct the prefix, append the chunk's fp16 rows,
    attend with the group's query heads (torch SDPA in fp32 with the causal
    offset mask), concatenate the heads; against the oracle's prefill."""
    P, hkv, hq, d, G, p0, T = 64, 4, 8, 128, 64, 700, 48
    case = build(P=P, hkv=hkv, d=d, G=G, hq=hq, lens=(p0,), seed=10)
    rng = np.random.default_rng(11)
    q = (rng.standard_normal((T, hq, d)) / np.sqrt(d)).astype(np.float16)
    kc, vc = workloads.gen_kv(12, T, hkv, d, 2)
    gq = hq // hkv
    mask = torch.ones((T, p0 + T), dtype=torch.bool, device=DEV)
    mask[:, p0:] = torch.tril(torch.ones((T, T), dtype=torch.bool, device=DEV))
    outs = []
    for j in range(hkv // 2):
        k, v = recon_gpu(case, p0, 2 * j, 2)
        K = torch.cat([torch.from_numpy(k).to(DEV),
                       torch.from_numpy(kc[:, 2 * j:2 * j + 2]).to(DEV).transpose(0, 1)], 1)
        V = torch.cat([torch.from_numpy(v).to(DEV),
                       torch.from_numpy(vc[:, 2 * j:2 * j + 2]).to(DEV).transpose(0, 1)], 1)
        K = K.float().repeat_interleave(gq, 0).contiguous()   # [2 gq][p0 + T][d]
        V = V.float().repeat_interleave(gq, 0).contiguous()
        Q = torch.from_numpy(q[:, 2 * j * gq:(2 * j + 2) * gq]).to(DEV).transpose(0, 1).float()
        O = torch.nn.functional.scaled_dot_product_attention(
            Q.contiguous(), K, V, attn_mask=mask, scale=1.0)
        outs.append(O.transpose(0, 1))                         # [T][2 gq][d]
    got = torch.cat(outs, 1).cpu().numpy()
    ref = oracle.prefill(case.host, q, kc, vc, case.tables[0], p0, 1.0)
    # operands rounded to fp16 once (2^-11 relative per element), fp32 SDPA
    err = np.abs(got - ref)
    assert np.all(err <= 2e-3 + 2.0 ** -10 * np.abs(ref)), "max err %.3e" % err.max()
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert rel <= 1e-3, "rel L2 %.3e" % rel
    log("  grouped SDPA max err %.2e rel L2 %.2e" % (err.max(), rel))
