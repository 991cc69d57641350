"""GPU fused decode step (append one row, then attend; one kernel) against
the oracle's append followed by its decode.

Bar: the pool bytes after every step equal the oracle's (codes, scales,
biases and placement bit-exact), the outputs are bitwise equal to the
library's two-call path (jf_kv_quantize_append, then jf_decode_attn_q4) and
within |o - o_ref| <= 2e-3 + 2^-11 |o_ref| of the oracle (with a few
positions an output is one outlier channel's value, |o| up to ~8, where the
fp16 output itself rounds by up to 2^-11 relative; the relative-L2 bound of
gpu_cases.check_tol still applies).
Steps cover odd and even slots (position-paired V halves), the last slot
of a page and the first slot of the next, a ragged batch, and a new row
whose page-table entry is invalid (nothing written, its positions skipped).
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import POISON, check_tol, log, pool_bytes_equal  # noqa: E402

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402

DEV = "cuda"


def _setup(P, hkv, d, G, hq, L0, n_steps, B, seed):
    """B requests of L0[b] cached rows each (own pages, shuffled pool) with
    room for n_steps more; both pools hold the same cached rows."""
    max_len = max(L0) + n_steps
    max_pages = -(-max_len // P)
    NP = B * max_pages + 2
    lay = jfkv.layout(P, hkv, d, G, NP)
    gpu = jfkv.KVPool(lay, fill=POISON)
    host = oracle.Pool(oracle.layout(P, hkv, d, G, NP), fill=POISON)
    pp = jfkv.PagePool(NP, P, shuffle_seed=seed)
    seqs = [pp.create() for _ in range(B)]
    for s, L in zip(seqs, L0):
        pp.reserve(s, L + n_steps)
        pp.set_length(s, L)
    tables = np.array(pp.export(seqs, max_pages)[0], np.int32)
    k, v = workloads.gen_kv(seed, sum(L0) + B * n_steps, hkv, d, 2)
    cu = np.concatenate([[0], np.cumsum(L0)]).astype(np.int32)
    kc, vc = k[:cu[-1]], v[:cu[-1]]
    if cu[-1]:
        jfkv.jf_kv_quantize_append(gpu, torch.from_numpy(kc).to(DEV),
                                   torch.from_numpy(vc).to(DEV),
                                   torch.tensor(cu, dtype=torch.int32, device=DEV),
                                   torch.zeros(B, dtype=torch.int32, device=DEV),
                                   torch.from_numpy(tables).to(DEV))
        oracle.quantize_append(host, kc, vc, list(cu), [0] * B, tables)
    new_k = k[cu[-1]:].reshape(n_steps, B, hkv, d)
    new_v = v[cu[-1]:].reshape(n_steps, B, hkv, d)
    return gpu, host, tables, new_k, new_v


def _run_steps(P, hkv, d, G, hq, L0, n_steps, seed, bad=None, max_splits=64):
    B = len(L0)
    gpu, host, tables, new_k, new_v = _setup(P, hkv, d, G, hq, L0, n_steps, B, seed)
    # a twin pool for the two-call path
    twin = jfkv.KVPool(gpu.layout, device=DEV)
    for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
        getattr(twin, n).copy_(getattr(gpu, n))
    gtab = torch.from_numpy(tables).to(DEV)
    rng = np.random.default_rng(seed + 7)
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, hq, d, max_splits), dtype=torch.uint8,
                     device=DEV)
    ws2 = torch.zeros_like(ws)
    for s in range(n_steps):
        lens = [L + s + 1 for L in L0]
        use_tab, use_gtab = tables, gtab
        if bad is not None and s == bad[0]:  # the new row's page entry is invalid
            use_tab = tables.copy()
            b_bad = bad[1]
            use_tab[b_bad, (lens[b_bad] - 1) // P] = -1
            use_gtab = torch.from_numpy(use_tab).to(DEV)
        log("step %d lens %s" % (s, lens))
        q = (rng.standard_normal((B, hq, d)) / np.sqrt(d)).astype(np.float16)
        kn = torch.from_numpy(np.ascontiguousarray(new_k[s])).to(DEV)
        vn = torch.from_numpy(np.ascontiguousarray(new_v[s])).to(DEV)
        qt = torch.from_numpy(q).to(DEV)
        lt = torch.tensor(lens, dtype=torch.int32, device=DEV)
        out = torch.empty((B, hq, d), dtype=torch.float16, device=DEV)
        jfkv.jf_decode_step_q4(gpu, kn, vn, qt, use_gtab, lt, 1.0, max_splits, ws, out)
        # two-call path on the twin pool
        out2 = torch.empty_like(out)
        jfkv.jf_kv_quantize_append(twin, kn, vn,
                                   torch.arange(B + 1, dtype=torch.int32, device=DEV),
                                   torch.tensor([L - 1 for L in lens], dtype=torch.int32,
                                                device=DEV), use_gtab)
        jfkv.jf_decode_attn_q4(twin, qt, use_gtab, lt, 1.0, max_splits, ws2, out2)
        # oracle: append the rows whose page entry is valid, then decode
        for b in range(B):
            if use_tab[b, (lens[b] - 1) // P] >= 0:
                oracle.quantize_append(host, new_k[s, b][None], new_v[s, b][None], [0, 1],
                                       [lens[b] - 1], use_tab[b:b + 1])
        torch.cuda.synchronize()
        bad_bytes = pool_bytes_equal(type("C", (), {"gpu": gpu, "host": host})())
        assert not bad_bytes, "step %d: %s" % (s, bad_bytes)
        got = out.cpu().numpy()
        assert np.array_equal(got, out2.cpu().numpy()), "step %d: fused != two calls" % s
        if bad is not None and s == bad[0]:
            # positions of the invalid page do not contribute: compare with the
            # oracle over the table with that page's entry dropped (attention
            # is order-free over positions)
            b_bad = bad[1]
            keep = [p for i, p in enumerate(use_tab[b_bad]) if i != (lens[b_bad] - 1) // P]
            n_drop = min(P, lens[b_bad] - ((lens[b_bad] - 1) // P) * P)
            ref_bad = oracle.decode(host, q[b_bad:b_bad + 1],
                                    np.array([keep + [-1]], np.int32), [lens[b_bad] - n_drop], 1.0)
            others = [b for b in range(B) if b != b_bad]
            if others:
                ref_o = oracle.decode(host, q[others], use_tab[others], [lens[b] for b in others],
                                      1.0)
                check_tol(got[others], ref_o, rel_elem=2.0 ** -11, what="step %d others" % s)
            check_tol(got[b_bad:b_bad + 1], ref_bad, rel_elem=2.0 ** -11,
                      what="step %d invalid page" % s)
        else:
            check_tol(got, oracle.decode(host, q, use_tab, lens, 1.0), rel_elem=2.0 ** -11,
                      what="step %d" % s)


def test_single_request_steps_across_a_page_boundary():
    # positions 61 (odd), 62 (even), 63 (last slot of page 0 of P = 64), 64 (next page), 65
    _run_steps(P=64, hkv=2, d=128, G=64, hq=8, L0=(61,), n_steps=5, seed=3)


def test_first_row_of_an_empty_request():
    _run_steps(P=64, hkv=1, d=128, G=64, hq=4, L0=(0,), n_steps=3, seed=4)


def test_ragged_batch_with_an_invalid_page_entry():
    # request 1's new row at step 1 lands on a page whose entry is -1
    _run_steps(P=256, hkv=8, d=128, G=64, hq=32, L0=(700, 1290), n_steps=3, seed=5, bad=(1, 1))


@pytest.mark.parametrize("d,G", [(64, 32), (128, 32), (128, 128), (256, 64)])
def test_other_geometries(d, G):
    _run_steps(P=64, hkv=2, d=d, G=G, hq=6, L0=(130,), n_steps=2, seed=6)


# One split (max_splits = 1) of 21 to 70 pages: every wave runs many ring
# cycles, and past 64 pages the split's page IDs take a second group.  A row
# r of the split is streamed by wave r % 8 into ring stage (r / 8) % 3 (eight
# waves, three stages at d = 128), so these lengths put the step's row into
# stages 0, 1 and 2, inside and beyond the first 64 pages (there its page ID
# is read from the table, not from the wave's current group).
@pytest.mark.parametrize("L0", [70 * 256 - 1, 65 * 256 - 101, 66 * 256 - 1, 20 * 256 + 5,
                                40 * 256 + 31])
def test_long_split_many_ring_cycles(L0):
    pos = L0
    log("long split: new row at %d, split row %d, wave %d, stage %d" % (
        pos, pos // 32, (pos // 32) % 8, (pos // 32 // 8) % 3))
    _run_steps(P=256, hkv=1, d=128, G=64, hq=4, L0=(L0,), n_steps=2, seed=9, max_splits=1)
