"""Builders shared by the GPU parity tests.

A case holds the same paged cache twice: once in device memory written by the
library's quantize-append kernel, once in host memory written by the CPU
oracle, from the same seeded rows and the same page tables (drawn from the
library's host page allocator, which is product code, not oracle code).
"""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import torch

import oracle
from paper_2609_17475_amd import jfkv, workloads

POISON = 0xA5


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class Case:
    lay: object          # jfkv.Layout
    olay: object         # oracle.Layout
    gpu: jfkv.KVPool
    host: oracle.Pool
    tables: np.ndarray   # int32 [B][max_pages]
    lens: list
    hq: int
    k_rows: list         # per request: fp16 [len][Hkv][d] (logical order)
    v_rows: list


def append_both(case: Case, k, v, cu, start, tables):
    """Append rows on the GPU (library) and on the host (oracle)."""
    dev = "cuda"
    jfkv.jf_kv_quantize_append(case.gpu, torch.from_numpy(k).to(dev), torch.from_numpy(v).to(dev),
                               torch.tensor(cu, dtype=torch.int32, device=dev),
                               torch.tensor(start, dtype=torch.int32, device=dev),
                               torch.from_numpy(np.ascontiguousarray(tables)).to(dev))
    oracle.quantize_append(case.host, k, v, cu, start, tables)


def build(P=256, hkv=1, d=128, G=64, hq=4, lens=(1000,), shared_prefix=0, n_out=2, seed=0,
          shuffle_seed=1, extra_pages=3, kv_scale=1.0) -> Case:
    """Requests with lengths `lens`; the first `shared_prefix` positions (a
    multiple of P) are one physical copy shared by every request."""
    B = len(lens)
    max_len = max(lens)
    own_pages = sum(-(-(L - shared_prefix) // P) for L in lens)
    NP = shared_prefix // P + own_pages + extra_pages
    lay = jfkv.layout(P, hkv, d, G, NP)
    olay = oracle.layout(P, hkv, d, G, NP)
    pp = jfkv.PagePool(NP, P, shuffle_seed=shuffle_seed)
    seqs = [pp.create()]
    if shared_prefix:
        pp.reserve(seqs[0], shared_prefix)
        pp.set_length(seqs[0], shared_prefix)
        for _ in range(1, B):
            seqs.append(pp.fork(seqs[0], shared_prefix))
    else:
        for _ in range(1, B):
            seqs.append(pp.create())
    for s, L in zip(seqs, lens):
        pp.reserve(s, L)
        pp.set_length(s, L)
    max_pages = -(-max_len // P)
    tables, got_lens = pp.export(seqs, max_pages)
    tables = np.array(tables, np.int32)
    assert got_lens == list(lens)

    n_rows = shared_prefix + sum(L - shared_prefix for L in lens)
    k, v = workloads.gen_kv(seed, n_rows, hkv, d, n_out)
    if kv_scale != 1.0:
        k = (k.astype(np.float32) * kv_scale).astype(np.float16)
        v = (v.astype(np.float32) * kv_scale).astype(np.float16)
    case = Case(lay, olay, jfkv.KVPool(lay, fill=POISON), oracle.Pool(olay, fill=POISON),
                tables, list(lens), hq, [], [])
    pre_k, pre_v = k[:shared_prefix], v[:shared_prefix]
    if shared_prefix:
        append_both(case, pre_k, pre_v, [0, shared_prefix], [0], tables[:1])
    own_k, own_v = k[shared_prefix:], v[shared_prefix:]
    cu = [0]
    for L in lens:
        cu.append(cu[-1] + L - shared_prefix)
    if cu[-1]:
        append_both(case, own_k, own_v, cu, [shared_prefix] * B, tables)
    for b in range(B):
        case.k_rows.append(np.concatenate([pre_k, own_k[cu[b]:cu[b + 1]]]))
        case.v_rows.append(np.concatenate([pre_v, own_v[cu[b]:cu[b + 1]]]))
    torch.cuda.synchronize()
    return case


def pool_bytes_equal(case: Case):
    """Compare every byte of the device pools with the oracle's pools."""
    names = ("k_codes", "v_codes", "k_meta", "v_meta")
    bad = []
    for n in names:
        g = getattr(case.gpu, n).view(torch.uint8).cpu().numpy()
        h = getattr(case.host, n).view(np.uint8)
        if not np.array_equal(g, h):
            idx = np.nonzero(g != h)[0]
            bad.append("%s: %d bytes differ, first at %d (gpu %02x oracle %02x)" % (
                n, idx.size, idx[0], g[idx[0]], h[idx[0]]))
    return bad


def decode_gpu(case: Case, q: np.ndarray, max_splits=64, scale=1.0, lens=None, tables=None,
               ws=None):
    """`ws`: a workspace to reuse (zero-filled once by the caller)."""
    B = q.shape[0]
    dev = "cuda"
    tables = case.tables if tables is None else tables
    lens = case.lens if lens is None else lens
    if ws is None:
        ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, q.shape[1], q.shape[2], max_splits),
                         dtype=torch.uint8, device=dev)
    out = torch.empty(q.shape, dtype=torch.float16, device=dev)
    jfkv.jf_decode_attn_q4(case.gpu, torch.from_numpy(q).to(dev),
                           torch.from_numpy(np.ascontiguousarray(tables)).to(dev),
                           torch.tensor(lens, dtype=torch.int32, device=dev), scale, max_splits,
                           ws, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def decode_oracle(case: Case, q: np.ndarray, scale=1.0, lens=None, tables=None):
    tables = case.tables if tables is None else tables
    lens = case.lens if lens is None else lens
    return oracle.decode(case.host, q, tables, lens, scale)


def check_tol(got16: np.ndarray, ref: np.ndarray, atol=2e-3, rel_l2=1e-3, rel_elem=0.0,
              what=""):
    """|got - ref| <= atol + rel_elem*|ref| elementwise (atol 2e-3 is the bound
    for fp16 outputs with fp32 accumulation), and relative L2 error <= rel_l2.

    The relative L2 cap of 1e-3 follows from the decode arithmetic: the
    probabilities p are fp16, but the same rounded p enter the numerator and
    the denominator, so their rounding only perturbs the weights (relative
    2^-11 each, averaged over positions); W = p * scale is rounded to fp16
    once and multiplies centred codes (code - 8), so each position's value
    term moves by at most 2^-11 * 7.5 * p * scale, averaged over positions;
    the bias terms are exact fp32 products; the output is rounded to fp16
    once (rms ~2^-11 / sqrt(3) = 2.8e-4 relative).  Measured: 2e-4 to 5e-4.
    Short windows with an outlier group (scale ~3, a few hundred positions)
    reach max |err| ~1e-3, inside atol."""
    got = got16.astype(np.float64)
    err = np.abs(got - ref)
    lim = atol + rel_elem * np.abs(ref)
    worst = np.unravel_index(np.argmax(err - lim), err.shape)
    assert np.all(np.isfinite(got)), what + ": non-finite output"
    assert np.all(err <= lim), "%s: max err %.3e at %s (got %r ref %r)" % (
        what, err.max(), worst, got[worst], ref[worst])
    r = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert r <= rel_l2, "%s: rel L2 %.3e" % (what, r)
    return float(err.max()), float(r)
