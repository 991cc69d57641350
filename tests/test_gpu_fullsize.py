"""GPU parity at the workloads' full sizes, in the launch configuration the
bench times (64 splits), against the CPU oracle.

Each case builds the same paged cache twice from the same seeded rows: on
the GPU with the library's quantize-append and on the host with the oracle's,
compares every pool byte (codes, scales, biases, placement), then compares
attention outputs (decode: all query heads; prefill: sampled query rows,
which the oracle computes one by one).  Tolerances as in test_gpu_decode.
Inputs are drawn on the device with torch's seeded generator (the recipe of
paper_2609_17475_amd.workloads) and copied to the host for the oracle.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import POISON, check_tol, log  # noqa: E402

import oracle  # noqa: E402
from paper_2609_17475_amd import jfkv, workloads  # noqa: E402

DEV = "cuda"


def _i32(x):
    return torch.tensor(x, dtype=torch.int32, device=DEV)


class Pools:
    """One layer's cache on the GPU (library) and on the host (oracle)."""

    def __init__(self, P, hkv, d, G, NP):
        self.lay = jfkv.layout(P, hkv, d, G, NP)
        self.gpu = jfkv.KVPool(self.lay, device=DEV, fill=POISON)
        self.host = oracle.Pool(oracle.layout(P, hkv, d, G, NP), fill=POISON)

    def append(self, k, v, cu, start, tables):
        """k, v: device fp16 [n][hkv][d]; cu, start: lists; tables: int32 numpy."""
        jfkv.jf_kv_quantize_append(self.gpu, k, v, _i32(cu), _i32(start),
                                   torch.from_numpy(np.ascontiguousarray(tables)).to(DEV))
        oracle.quantize_append(self.host, k.cpu().numpy(), v.cpu().numpy(), cu, start, tables)

    def assert_equal(self, what):
        torch.cuda.synchronize()
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            g = getattr(self.gpu, n).view(torch.uint8).cpu().numpy()
            h = getattr(self.host, n).view(np.uint8)
            if not np.array_equal(g, h):
                idx = np.nonzero(g != h)[0]
                raise AssertionError("%s %s: %d bytes differ, first at %d" % (what, n, idx.size,
                                                                             idx[0]))


def _decode_gpu(pools, q_dev, tables, lens, max_splits=64):
    B, hq, d = q_dev.shape
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, hq, d, max_splits), dtype=torch.uint8,
                     device=DEV)
    out = torch.empty((B, hq, d), dtype=torch.float16, device=DEV)
    jfkv.jf_decode_attn_q4(pools.gpu, q_dev, torch.from_numpy(np.ascontiguousarray(tables)).to(DEV),
                           _i32(lens), 1.0, max_splits, ws, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_decode_4k_full():
    """4 q heads over 1 KV head, 4,096 cached positions in 16 shuffled pages of
    a 32-page pool, 4 outlier channels; the step appends one row and attends
    to all 4,097 positions."""
    wl = workloads.WORKLOADS["decode_4k"]
    log("fullsize decode_4k")
    L = wl.seq_lens[0]
    pools = Pools(wl.page_size, wl.num_kv_heads, wl.head_dim, wl.group_size, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, wl.page_size, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, L + 1)
    table = np.array(pp.export([s], 17)[0], np.int32)
    k, v, q, _ = workloads.gen_all(wl.seed, L + 1, wl.num_kv_heads, wl.head_dim, wl.n_outlier, 1,
                                   wl.num_q_heads, 1)
    kd, vd = torch.from_numpy(k).to(DEV), torch.from_numpy(v).to(DEV)
    pools.append(kd[:L], vd[:L], [0, L], [0], table)
    pools.append(kd[L:], vd[L:], [0, 1], [L], table)
    pools.assert_equal("decode_4k")
    got = _decode_gpu(pools, torch.from_numpy(q).to(DEV), table, [L + 1])
    ref = oracle.decode(pools.host, q, table, [L + 1], 1.0)
    err, rel = check_tol(got, ref, what="decode_4k")
    log("  max err %.2e rel L2 %.2e" % (err, rel))




def test_decode_256k_full():
    """32 q / 8 KV heads, 262,144 positions in 1,024 shuffled pages, in the
    launch configuration the bench times: the cache holds 262,143 rows from
    one bulk append, and the step's row at position 262,143 is appended and
    attended to by the fused step (jf_decode_step_q4) and, on a copy of the
    pool, by the two calls (jf_kv_quantize_append, jf_decode_attn_q4).  Both
    pools equal the oracle's byte for byte, the two outputs are bitwise
    equal, and they match the oracle's decode of all 32 heads."""
    wl = workloads.WORKLOADS["decode_256k"]
    log("fullsize decode_256k")
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    L = wl.seq_lens[0]
    pools = Pools(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, L)
    table = np.array(pp.export([s], L // P)[0], np.int32)
    k, v = workloads.gen_kv_device(wl.seed, L, hkv, d, wl.n_outlier, DEV)
    q = workloads.gen_q_device(wl.seed + 1, 1, hq, d, DEV)
    pools.append(k[:L - 1], v[:L - 1], [0, L - 1], [0], table)
    torch.cuda.synchronize()
    twin = jfkv.KVPool(pools.lay, device=DEV)
    for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
        getattr(twin, n).copy_(getattr(pools.gpu, n))
    t_table = torch.from_numpy(table).to(DEV)
    lens = _i32([L])
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, hq, d, 64), dtype=torch.uint8, device=DEV)
    fused = torch.empty((1, hq, d), dtype=torch.float16, device=DEV)
    jfkv.jf_decode_step_q4(pools.gpu, k[L - 1:], v[L - 1:], q, t_table, lens, 1.0, 64, ws, fused)
    two = torch.empty_like(fused)
    jfkv.jf_kv_quantize_append(twin, k[L - 1:], v[L - 1:], _i32([0, 1]), _i32([L - 1]), t_table)
    jfkv.jf_decode_attn_q4(twin, q, t_table, lens, 1.0, 64, ws, two)
    oracle.quantize_append(pools.host, k[L - 1:].cpu().numpy(), v[L - 1:].cpu().numpy(), [0, 1],
                           [L - 1], table)
    torch.cuda.synchronize()
    log("  appended; comparing pools")
    pools.assert_equal("decode_256k fused step")
    twin_pools = Pools.__new__(Pools)
    twin_pools.gpu, twin_pools.host = twin, pools.host
    twin_pools.assert_equal("decode_256k two calls")
    got = fused.cpu().numpy()
    assert np.array_equal(got, two.cpu().numpy()), "fused step != two calls"
    log("  decoded; oracle")
    ref = oracle.decode(pools.host, q.cpu().numpy(), table, [L], 1.0)
    err, rel = check_tol(got, ref, what="decode_256k")
    log("  max err %.2e rel L2 %.2e" % (err, rel))


def test_verify_256k_full():
    """The short verifier in the bench's configuration: 32 q / 8 KV heads,
    262,144 positions in 1,024 shuffled pages whose last three positions are
    the three query tokens (appended with the cache); pools byte-equal to the
    oracle's; tokens 0 and 2 (the shortest and the longest causal window)
    against the oracle's decode of all 32 heads over L - 2 and L positions."""
    wl = workloads.WORKLOADS["verify_256k"]
    log("fullsize verify_256k")
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    L, sq = wl.seq_lens[0], wl.queries
    pools = Pools(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, L)
    table = np.array(pp.export([s], L // P)[0], np.int32)
    k, v = workloads.gen_kv_device(wl.seed, L, hkv, d, wl.n_outlier, DEV)
    q = workloads.gen_q_device(wl.seed + 1, sq, hq, d, DEV)[None]  # [1][sq][hq][d]
    pools.append(k, v, [0, L], [0], table)
    pools.assert_equal("verify_256k")
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, hq * sq, d, wl.max_splits),
                     dtype=torch.uint8, device=DEV)
    out = torch.empty_like(q)
    jfkv.jf_verify_attn_q4(pools.gpu, q, torch.from_numpy(table).to(DEV), _i32([L]), 1.0,
                           wl.max_splits, ws, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    qh = q.cpu().numpy()
    for t in (0, sq - 1):
        log("  oracle token %d" % t)
        ref = oracle.decode(pools.host, np.ascontiguousarray(qh[:, t]), table,
                            [L - sq + 1 + t], 1.0)
        err, rel = check_tol(got[:, t], ref, rel_elem=2.0 ** -11, what="verify_256k token %d" % t)
        log("  token %d max err %.2e rel L2 %.2e" % (t, err, rel))


def test_ragged_shared_prefix_full():
    """Two requests of 196,608 and 131,072 cached positions whose first
    32,768 positions are one physical copy (forked pages, reference count 2),
    each then appends its step row; one batched decode of both."""
    wl = workloads.WORKLOADS["ragged_2req"]
    log("fullsize ragged_2req")
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    La, Lb = wl.seq_lens
    pre = wl.shared_prefix
    pools = Pools(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    a = pp.create()
    pp.reserve(a, pre)
    pp.set_length(a, pre)
    b = pp.fork(a, pre)
    pp.reserve(a, La + 1)
    pp.reserve(b, Lb + 1)
    max_pages = -(-(La + 1) // P)
    tables, _ = pp.export([a, b], max_pages)
    tables = np.array(tables, np.int32)
    assert np.array_equal(tables[0, :pre // P], tables[1, :pre // P])
    n_rows = pre + (La - pre) + (Lb - pre) + 2
    k, v = workloads.gen_kv_device(wl.seed, n_rows, hkv, d, wl.n_outlier, DEV)
    q = workloads.gen_q_device(wl.seed + 1, 2, hq, d, DEV)
    # shared prefix once, then each request's own rows, then one step row each
    pools.append(k[:pre], v[:pre], [0, pre], [0], tables[:1])
    r0 = pre
    own = [La - pre, Lb - pre]
    pools.append(k[r0:r0 + sum(own)], v[r0:r0 + sum(own)], [0, own[0], own[0] + own[1]],
                 [pre, pre], tables)
    r0 += sum(own)
    pools.append(k[r0:r0 + 2], v[r0:r0 + 2], [0, 1, 2], [La, Lb], tables)
    log("  appended; comparing pools")
    pools.assert_equal("ragged_2req")
    used = pp.stats()["used"]
    assert used == (pre // P) + (La + 1 - pre + P - 1) // P + (Lb + 1 - pre + P - 1) // P
    got = _decode_gpu(pools, q, tables, [La + 1, Lb + 1])
    log("  decoded; oracle")
    ref = oracle.decode(pools.host, q.cpu().numpy(), tables, [La + 1, Lb + 1], 1.0)
    err, rel = check_tol(got, ref, what="ragged_2req")
    log("  max err %.2e rel L2 %.2e" % (err, rel))


def test_prefill_chunk_full():
    """A 2,048-row chunk (32 q / 8 KV heads) over a 65,536-position prefix in
    256 shuffled pages; sampled query rows against the oracle, then the chunk
    is appended as 8 new pages (pool bytes compared)."""
    wl = workloads.WORKLOADS["prefill_chunk"]
    log("fullsize prefill_chunk")
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    p0, T = wl.seq_lens[0], wl.chunk
    pools = Pools(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, p0 + T)
    max_pages = (p0 + T) // P
    table = np.array(pp.export([s], max_pages)[0], np.int32)[0]
    k, v = workloads.gen_kv_device(wl.seed, p0 + T, hkv, d, wl.n_outlier, DEV)
    q = workloads.gen_q_device(wl.seed + 1, T, hq, d, DEV)
    pools.append(k[:p0], v[:p0], [0, p0], [0], table[None])
    out = torch.empty((T, hq, d), dtype=torch.float16, device=DEV)
    t_table = torch.from_numpy(table).to(DEV)
    jfkv.jf_prefill_attn_q4(pools.gpu, q, k[p0:].contiguous(), v[p0:].contiguous(), t_table, p0,
                            1.0, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    rows = np.array(sorted({0, 1, 63, 64, 511, 1024, 2046, 2047} |
                           set(np.random.default_rng(7).integers(0, T, 8).tolist())), np.int32)
    log("  prefilled; oracle on %d rows" % len(rows))
    ref = oracle.prefill(pools.host, q.cpu().numpy(), k[p0:].cpu().numpy(), v[p0:].cpu().numpy(),
                         table, p0, 1.0, rows=rows)
    err, rel = check_tol(got[rows], ref, atol=2e-3, rel_elem=2.0 ** -11, rel_l2=1e-3,
                         what="prefill_chunk")
    log("  max err %.2e rel L2 %.2e" % (err, rel))
    pools.append(k[p0:], v[p0:], [0, T], [p0], table[None])
    pools.assert_equal("prefill_chunk append")


def test_prefill_reduced_chunk_every_row():
    """The prefill workload's geometry (32 q / 8 KV heads, 65,536-position
    prefix in 256 shuffled pages) with a reduced chunk of 256 rows, every
    row of every head checked against the oracle."""
    wl = workloads.WORKLOADS["prefill_chunk"]
    log("fullsize prefill_chunk, T = 256, all rows")
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    p0, T = wl.seq_lens[0], 256
    pools = Pools(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, p0 + T)
    table = np.array(pp.export([s], (p0 + T) // P)[0], np.int32)[0]
    k, v = workloads.gen_kv_device(wl.seed, p0 + T, hkv, d, wl.n_outlier, DEV)
    q = workloads.gen_q_device(wl.seed + 2, T, hq, d, DEV)
    pools.append(k[:p0], v[:p0], [0, p0], [0], table[None])
    out = torch.empty((T, hq, d), dtype=torch.float16, device=DEV)
    jfkv.jf_prefill_attn_q4(pools.gpu, q, k[p0:].contiguous(), v[p0:].contiguous(),
                            torch.from_numpy(table).to(DEV), p0, 1.0, out)
    torch.cuda.synchronize()
    log("  prefilled; oracle on all %d rows" % T)
    ref = oracle.prefill(pools.host, q.cpu().numpy(), k[p0:].cpu().numpy(), v[p0:].cpu().numpy(),
                         table, p0, 1.0)
    err, rel = check_tol(out.cpu().numpy(), ref, atol=2e-3, rel_elem=2.0 ** -11, rel_l2=1e-3,
                         what="prefill T=256")
    log("  max err %.2e rel L2 %.2e" % (err, rel))


def test_decode_32k_loop_steps():
    """32,768 cached positions, then sequential steps of append(1) + decode
    (pages reserved as the length crosses page boundaries); outputs checked
    at steps that start, cross and follow a page boundary."""
    wl = workloads.WORKLOADS["decode_32k_loop"]
    log("fullsize decode_32k_loop")
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    L0 = wl.seq_lens[0]
    n_steps = 260
    check = {0, 1, 2, 254, 255, 256, 259}
    pools = Pools(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, L0)
    pp.set_length(s, L0)
    max_pages = -(-(L0 + n_steps) // P)
    k, v = workloads.gen_kv_device(wl.seed, L0 + n_steps, hkv, d, wl.n_outlier, DEV)
    q = workloads.gen_q_device(wl.seed + 1, n_steps, hq, d, DEV)
    table = np.array(pp.export([s], max_pages)[0], np.int32)[0]
    pools.append(k[:L0], v[:L0], [0, L0], [0], table[None])
    for step in range(n_steps):
        L = L0 + step
        pp.reserve(s, L + 1)
        table = np.array(pp.export([s], max_pages)[0], np.int32)[0]
        jfkv.jf_kv_quantize_append(pools.gpu, k[L:L + 1], v[L:L + 1], _i32([0, 1]), _i32([L]),
                                   torch.from_numpy(table[None]).to(DEV))
        pp.set_length(s, L + 1)
        if step in check:
            oracle_rows = (k[:L + 1].cpu().numpy(), v[:L + 1].cpu().numpy())
            pools.host = oracle.Pool(pools.host.layout, fill=POISON)
            oracle.quantize_append(pools.host, oracle_rows[0], oracle_rows[1], [0, L + 1], [0],
                                   table[None])
            pools.assert_equal("loop step %d" % step)
            got = _decode_gpu(pools, q[step:step + 1], table[None], [L + 1])
            ref = oracle.decode(pools.host, q[step:step + 1].cpu().numpy(), table[None], [L + 1],
                                1.0)
            err, rel = check_tol(got, ref, what="loop step %d" % step)
            log("  step %d (L=%d, %d pages): max err %.2e rel L2 %.2e" % (
                step, L + 1, -(-(L + 1) // P), err, rel))
        else:
            _decode_gpu(pools, q[step:step + 1], table[None], [L + 1])
