#!/usr/bin/env python
"""Decode attention over a 4-bit paged KV cache at a 262,144-position window.

One step (the default workload, decode_256k) = one decode step of one layer
for one request: host page reservation, then one launch of the fused step
(jf_decode_step_q4): quantize-append of the step's new K/V row at position
262,143, split-K decode attention of 32 query heads (8 KV heads, d=128, GQA
4:1) over all 262,144 positions through a 1,024-entry shuffled page table,
and the log-sum-exp combine.  Inputs (cache, page table, the steps' new rows
and queries) are resident in HBM before timing.  Consecutive steps use
different layers' pools (--layers, default 8 x 302 MB), so a step never finds
the previous step's cache lines in the 256 MB last-level cache, as in a model
whose layers each own a pool.

Prints one JSON line: KV positions/s/layer (value), HBM GB/s of the step
kernel against the 8 TB/s peak (roofline), and the CPU oracle timed on a
bounded sample, on one core and on all of them (cpu_baseline).

Other workloads (--workload) print their own line:
  decode_4k        4 q / 1 KV head, 4,096 cached positions + 1 appended row
                   (launch-bound, cache-resident: reported in us and GB/s)
  decode_32k_loop  32 q / 8 KV heads, 32,768 cached positions then 6,144
                   sequential steps of append + attend (pages reserved as the
                   length crosses page boundaries); cache-resident
  ragged_2req      two requests of 196,608 and 131,072 positions sharing a
                   32,768-position prefix, one batched fused step (+1 row each)
  prefill_chunk    2,048-row chunk over a 65,536-position prefix (MFMA roofline)
  quantize_bulk    262,143 rows x 8 KV heads quantize-append (HBM roofline)
  tq4_encode_bulk  TQ4 encode-append, 262,143 rows x 4 KV heads, d 256
  tq4_decode_256k  TQ4 decode attention in the paper's geometry (24 q / 4 KV
                   heads, d 256) over 262,144 positions
  verify_256k      the short packed verifier: 3 causal query tokens over
                   decode_256k's 262,144-position cache
  reconstruct_grouped  page -> operand reconstruction of a 2-KV-head group
                   over prefill_chunk's prefix (HBM roofline), the grouped
                   reconstruct + SDPA prefill against the fused prefill, and
                   TQ4 reconstruction at 196,608 positions
  snapshot_224k    16 layers x 229,376 positions saved to a file and restored
                   through 64 MiB staging buffers (pack kernel: HBM roofline)
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn KV positions/s/layer + achieved HBM GB/s (% of peak) at 256K ctx"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 / bf16 matrix peak


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _host():
    return {"host_cpus": len(os.sched_getaffinity(0)), "cpu_model": _cpu_model()}


CSRC = os.path.join(ROOT, "paper_2609_17475_amd", "csrc")
TRAFFIC_PROFILES = {  # kernel -> (counter profile, source it was taken from)
    "decode": (os.path.join(ROOT, "profiles", "decode_kernel_decode_256k_traffic.md"), "decode.hip"),
    "quantize": (os.path.join(ROOT, "profiles", "quantize_rows_kernel_quantize_bulk.md"),
                 "quantize.hip"),
}


def measured_traffic(kernel="decode"):
    """HBM bytes per call from the committed counter profile (FETCH_SIZE and
    WRITE_SIZE, calibrated), or None when the kernel's source has changed
    since the counters were taken."""
    import hashlib
    path, src = TRAFFIC_PROFILES[kernel]
    try:
        text = open(path).read()
    except OSError:
        return None
    sha = hashlib.sha256(open(os.path.join(CSRC, src), "rb").read()).hexdigest()
    m_sha = re.search(kernel + r"_source_sha256:\s*([0-9a-f]{64})", text)
    m_b = re.search(r"traffic_bytes_per_call:\s*([0-9]+)", text)
    if not m_sha or not m_b or m_sha.group(1) != sha:
        return None
    return int(m_b.group(1))


def copy_calibration(n_bytes: int, reps: int):
    """A plain device copy of known size, run under the FETCH_SIZE/WRITE_SIZE
    counters to scale them to bytes."""
    import torch
    dev = torch.device("cuda:0")
    src = torch.ones(n_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n_bytes, "copy_bytes_written": n_bytes, "reps": reps}),
          flush=True)


def read_calibration(n_bytes: int, args):
    """The practical read ceiling: jf_calib_read_stream (the kernels' 16-byte
    non-temporal loads, nothing else) over n_bytes, 8 rotated buffers, timed
    with HIP events over 20 and over 200 back-to-back calls per grid size."""
    import torch
    from paper_2609_17475_amd import jfkv
    dev = torch.device("cuda:0")
    n_bytes -= n_bytes % 16
    bufs = [torch.ones(n_bytes, dtype=torch.uint8, device=dev) for _ in range(8)]
    sink = torch.zeros(4, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    rows = []
    for blocks in (256, 1024, 2048):
        for i in range(8):
            jfkv.jf_calib_read_stream(bufs[i], blocks, sink, stream)
        torch.cuda.synchronize()
        for reps in (20, 200):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for i in range(reps):
                jfkv.jf_calib_read_stream(bufs[i % 8], blocks, sink, stream)
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            rows.append({"blocks": blocks, "reps": reps, "us_per_call": round(us, 2),
                         "GBs": round(n_bytes / (us * 1e-6) / 1e9, 1),
                         "frac_of_8TBs": round(n_bytes / (us * 1e-6) / 8e12, 4)})
    print(json.dumps({"read_calibration": {"bytes": n_bytes, "buffers": 8, "threads_per_block": 512,
                                           "load": "16-byte non-temporal, 8 in flight per lane",
                                           "results": rows}}), flush=True)


def _timed(calls, warmup, steps, stream):
    """Mean HIP-event duration (us) of each step's calls, and wall us/step."""
    import numpy as np
    import torch
    for i in range(warmup):
        for c in calls[i % len(calls)]:
            c()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls[0]) + 1)]
          for _ in range(steps)]
    t0 = time.perf_counter()
    for s in range(steps):
        ev[s][0].record(stream)
        for i, c in enumerate(calls[(warmup + s) % len(calls)]):
            c()
            ev[s][i + 1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e6
    per = [float(np.mean([ev[s][i].elapsed_time(ev[s][i + 1]) * 1e3 for s in range(steps)]))
           for i in range(len(calls[0]))]
    return per, wall


def _back_to_back(step, warmup, steps, stream):
    """Run warmup steps, then time `steps` steps back to back: one HIP event
    pair on the kernels' stream brackets them (GPU us per step, launch gaps
    included) and the host clock between two synchronizations (wall)."""
    import torch
    for s in range(warmup):
        step(s)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for s in range(warmup, warmup + steps):
        step(s)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e6
    return e0.elapsed_time(e1) * 1e3 / steps, wall


def _repeat(fn, min_seconds):
    """Call fn until min_seconds have passed; (calls, seconds)."""
    n = 0
    t0 = time.perf_counter()
    while True:
        fn()
        n += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            return n, dt


# --------------------------------------------------------------- fused steps
DECODE_STEP_WORKLOADS = ("decode_256k", "decode_4k", "ragged_2req")


def _build_decode_case(name, args, n_steps_total):
    """Pools (args.layers copies), page tables, the steps' rows and queries of
    a fused-step workload.  Returns a dict."""
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS[name]
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    if name == "decode_256k":
        window = args.positions or wl.seq_lens[0]
        if window < P or window % P:
            raise SystemExit("--positions must be a positive multiple of the page size (%d)" % P)
        cached = [window - 1]  # the step's row lands in the window's last slot
        NP = window // P + (wl.pool_pages - wl.seq_lens[0] // P)
    else:
        cached = list(wl.seq_lens)
        NP = wl.pool_pages
    B = len(cached)
    lens = [c + 1 for c in cached]
    pre = wl.shared_prefix
    pp = jfkv.PagePool(NP, P, shuffle_seed=wl.seed)
    seqs = [pp.create()]
    if pre:
        pp.reserve(seqs[0], pre)
        pp.set_length(seqs[0], pre)
        seqs += [pp.fork(seqs[0], pre) for _ in range(1, B)]
    else:
        seqs += [pp.create() for _ in range(1, B)]
    for s, c in zip(seqs, cached):
        pp.reserve(s, c + 1)
        pp.set_length(s, c)
    max_pages = -(-max(lens) // P)
    table = np.array(pp.export(seqs, max_pages)[0], np.int32)
    t_table = torch.from_numpy(table).to(dev)
    # rows: the shared prefix once, each request's own cached rows, then one
    # new row per request and step
    own = [c - pre for c in cached]
    n_rows = pre + sum(own) + B * n_steps_total
    t0 = time.perf_counter()
    k, v = workloads.gen_kv_device(wl.seed, n_rows, hkv, d, wl.n_outlier, dev)
    q = workloads.gen_q_device(wl.seed + 1, n_steps_total * B, hq, d, dev)
    lay = jfkv.layout(P, hkv, d, G, NP)
    pools = [jfkv.KVPool(lay, device=dev) for _ in range(args.layers)]
    i32 = lambda x: torch.tensor(x, dtype=torch.int32, device=dev)  # noqa: E731
    if pre:
        jfkv.jf_kv_quantize_append(pools[0], k[:pre], v[:pre], i32([0, pre]), i32([0]),
                                   t_table[:1].contiguous())
    cu = [0]
    for o in own:
        cu.append(cu[-1] + o)
    if cu[-1]:
        jfkv.jf_kv_quantize_append(pools[0], k[pre:pre + cu[-1]], v[pre:pre + cu[-1]], i32(cu),
                                   i32([pre] * B), t_table)
    torch.cuda.synchronize()
    for p in pools[1:]:
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            getattr(p, n).copy_(getattr(pools[0], n))
    torch.cuda.synchronize()
    log("%s: inputs and %d layer pools built in %.1fs" % (name, args.layers,
                                                         time.perf_counter() - t0))
    new0 = pre + cu[-1]
    return dict(wl=wl, P=P, hkv=hkv, hq=hq, d=d, G=G, B=B, cached=cached, lens=lens, pre=pre,
                NP=NP, pp=pp, seqs=seqs, table=table, t_table=t_table, k=k, v=v, q=q,
                pools=pools, new0=new0, own=own, cu=cu, dev=dev)


def _decode_oracle_baseline(c, name, args):
    """The oracle (C, fp64 attention) on the same step: append each request's
    row, attend; all cores on the full step, one core on a sample of the
    first positions of request 0."""
    import numpy as np
    import oracle
    k_all, v_all = c["k"].cpu().numpy(), c["v"].cpu().numpy()
    q0 = c["q"][:c["B"]].cpu().numpy()
    P, hkv, d, G, B = c["P"], c["hkv"], c["d"], c["G"], c["B"]
    pre, cu, new0 = c["pre"], c["cu"], c["new0"]
    table = c["table"]

    def build(lens_cached, b_rows):
        pool = oracle.Pool(oracle.layout(P, hkv, d, G, c["NP"]))
        if pre:
            oracle.quantize_append(pool, k_all[:pre], v_all[:pre], [0, pre], [0], table[:1])
        for b in b_rows:
            n = lens_cached[b] - pre
            if n > 0:
                s = pre + cu[b]
                oracle.quantize_append(pool, k_all[s:s + n], v_all[s:s + n], [0, n], [pre],
                                       table[b:b + 1])
        return pool

    def step(pool, lens_cached, b_rows):
        for b in b_rows:
            r = new0 + b
            oracle.quantize_append(pool, k_all[r:r + 1], v_all[r:r + 1], [0, 1],
                                   [lens_cached[b]], table[b:b + 1])
        oracle.decode(pool, q0[b_rows], table[b_rows], [lens_cached[b] + 1 for b in b_rows], 1.0)

    rows = list(range(B))
    all_cores = oracle.max_threads()
    pool = build(c["cached"], rows)
    n, dt = _repeat(lambda: step(pool, c["cached"], rows), args.cpu_seconds)
    positions = sum(l_ + 1 for l_ in c["cached"])
    res = {"value": positions * n / dt, "unit": "KV positions/s/layer", "cores": all_cores,
           "kind": "oracle", "seconds": dt, "steps": n,
           "sample": "%d full step(s) of %s (quantize-append of the step rows + fp64 "
                     "attention of all %d query heads over all %d positions), %d threads" % (
                         n, name, c["hq"], positions, all_cores)}
    res.update(_host())
    # one core, on the first positions of request 0 (the oracle's cost is
    # linear in the positions)
    n1 = min(args.cpu_sample_1t, c["cached"][0])
    if n1 > 0:
        lens1 = [n1] + c["cached"][1:]
        pool1 = build(lens1, [0])
        oracle.set_threads(1)
        try:
            m, dt1 = _repeat(lambda: step(pool1, lens1, [0]), args.cpu_seconds_1t)
        finally:
            oracle.set_threads(all_cores)
        res["single_thread"] = {"value": (n1 + 1) * m / dt1, "unit": "KV positions/s/layer",
                                "cores": 1, "seconds": dt1, "steps": m,
                                "sample": "request 0's first %d positions + the step row, "
                                          "all %d query heads" % (n1, c["hq"])}
    return res


def bench_decode_steps(name, args):
    """A fused decode step (append one row per request, attend) repeated on
    rotated layer pools, timed back to back."""
    import torch
    from paper_2609_17475_amd import jfkv
    n_steps_total = args.warmup + args.steps
    c = _build_decode_case(name, args, n_steps_total)
    P, hkv, hq, d, G, B = c["P"], c["hkv"], c["hq"], c["d"], c["G"], c["B"]
    stream = torch.cuda.current_stream()
    lens_t = torch.tensor(c["lens"], dtype=torch.int32, device=c["dev"])
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(B, hq, d, args.max_splits),
                     dtype=torch.uint8, device=c["dev"])
    out = torch.empty((n_steps_total, B, hq, d), dtype=torch.float16, device=c["dev"])
    calls = []
    for s in range(n_steps_total):
        pool = c["pools"][s % args.layers]
        r = c["new0"] + B * s
        calls.append(jfkv.bind_decode_step(pool, c["k"][r:r + B], c["v"][r:r + B],
                                           c["q"][B * s:B * s + B], c["t_table"], lens_t, 1.0,
                                           args.max_splits, ws, out[s], stream))
    pp, seqs, lens = c["pp"], c["seqs"], c["lens"]

    def step(s):
        for sq, L in zip(seqs, lens):
            pp.reserve(sq, L)  # host page reservation (satisfied: the rows' pages exist)
        calls[s]()

    gpu_us, wall_us = _back_to_back(step, args.warmup, args.steps, stream)
    assert torch.isfinite(out.float()).all().item(), "non-finite decode output"
    bpp = 2 * hkv * (d // 2 + 4 * d // G)            # bytes per position and layer
    logical = sum(lens)
    unique = logical - (B - 1) * c["pre"]            # shared prefix pages read through each table
    nbytes = unique * bpp + B * (2 * hkv * d * 2 + bpp)  # + the rows read and written
    achieved = nbytes / (gpu_us * 1e-6) / 1e9
    wl = c["wl"]
    L0 = lens[0]
    window = name == "decode_256k" and L0 == wl.seq_lens[0]
    label = name if (name != "decode_256k" or window) else "decode_%d" % L0
    split_cap = min(args.max_splits,
                    max(1, torch.cuda.get_device_properties(0).multi_processor_count
                        // (hkv * -(-(hq // hkv) // jfkv.decode_head_chunk(d, G, hq // hkv)))))
    result = {
        "metric": METRIC if window else "decode-attn KV positions/s/layer (%s)" % label,
        "value": logical / (wall_us * 1e-6), "unit": "KV positions/s/layer", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall_us / 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u4 codes x f16 -> f32", "data": "synthetic",
        "config": {"workload": label, "positions": lens, "batch": B, "num_q_heads": hq,
                   "num_kv_heads": hkv, "head_dim": d, "page_size": P, "group_size": G,
                   "shared_prefix": c["pre"], "max_splits": args.max_splits,
                   "splits_used": [min(split_cap, -(-L // P)) for L in lens],
                   "layers_rotated": args.layers,
                   "step": "jf_decode_step_q4 (append + attend, one kernel)"},
        "hbm_GBs": achieved, "hbm_pct_of_peak": 100.0 * achieved / HBM_PEAK_GBS,
        "us_per_step": {"step_kernel": gpu_us, "wall": wall_us},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic() if window else None,
                     "kernel": "decode_kernel, fused step (row append, split-K partials, "
                               "in-kernel combine)",
                     "algorithmic_bytes": nbytes,
                     "bytes_per_position": bpp, "unique_positions": unique},
    }
    if name == "decode_4k":
        result["roofline"]["regime"] = ("launch-bound: %.1f MB per step stays in the "
                                        "last-level cache" % (nbytes / 1e6))
    log("%s: gpu %.2f us/step, wall %.2f us/step, %.0f GB/s" % (label, gpu_us, wall_us,
                                                                achieved))
    if args.cpu_seconds > 0:
        try:
            result["cpu_baseline"] = _decode_oracle_baseline(c, label, args)
        except Exception as e:  # the baseline is a report, not the product
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def bench_decode_loop(args):
    """decode_32k_loop: 32,768 cached positions, then 6,144 sequential steps;
    each step reserves pages on the host (a new page every 256 steps, its
    table entry copied to the device), then one fused step appends the row at
    position L and attends L + 1 positions.  All steps are timed."""
    import numpy as np
    import torch
    import oracle
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS["decode_32k_loop"]
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    L0, n_steps = wl.seq_lens[0], wl.steps
    max_pages = -(-(L0 + n_steps) // P)
    k, v = workloads.gen_kv_device(wl.seed, L0 + n_steps, hkv, d, wl.n_outlier, dev)
    q = workloads.gen_q_device(wl.seed + 1, n_steps, hq, d, dev)
    lay = jfkv.layout(P, hkv, d, G, wl.pool_pages)
    stream = torch.cuda.current_stream()
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, hq, d, args.max_splits),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((n_steps, 1, hq, d), dtype=torch.float16, device=dev)
    i32 = lambda x: torch.tensor(x, dtype=torch.int32, device=dev)  # noqa: E731

    def setup():
        pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
        s = pp.create()
        pp.reserve(s, L0)
        pp.set_length(s, L0)
        table = np.array(pp.export([s], max_pages)[0], np.int32)
        t_table = torch.from_numpy(table).to(dev)
        pool = jfkv.KVPool(lay, device=dev)
        jfkv.jf_kv_quantize_append(pool, k[:L0], v[:L0], i32([0, L0]), i32([0]), t_table)
        lens = torch.tensor([L0 + 1 + i for i in range(n_steps)], dtype=torch.int32,
                            device=dev).view(n_steps, 1)
        calls = [jfkv.bind_decode_step(pool, k[L0 + i:L0 + i + 1], v[L0 + i:L0 + i + 1],
                                       q[i:i + 1].view(1, hq, d), t_table, lens[i], 1.0,
                                       args.max_splits, ws, out[i], stream)
                 for i in range(n_steps)]
        torch.cuda.synchronize()
        return pp, s, table, t_table, pool, lens, calls

    def run(n, state):
        pp, s, table, t_table, pool, lens, calls = state
        pinned = torch.empty(max_pages, dtype=torch.int32).pin_memory()
        n_pages = -(-L0 // P)
        for i in range(n):
            L = L0 + i
            if (L + 1 + P - 1) // P > n_pages:  # the row opens a new page
                pp.reserve(s, L + 1)
                tab = pp.export([s], max_pages)[0][0]
                n_pages += 1
                pinned[n_pages - 1] = tab[n_pages - 1]
                t_table[0, n_pages - 1:n_pages].copy_(pinned[n_pages - 1:n_pages],
                                                      non_blocking=True)
            calls[i]()
            pp.set_length(s, L + 1)

    warm = setup()
    run(min(64, n_steps), warm)  # warm-up on a separate pool
    torch.cuda.synchronize()
    del warm
    state = setup()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    run(n_steps, state)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / n_steps * 1e6
    gpu = e0.elapsed_time(e1) * 1e3 / n_steps
    assert torch.isfinite(out.float()).all().item(), "non-finite decode output"
    bpp = 2 * hkv * (d // 2 + 4 * d // G)
    positions = sum(L0 + 1 + i for i in range(n_steps))
    nbytes = positions * bpp + n_steps * (2 * hkv * d * 2 + bpp)
    eff = nbytes / (gpu * 1e-6 * n_steps) / 1e9
    result = {
        "metric": "decode-attn KV positions/s/layer (decode_32k_loop: 6,144 sequential steps)",
        "value": positions / (wall * 1e-6 * n_steps), "unit": "KV positions/s/layer",
        "n_gpus": 1, "steps": n_steps, "warmup": 64, "ms_per_step": wall / 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u4 codes x f16 -> f32", "data": "synthetic",
        "config": {"workload": "decode_32k_loop", "positions": [L0 + 1, L0 + n_steps],
                   "num_q_heads": hq, "num_kv_heads": hkv, "head_dim": d, "page_size": P,
                   "group_size": G, "max_splits": args.max_splits,
                   "step": "host reserve (+ page-table entry copy every 256 steps) + "
                           "jf_decode_step_q4"},
        "us_per_step": {"gpu": gpu, "wall": wall},
        "roofline": {"bound": "hbm", "achieved": eff, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": eff / HBM_PEAK_GBS, "traffic": None, "kernel": "decode_kernel",
                     "algorithmic_bytes": nbytes,
                     "regime": "effective GB/s: the 38-45 MB working set stays in the "
                               "256 MB last-level cache across steps"},
    }
    log("decode_32k_loop: gpu %.2f us/step, wall %.2f us/step" % (gpu, wall))
    if args.cpu_seconds > 0:
        try:  # the oracle over the first 64 steps, extrapolated linearly in positions
            kh, vh, qh = k.cpu().numpy(), v.cpu().numpy(), q.cpu().numpy()
            pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
            s = pp.create()
            pp.reserve(s, L0 + 64)
            table = np.array(pp.export([s], max_pages)[0], np.int32)
            opool = oracle.Pool(oracle.layout(P, hkv, d, G, wl.pool_pages))
            oracle.quantize_append(opool, kh[:L0], vh[:L0], [0, L0], [0], table)
            t0 = time.perf_counter()
            pos = 0
            for i in range(64):
                L = L0 + i
                oracle.quantize_append(opool, kh[L:L + 1], vh[L:L + 1], [0, 1], [L], table)
                oracle.decode(opool, qh[i:i + 1], table, [L + 1], 1.0)
                pos += L + 1
            dt = time.perf_counter() - t0
            result["cpu_baseline"] = dict(
                value=pos / dt, unit="KV positions/s/layer", cores=oracle.max_threads(),
                kind="oracle", seconds=dt, steps=64,
                sample="the first 64 of the 6,144 steps (append + fp64 attention of 32 heads "
                       "over 32,769..32,832 positions); the full loop extrapolates to %.1f s"
                       % (dt * positions / pos), **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


# --------------------------------------------------------------- prefill
def bench_prefill(args):
    """Chunked prefill: a 2,048-row chunk (32 q / 8 KV heads, d 128) attends
    to a 65,536-position 4-bit prefix in 256 shuffled pages plus itself
    (causal), then the chunk is appended as 8 pages.  MFMA roofline over the
    attention kernel: FLOP = 4 d Hq sum_i (p0 + i + 1)."""
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS["prefill_chunk"]
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    p0, T = wl.seq_lens[0], wl.chunk
    lay = jfkv.layout(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, p0 + T)
    table_np = np.array(pp.export([s], (p0 + T) // P)[0], np.int32)
    table = torch.from_numpy(table_np).to(dev)
    k, v = workloads.gen_kv_device(wl.seed, p0 + T, hkv, d, wl.n_outlier, dev)
    q = workloads.gen_q_device(wl.seed + 1, T, hq, d, dev)
    pool = jfkv.KVPool(lay, device=dev)
    jfkv.jf_kv_quantize_append(pool, k[:p0], v[:p0], torch.tensor([0, p0], dtype=torch.int32,
                                                                  device=dev),
                               torch.tensor([0], dtype=torch.int32, device=dev), table)
    kc, vc = k[p0:].contiguous(), v[p0:].contiguous()
    out = torch.empty((T, hq, d), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    attn = jfkv.bind_prefill(pool, q, kc, vc, table[0].contiguous(), p0, 1.0, out, stream)
    app = jfkv.bind_quantize_append(pool, kc, vc, torch.tensor([0, T], dtype=torch.int32,
                                                               device=dev),
                                    torch.tensor([p0], dtype=torch.int32, device=dev), table,
                                    stream)
    steps = max(1, args.steps // 3)
    (t_attn, t_app), wall = _timed([[attn, app]], args.warmup, steps, stream)
    flop = 4.0 * d * hq * sum(p0 + i + 1 for i in range(T))
    achieved = flop / (t_attn * 1e-6) / 1e12
    assert torch.isfinite(out.float()).all().item(), "non-finite prefill output"
    result = {
        "metric": "chunked-prefill attention TFLOP/s over a 4-bit paged prefix",
        "value": flop / (wall * 1e-6) / 1e12, "unit": "TFLOP/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": wall / 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u4 codes x f16 -> f32 (MFMA f16)",
        "data": "synthetic",
        "config": {"workload": "prefill_chunk", "chunk": T, "prefix": p0, "num_q_heads": hq,
                   "num_kv_heads": hkv, "head_dim": d, "page_size": P, "group_size": G},
        "us_per_step": {"attention": t_attn, "append": t_app, "wall": wall},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_F16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / MFMA_F16_PEAK_TFLOPS, "traffic": None,
                     "kernel": "prefill_kernel", "algorithmic_flop": flop}}
    if args.cpu_seconds > 0:
        try:  # the oracle on 64 evenly spaced query rows, scaled to the chunk
            import oracle
            opool = oracle.Pool(oracle.layout(P, hkv, d, G, wl.pool_pages))
            kh, vh = k.cpu().numpy(), v.cpu().numpy()
            oracle.quantize_append(opool, kh[:p0], vh[:p0], [0, p0], [0], table_np)
            rows = np.linspace(0, T - 1, 64).astype(np.int32)
            t0 = time.perf_counter()
            oracle.prefill(opool, q.cpu().numpy(), kh[p0:], vh[p0:], table_np[0], p0, 1.0,
                           rows=rows)
            dt = time.perf_counter() - t0
            f_rows = 4.0 * d * hq * float(sum(p0 + int(i) + 1 for i in rows))
            result["cpu_baseline"] = dict(
                value=f_rows / dt / 1e12, unit="TFLOP/s", cores=oracle.max_threads(),
                kind="oracle", seconds=dt,
                sample="64 evenly spaced query rows of the chunk (all 32 heads, fp64), "
                       "FLOP counted as in the roofline", **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


# --------------------------------------------------------------- bulk encodes
def bench_quantize_bulk(args):
    """Bulk quantize-append of 262,143 rows x 8 KV heads (the cache of the
    256K decode workload) into 1,024 shuffled pages; HBM roofline over the
    kernel: 2 x 256 B read and 2 x (64 + 8) B written per (row, KV head)."""
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS["decode_256k"]
    P, hkv, d, G = wl.page_size, wl.num_kv_heads, wl.head_dim, wl.group_size
    L = wl.seq_lens[0] - 1
    lay = jfkv.layout(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s = pp.create()
    pp.reserve(s, L + 1)
    table_np = np.array(pp.export([s], (L + 1) // P)[0], np.int32)
    table = torch.from_numpy(table_np).to(dev)
    k, v = workloads.gen_kv_device(wl.seed, L, hkv, d, wl.n_outlier, dev)
    pools = [jfkv.KVPool(lay, device=dev) for _ in range(4)]
    cu = torch.tensor([0, L], dtype=torch.int32, device=dev)
    st = torch.tensor([0], dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    calls = [[jfkv.bind_quantize_append(p, k, v, cu, st, table, stream)] for p in pools]
    steps = max(1, args.steps // 4)
    (t_q,), wall = _timed(calls, args.warmup, steps, stream)
    nbytes = L * hkv * 2 * (2 * d + d // 2 + 4 * d // G)
    achieved = nbytes / (t_q * 1e-6) / 1e9
    result = {
        "metric": "bulk quantize-append GB/s (262,143 rows x 8 KV heads)",
        "value": nbytes / (wall * 1e-6) / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": wall / 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16 -> u4 codes + f16 meta",
        "data": "synthetic",
        "config": {"workload": "quantize_bulk", "rows": L, "num_kv_heads": hkv, "head_dim": d,
                   "page_size": P, "group_size": G},
        "us_per_step": {"quantize": t_q, "wall": wall},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic("quantize"),
                     "kernel": "quantize_rows_kernel", "algorithmic_bytes": nbytes}}
    if args.cpu_seconds > 0:
        try:  # the whole bulk append in the oracle
            import oracle
            opool = oracle.Pool(oracle.layout(P, hkv, d, G, wl.pool_pages))
            kh, vh = k.cpu().numpy(), v.cpu().numpy()
            t0 = time.perf_counter()
            oracle.quantize_append(opool, kh, vh, [0, L], [0], table_np)
            dt = time.perf_counter() - t0
            result["cpu_baseline"] = dict(value=nbytes / dt / 1e9, unit="GB/s", cores=1,
                                          kind="oracle", seconds=dt,
                                          sample="the full append (262,143 rows x 8 KV heads, "
                                                 "single-threaded loop), same bytes", **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def _tq4_inputs(P, hkv, L, NP, seed, dev):
    import numpy as np
    import torch
    rng = np.random.default_rng(seed)
    table = rng.permutation(NP)[:-(-L // P)][None].astype(np.int32)
    signs = [torch.tensor(np.where(rng.random(256) < 0.5, -1.0, 1.0), dtype=torch.float32,
                          device=dev) for _ in range(2)]
    return table, signs


def bench_tq4_encode(args):
    """TQ4 bulk encode-and-append of 262,143 rows x 4 KV heads (d 256, the
    paper's full-attention geometry) into 1,024 shuffled pages; HBM roofline
    over the kernel: 512 B read and 128 + 2 B written per vector."""
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv
    dev = torch.device("cuda:0")
    P, hkv, d, L = 256, 4, 256, 262143
    NP = L // P + 1 + 8
    table_np, (signs, _) = _tq4_inputs(P, hkv, L + 1, NP, 4, dev)
    table = torch.from_numpy(table_np).to(dev)
    g = torch.Generator(device=dev).manual_seed(4)
    x = torch.randn((L, hkv, d), generator=g, device=dev, dtype=torch.float32).half()
    # signs and centroids are inputs of the kernel: any +-1 vector and any
    # ascending 16 values time the same; these are fixed stand-ins
    cents = torch.linspace(-0.17, 0.17, 16, dtype=torch.float32, device=dev)
    lay = jfkv.layout(P, hkv, d, 64, NP)
    pools = [jfkv.TQ4Pool(lay, device=dev) for _ in range(4)]
    cu = torch.tensor([0, L], dtype=torch.int32, device=dev)
    st = torch.tensor([0], dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    calls = [[jfkv.bind_tq4_encode_append(p, x, signs, cents, cu, st, table, stream)]
             for p in pools]
    steps = max(1, args.steps // 4)
    (t_e,), wall = _timed(calls, args.warmup, steps, stream)
    nbytes = L * hkv * (2 * d + d // 2 + 2)
    achieved = nbytes / (t_e * 1e-6) / 1e9
    result = {
        "metric": "TQ4 bulk encode-append GB/s (262,143 rows x 4 KV heads, d 256)",
        "value": nbytes / (wall * 1e-6) / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": wall / 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16 -> u4 indices + f16 norm",
        "data": "synthetic",
        "config": {"workload": "tq4_encode_bulk", "rows": L, "num_kv_heads": hkv, "head_dim": d,
                   "page_size": P},
        "us_per_step": {"tq4_encode": t_e, "wall": wall},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "tq4_encode_kernel", "algorithmic_bytes": nbytes}}
    if args.cpu_seconds > 0:
        try:  # the numpy TQ4 oracle's encode on 32,768 rows x 4 heads, scaled
            from oracle import tq4
            c = tq4.codebook(d)[0]
            s_np = signs.cpu().numpy().astype(np.float64)
            xs = x[:32768].cpu().numpy()
            t0 = time.perf_counter()
            for h in range(hkv):
                idx, nrm, _ = tq4.encode(xs[:, h], s_np, c)
                tq4.pack(idx)
            dt = time.perf_counter() - t0
            nb = 32768 * hkv * (2 * d + d // 2 + 2)
            result["cpu_baseline"] = dict(value=nb / dt / 1e9, unit="GB/s", cores=_blas_threads(),
                                          kind="oracle", seconds=dt,
                                          sample="encode + pack of the first 32,768 rows x 4 "
                                                 "heads (numpy, float64), same bytes per vector",
                                          **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        return None


def bench_tq4_decode(args):
    """TQ4 decode attention in the paper's geometry: 24 query heads over 4 KV
    heads, d 256, 262,144 positions in 1,024 shuffled pages (rotated layer
    pools); HBM roofline over the kernel: 2 x 4 x (128 + 2) B per position."""
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS["tq4_decode_256k"]
    P, hkv, hq, d = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim
    L, NP = wl.seq_lens[0], wl.pool_pages
    table_np, (sk, sv) = _tq4_inputs(P, hkv, L, NP, wl.seed, dev)
    table = torch.from_numpy(table_np).to(dev)
    # signs and centroids are inputs of the kernel: any +-1 vectors and any
    # ascending 16 values time the same; these are fixed stand-ins
    cents = torch.linspace(-0.17, 0.17, 16, dtype=torch.float32, device=dev)
    k, v = workloads.gen_kv_device(wl.seed, L, hkv, d, wl.n_outlier, dev)
    lay = jfkv.layout(P, hkv, d, 64, NP)
    cu = torch.tensor([0, L], dtype=torch.int32, device=dev)
    st = torch.tensor([0], dtype=torch.int32, device=dev)
    kp, vp = jfkv.TQ4Pool(lay, device=dev), jfkv.TQ4Pool(lay, device=dev)
    jfkv.jf_tq4_encode_append(kp, k, sk, cents, cu, st, table)
    jfkv.jf_tq4_encode_append(vp, v, sv, cents, cu, st, table)
    pools = [(kp, vp)]
    for _ in range(args.layers - 1):
        a, b = jfkv.TQ4Pool(lay, device=dev), jfkv.TQ4Pool(lay, device=dev)
        for dst, src in ((a, kp), (b, vp)):
            dst.words.copy_(src.words)
            dst.norms.copy_(src.norms)
        pools.append((a, b))
    torch.cuda.synchronize()
    n_total = args.warmup + args.steps
    q = workloads.gen_q_device(wl.seed + 1, n_total, hq, d, dev)
    lens = torch.tensor([L], dtype=torch.int32, device=dev)
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, hq, d, args.max_splits),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((n_total, 1, hq, d), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    calls = [jfkv.bind_tq4_decode(*pools[s % args.layers], sk, sv, cents, q[s:s + 1], table,
                                  lens, 1.0, args.max_splits, ws, out[s], stream)
             for s in range(n_total)]
    gpu_us, wall_us = _back_to_back(lambda s: calls[s](), args.warmup, args.steps, stream)
    assert torch.isfinite(out.float()).all().item(), "non-finite TQ4 decode output"
    bpp = 2 * hkv * (d // 2 + 2)
    nbytes = L * bpp
    achieved = nbytes / (gpu_us * 1e-6) / 1e9
    result = {
        "metric": "TQ4 decode-attn KV positions/s/layer (24 q / 4 KV heads, d 256, 256K ctx)",
        "value": L / (wall_us * 1e-6), "unit": "KV positions/s/layer", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall_us / 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u4 indices -> f16 centroids x f16 -> f32", "data": "synthetic",
        "config": {"workload": "tq4_decode_256k", "positions": L, "num_q_heads": hq,
                   "num_kv_heads": hkv, "head_dim": d, "page_size": P,
                   "max_splits": args.max_splits, "layers_rotated": args.layers},
        "us_per_step": {"kernel": gpu_us, "wall": wall_us},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "tq4_decode_kernel", "algorithmic_bytes": nbytes,
                     "bytes_per_position": bpp}}
    log("tq4_decode_256k: gpu %.2f us/step, %.0f GB/s" % (gpu_us, achieved))
    if args.cpu_seconds > 0:
        try:  # the numpy TQ4 oracle's decode on the first 32,768 positions
            from oracle import tq4
            n = 32768
            c = cents.cpu().numpy()
            s_k, s_v = sk.cpu().numpy().astype(np.float64), sv.cpu().numpy().astype(np.float64)
            kw, kn = tq4.gather(kp.words.cpu().numpy().view(np.uint32), kp.norms.cpu().numpy(),
                                table_np[0], n)
            vw, vn = tq4.gather(vp.words.cpu().numpy().view(np.uint32), vp.norms.cpu().numpy(),
                                table_np[0], n)
            qh = q[0].cpu().numpy()
            t0 = time.perf_counter()
            tq4.decode_attention(qh, kw, kn, vw, vn, s_k, s_v, c, 1.0)
            dt = time.perf_counter() - t0
            result["cpu_baseline"] = dict(value=n / dt, unit="KV positions/s/layer",
                                          cores=_blas_threads(), kind="oracle", seconds=dt,
                                          sample="fp64 decode of all 24 heads over the first "
                                                 "32,768 positions (numpy)", **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def bench_verify(args):
    """verify_256k: the short packed verifier over decode_256k's cache, three
    causal query tokens per request (32 q / 8 KV heads, d 128), rotated layer
    pools.  HBM roofline over the kernel with the cache counted once
    (1,152 B per position): the bytes a verifier that scans the pages once
    per step must move."""
    import numpy as np
    import torch
    import oracle
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS["verify_256k"]
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    L, sq, NP = wl.seq_lens[0], wl.queries, wl.pool_pages
    pp = jfkv.PagePool(NP, P, shuffle_seed=wl.seed)
    s0 = pp.create()
    pp.reserve(s0, L)
    pp.set_length(s0, L)
    table = np.array(pp.export([s0], L // P)[0], np.int32)
    t_table = torch.from_numpy(table).to(dev)
    k, v = workloads.gen_kv_device(wl.seed, L, hkv, d, wl.n_outlier, dev)
    n_total = args.warmup + args.steps
    q = workloads.gen_q_device(wl.seed + 1, n_total * sq, hq, d, dev).view(n_total, 1, sq, hq, d)
    lay = jfkv.layout(P, hkv, d, G, NP)
    pools = [jfkv.KVPool(lay, device=dev) for _ in range(args.layers)]
    i32 = lambda x: torch.tensor(x, dtype=torch.int32, device=dev)  # noqa: E731
    jfkv.jf_kv_quantize_append(pools[0], k, v, i32([0, L]), i32([0]), t_table)
    torch.cuda.synchronize()
    for p in pools[1:]:
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            getattr(p, n).copy_(getattr(pools[0], n))
    lens = i32([L])
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, hq * sq, d, args.max_splits),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((n_total, 1, sq, hq, d), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    calls = [jfkv.bind_verify(pools[s % args.layers], q[s], t_table, lens, 1.0, args.max_splits,
                              ws, out[s], stream) for s in range(n_total)]
    torch.cuda.synchronize()
    gpu_us, wall_us = _back_to_back(lambda s: calls[s](), args.warmup, args.steps, stream)
    assert torch.isfinite(out.float()).all().item(), "non-finite verify output"
    bpp = 2 * hkv * (d // 2 + 4 * d // G)
    nbytes = L * bpp + 2 * sq * hq * d * 2
    achieved = nbytes / (gpu_us * 1e-6) / 1e9
    gqv = hq // hkv * sq
    n_hchunks = -(-gqv // jfkv.decode_head_chunk(d, G, gqv))
    result = {
        "metric": "verify-attn KV positions/s/layer (3 causal query tokens, 32 q / 8 KV heads, "
                  "256K ctx)",
        "value": L / (wall_us * 1e-6), "unit": "KV positions/s/layer", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall_us / 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u4 codes x f16 -> f32", "data": "synthetic",
        "config": {"workload": "verify_256k", "positions": L, "query_tokens": sq,
                   "num_q_heads": hq, "num_kv_heads": hkv, "head_dim": d, "page_size": P,
                   "group_size": G, "max_splits": args.max_splits,
                   "head_chunks_per_kv_head": n_hchunks, "layers_rotated": args.layers},
        "us_per_step": {"kernel": gpu_us, "wall": wall_us},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "decode_kernel (verifier: per-token causal limits)",
                     "algorithmic_bytes": nbytes, "bytes_per_position": bpp}}
    log("verify_256k: gpu %.2f us/step, %.0f GB/s (cache counted once)" % (gpu_us, achieved))
    if args.cpu_seconds > 0:
        try:  # the C oracle's verify (fp64) on the first positions of the cache
            n = min(args.cpu_sample or 32768, L)
            pool = oracle.Pool(oracle.layout(P, hkv, d, G, NP))
            kh, vh = k[:n].cpu().numpy(), v[:n].cpu().numpy()
            oracle.quantize_append(pool, kh, vh, [0, n], [0], table)
            qh = q[0].cpu().numpy()
            m, dt = _repeat(lambda: oracle.verify(pool, qh, table, [n], 1.0), args.cpu_seconds)
            result["cpu_baseline"] = dict(
                value=n * m / dt, unit="KV positions/s/layer", cores=oracle.max_threads(),
                kind="oracle", seconds=dt, steps=m,
                sample="fp64 verification of 3 tokens x 32 heads over the first %d positions "
                       "(one decode per token), %d step(s)" % (n, m), **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def bench_reconstruct(args):
    """reconstruct_grouped: page -> operand reconstruction of one two-KV-head
    group (the paper's grouping) over prefill_chunk's 65,536-position prefix
    (8 KV heads, d 128, group 64), HBM roofline over the kernel (per position
    and head: 2 x (64 + 8) B read, 2 x 256 B written).  Beside it, the
    grouped prefill the paper runs (reconstruct a group, append the chunk's
    fp16 rows, SDPA for the group's query heads, next group) against the fused
    matrix-core prefill on the same chunk: time and incremental peak device
    memory.  And TQ4 reconstruction at the paper's head-group probe geometry
    (4 KV heads, d 256, 196,608 positions, groups of two)."""
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv, workloads
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS["prefill_chunk"]
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    p0, T, grp = wl.seq_lens[0], wl.chunk, 2
    gq = hq // hkv
    lay = jfkv.layout(P, hkv, d, G, wl.pool_pages)
    pp = jfkv.PagePool(wl.pool_pages, P, shuffle_seed=wl.seed)
    s0 = pp.create()
    pp.reserve(s0, p0 + T)
    table_np = np.array(pp.export([s0], (p0 + T) // P)[0], np.int32)
    table = torch.from_numpy(table_np).to(dev)
    k, v = workloads.gen_kv_device(wl.seed, p0 + T, hkv, d, wl.n_outlier, dev)
    q = workloads.gen_q_device(wl.seed + 1, T, hq, d, dev)
    pool = jfkv.KVPool(lay, device=dev)
    i32 = lambda x: torch.tensor(x, dtype=torch.int32, device=dev)  # noqa: E731
    jfkv.jf_kv_quantize_append(pool, k[:p0], v[:p0], i32([0, p0]), i32([0]), table)
    kc, vc = k[p0:].contiguous(), v[p0:].contiguous()
    t1 = table[0].contiguous()
    kr = torch.empty((grp, p0, d), dtype=torch.float16, device=dev)
    vr = torch.empty_like(kr)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def recon(j):
        jfkv.jf_reconstruct_q4(pool, t1, p0, grp * j, grp, kr, vr, stream)

    n_groups = hkv // grp
    steps = max(4, args.steps // 4) * n_groups
    # one group per call, the groups in turn, back to back
    t_rec, wall = _back_to_back(lambda s: recon(s % n_groups), args.warmup, steps, stream)
    per_pos_head = 2 * (d // 2 + 4 * d // G) + 2 * 2 * d
    nbytes = grp * p0 * per_pos_head
    achieved = nbytes / (t_rec * 1e-6) / 1e9
    vectors = 2 * grp * p0
    result = {
        "metric": "page->operand reconstruction, K+V vectors/s (2-KV-head group, 65,536 "
                  "positions, d 128, group 64)",
        "value": vectors / (t_rec * 1e-6), "unit": "vectors/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": wall / 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u4 codes -> f16 (exact rounding)",
        "data": "synthetic",
        "config": {"workload": "reconstruct_grouped", "positions": p0, "group_kv_heads": grp,
                   "num_kv_heads": hkv, "head_dim": d, "page_size": P, "group_size": G,
                   "operand_bytes": 2 * grp * p0 * d * 2},
        "us_per_step": {"reconstruct_group": t_rec, "wall": wall},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "reconstruct_kernel (K and V in one launch)",
                     "algorithmic_bytes": nbytes, "bytes_per_position_and_head": per_pos_head}}
    log("reconstruct group: %.2f us, %.0f GB/s" % (t_rec, achieved))

    # grouped prefill (reconstruct + SDPA per group) against the fused prefill
    mask = torch.ones((T, p0 + T), dtype=torch.bool, device=dev)
    mask[:, p0:] = torch.tril(torch.ones((T, T), dtype=torch.bool, device=dev))
    mask4 = mask[None, None]
    out_g = torch.empty((T, hq, d), dtype=torch.float16, device=dev)
    out_f = torch.empty_like(out_g)

    def grouped():
        from torch.nn.attention import SDPBackend, sdpa_kernel
        for j in range(n_groups):
            recon(j)
            # the group's K/V rows for each of its query heads (the backend
            # takes no grouped heads)
            K = torch.cat([kr, kc[:, grp * j:grp * (j + 1)].transpose(0, 1)], 1)
            V = torch.cat([vr, vc[:, grp * j:grp * (j + 1)].transpose(0, 1)], 1)
            K = K.repeat_interleave(gq, 0)[None]
            V = V.repeat_interleave(gq, 0)[None]
            Q = q[:, grp * j * gq:grp * (j + 1) * gq].transpose(0, 1)[None].contiguous()
            with sdpa_kernel([SDPBackend.EFFICIENT_ATTENTION]):
                O = torch.nn.functional.scaled_dot_product_attention(
                    Q, K, V, attn_mask=mask4, scale=1.0)
            out_g[:, grp * j * gq:grp * (j + 1) * gq] = O[0].transpose(0, 1)

    fused = jfkv.bind_prefill(pool, q, kc, vc, t1, p0, 1.0, out_f, stream)
    cmp = {}
    try:
        for name, fn in (("grouped_reconstruct_sdpa", grouped), ("fused_prefill", fused)):
            fn()
            torch.cuda.synchronize()
            base = torch.cuda.memory_allocated()
            torch.cuda.reset_peak_memory_stats()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = 3
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            cmp[name] = {"ms_per_chunk": e0.elapsed_time(e1) / reps,
                         "incremental_peak_MiB": (torch.cuda.max_memory_allocated() - base) / 2**20}
        diff = (out_g.float() - out_f.float()).abs().max().item()
        cmp["max_abs_diff_between_paths"] = diff
        cmp["sdpa_backend"] = ("torch efficient attention (fp16, [1,1,T,L] boolean mask, K/V "
                                "rows repeated per query head)")
        cmp["chunk"] = T
        cmp["prefix"] = p0
    except Exception as e:  # the consumer is torch's; the comparison is a report
        log("grouped SDPA comparison unavailable: %r" % (e,))
        cmp = {"error": repr(e)[:200]}
    result["grouped_prefill_vs_fused"] = cmp

    # TQ4 reconstruction at the paper's probe geometry
    try:
        L4, P4, h4 = 196608, 256, 4
        NP4 = L4 // P4 + 4
        tnp, (sk, sv) = _tq4_inputs(P4, h4, L4, NP4, 8, dev)
        t4 = torch.from_numpy(tnp[0]).to(dev)
        lay4 = jfkv.layout(P4, h4, 256, 64, NP4)
        cents = torch.linspace(-0.17, 0.17, 16, dtype=torch.float32, device=dev)
        kp, vp = jfkv.TQ4Pool(lay4, device=dev), jfkv.TQ4Pool(lay4, device=dev)
        g4 = torch.Generator(device=dev).manual_seed(8)
        for pl, sg in ((kp, sk), (vp, sv)):
            x = torch.randn((L4, h4, 256), generator=g4, device=dev, dtype=torch.float32).half()
            jfkv.jf_tq4_encode_append(pl, x, sg, cents, i32([0, L4]), i32([0]), t4[None])
            del x
        k4 = torch.empty((2, L4, 256), dtype=torch.float16, device=dev)
        v4 = torch.empty_like(k4)
        t_tq4, _ = _back_to_back(
            lambda s: jfkv.jf_tq4_reconstruct(kp, vp, sk, sv, cents, t4, L4, 2 * (s % 2), 2, k4,
                                              v4, stream), args.warmup, steps, stream)
        b4 = 2 * L4 * 2 * (128 + 2 + 512)
        result["tq4_reconstruct_group"] = {
            "positions": L4, "group_kv_heads": 2, "head_dim": 256, "us": t_tq4,
            "GBs": b4 / (t_tq4 * 1e-6) / 1e9, "frac_of_hbm_peak": b4 / (t_tq4 * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "operand_MiB_group_of_2": 2 * 2 * L4 * 256 * 2 / 2**20,
            "operand_MiB_all_4_heads": 2 * 4 * L4 * 256 * 2 / 2**20}
    except Exception as e:
        log("tq4 reconstruct timing failed: %r" % (e,))
        result["tq4_reconstruct_group"] = None

    if args.cpu_seconds > 0:
        try:  # the oracle's reconstruction of the group over the first positions
            import oracle
            n = min(args.cpu_sample or 8192, p0)
            opool = oracle.Pool(oracle.layout(P, hkv, d, G, wl.pool_pages))
            oracle.quantize_append(opool, k[:n].cpu().numpy(), v[:n].cpu().numpy(), [0, n], [0],
                                   table_np)
            m, dt = _repeat(lambda: oracle.reconstruct(opool, table_np[0], n, 0, grp),
                            args.cpu_seconds)
            result["cpu_baseline"] = dict(value=2 * grp * n * m / dt, unit="vectors/s", cores=1,
                                          kind="oracle", seconds=dt, steps=m,
                                          sample="K and V of a 2-head group over the first %d "
                                                 "positions, %d time(s)" % (n, m), **_host())
        except Exception as e:
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def bench_snapshot(args):
    """snapshot_224k: a 229,376-position (224K) prefix of one request in 16
    layers' pools (8 KV heads, d 128, group 64: 896 pages, 264 MB per layer,
    4.2 GB in all; the paper's snapshot probe uses 16 packed cache layers at
    224K), saved to a file and restored into another request's pages through
    64 MiB of device and 64 MiB of pinned host staging.  The page bytes are
    random (the copies do not look at them).  HBM roofline over the page-pack
    kernel packing one layer into device memory (each byte read and written
    once); save and restore are reported end to end (file on the host's
    temporary directory, removed afterwards)."""
    import shutil
    import tempfile
    import numpy as np
    import torch
    from paper_2609_17475_amd import jfkv
    dev = torch.device("cuda:0")
    P, hkv, d, G, n_layers, L = 256, 8, 128, 64, 16, 229376
    n_pages = L // P
    NP = n_pages + 8
    lay = jfkv.layout(P, hkv, d, G, NP)
    pb = jfkv.kv_page_bytes(lay)
    g = torch.Generator(device=dev).manual_seed(11)
    pools = []
    for _ in range(n_layers):
        pl = jfkv.KVPool(lay, device=dev)
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            t = getattr(pl, n).view(torch.uint8)
            t.copy_(torch.randint(0, 256, t.shape, generator=g, device=dev, dtype=torch.uint8))
        pools.append(pl)
    rng = np.random.default_rng(11)
    table = rng.permutation(NP)[:n_pages].astype(np.int32)
    table2 = rng.permutation(NP)[:n_pages].astype(np.int32)
    t_dev, t2_dev = torch.from_numpy(table).to(dev), torch.from_numpy(table2).to(dev)
    stage = 64 << 20
    sd = torch.empty(stage, dtype=torch.uint8, device=dev)
    sh = torch.empty(stage, dtype=torch.uint8).pin_memory()
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    # the pack kernel, one layer into device memory
    buf = torch.empty(n_pages * pb, dtype=torch.uint8, device=dev)
    steps = max(4, args.steps // 16)
    t_pack, _ = _back_to_back(lambda s: jfkv.jf_kv_pack_pages(pools[s % n_layers], t_dev, 0,
                                                              n_pages, buf, stream),
                              args.warmup, steps, stream)
    nbytes = 2 * n_pages * pb
    achieved = nbytes / (t_pack * 1e-6) / 1e9
    del buf
    tmp = tempfile.mkdtemp(prefix="jfkv_snap_")
    try:
        path = os.path.join(tmp, "prefix.safetensors")
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        t0 = time.perf_counter()
        jfkv.snapshot_save(path, pools, t_dev, table, L, sd, sh, stream)
        t_save = time.perf_counter() - t0
        peak_save = (torch.cuda.max_memory_allocated() - base) / 2**20
        size = os.path.getsize(path)
        pools2 = [jfkv.KVPool(lay, device=dev) for _ in range(n_layers)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        n_pos = jfkv.snapshot_restore(path, pools2, t2_dev, table2, sd, sh, stream)
        t_restore = time.perf_counter() - t0
        assert n_pos == L
        # spot check: a layer's pages, packed from both pools
        a = torch.empty(8 * pb, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for layer in (0, n_layers - 1):
            jfkv.jf_kv_pack_pages(pools[layer], t_dev, n_pages - 8, 8, a, stream)
            jfkv.jf_kv_pack_pages(pools2[layer], t2_dev, n_pages - 8, 8, b, stream)
            torch.cuda.synchronize()
            assert torch.equal(a, b), "restored pages differ"
        cpu = None
        if args.cpu_seconds > 0:  # the definition: page bytes gathered in order, written
            host = [getattr(pools[0], n).view(torch.uint8).cpu().numpy().reshape(NP, -1)
                    for n in ("k_codes", "k_meta", "v_codes", "v_meta")]
            n_s = min(128, n_pages)
            cpath = os.path.join(tmp, "cpu.bin")

            def gather_write():
                with open(cpath, "wb") as f:
                    for i in range(n_s):
                        f.write(np.concatenate([h[table[i]] for h in host]).tobytes())
            m, dt = _repeat(gather_write, args.cpu_seconds)
            cpu = dict(value=n_s * pb * m / dt / 1e9, unit="GB/s", cores=1, kind="oracle",
                       seconds=dt, steps=m,
                       sample="numpy gather of %d pages of one layer (logical order) and "
                              "their write to a file, %d time(s)" % (n_s, m), **_host())
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    result = {
        "metric": "prefix snapshot save GB/s (16 layers x 229,376 positions, 4.2 GB, bounded "
                  "staging)",
        "value": size / t_save / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": 1,
        "warmup": 0, "ms_per_step": t_save * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u8 (packed pages)", "data": "synthetic (random bytes)",
        "config": {"workload": "snapshot_224k", "positions": L, "layers": n_layers,
                   "num_kv_heads": hkv, "head_dim": d, "group_size": G, "page_size": P,
                   "page_bytes": pb, "file_bytes": size, "staging_MiB_device": stage >> 20,
                   "staging_MiB_host": stage >> 20},
        "seconds": {"save": t_save, "restore": t_restore},
        "restore_GBs": size / t_restore / 1e9,
        "incremental_device_peak_MiB_during_save": peak_save,
        "us_per_step": {"pack_one_layer": t_pack},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "page_runs_kernel (pack, one layer into device memory)",
                     "algorithmic_bytes": nbytes}}
    if cpu is not None:
        result["cpu_baseline"] = cpu
    log("snapshot: save %.3f s, restore %.3f s, pack %.1f us (%.0f GB/s)" % (
        t_save, t_restore, t_pack, achieved))
    print(json.dumps(result), flush=True)


WORKLOADS = ("decode_256k", "decode_4k", "decode_32k_loop", "ragged_2req", "prefill_chunk",
             "quantize_bulk", "tq4_encode_bulk", "tq4_decode_256k", "verify_256k",
             "reconstruct_grouped", "snapshot_224k")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--layers", type=int, default=8, help="pools rotated across steps")
    ap.add_argument("--max-splits", type=int, default=64)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the all-core CPU oracle step for at least this long "
                         "(0 = no cpu_baseline)")
    ap.add_argument("--cpu-seconds-1t", type=float, default=4.0,
                    help="repeat the one-core CPU oracle step for at least this long")
    ap.add_argument("--cpu-sample-1t", type=int, default=32768,
                    help="positions of the one-core CPU oracle sample (0 = skip)")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="0 skips the CPU baseline (same as --cpu-seconds 0)")
    ap.add_argument("--positions", type=int, default=0,
                    help="decode_256k: context length in positions, a multiple of the page size "
                         "(0 = the 262,144-position window); other lengths print a "
                         "decode_<positions> line without the counter traffic")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes (counter calibration)")
    ap.add_argument("--read-calibration", type=int, default=0, metavar="BYTES",
                    help="only time one read pass over BYTES bytes (the practical read ceiling)")
    ap.add_argument("--workload", default="decode_256k", choices=WORKLOADS)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.cpu_sample == 0:
        args.cpu_seconds = 0.0
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, max(1, args.steps))
        return
    import torch
    torch.cuda.set_device(torch.device("cuda:0"))
    if args.read_calibration:
        read_calibration(args.read_calibration, args)
        return
    if args.workload in DECODE_STEP_WORKLOADS:
        bench_decode_steps(args.workload, args)
    elif args.workload == "decode_32k_loop":
        bench_decode_loop(args)
    elif args.workload == "prefill_chunk":
        bench_prefill(args)
    elif args.workload == "quantize_bulk":
        bench_quantize_bulk(args)
    elif args.workload == "tq4_encode_bulk":
        bench_tq4_encode(args)
    elif args.workload == "verify_256k":
        bench_verify(args)
    elif args.workload == "reconstruct_grouped":
        bench_reconstruct(args)
    elif args.workload == "snapshot_224k":
        bench_snapshot(args)
    else:
        bench_tq4_decode(args)


if __name__ == "__main__":
    main()
