#!/usr/bin/env python
"""Decode attention over a 4-bit paged KV cache at a 262,144-position window.

One step = one decode step of one layer for one request: host page
reservation, quantize-append of the step's new K/V row into its page (position
262,143), then split-K decode attention of 32 query heads (8 KV heads, d=128,
GQA 4:1) over all 262,144 positions through a 1,024-entry shuffled page table,
with the log-sum-exp combine.  Inputs (cache, page table, the steps' new rows
and queries) are resident in HBM before timing.  Consecutive steps use
different layers' pools (--layers, default 8 x 302 MB), so a step never finds
the previous step's cache lines in the 256 MB last-level cache, as in a model
whose layers each own a pool.

Prints one JSON line: KV positions/s/layer (value), HBM GB/s of the decode
kernels against the 8 TB/s peak (roofline), and the CPU oracle timed on a
bounded sample (cpu_baseline).
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
BYTES_PER_POSITION = 1152  # 2 * Hkv * (d/2 + 4*d/G) at Hkv=8, d=128, G=64


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(k16, v16, q16, table, n_sample: int, min_seconds: float):
    """The CPU oracle on a bounded sample of the same workload: one decode step
    (append one row, attend) over the first n_sample positions of the window
    (by default all of it), all 32 query heads.  Building the sample's cache
    is untimed setup."""
    import oracle
    P, hkv, d, G = 256, 8, 128, 64
    NP = int(table.max()) + 1
    lay = oracle.layout(P, hkv, d, G, NP)
    pool = oracle.Pool(lay)
    n_cached = n_sample - 1
    oracle.quantize_append(pool, k16[:n_cached], v16[:n_cached], [0, n_cached], [0], table[None])
    steps = 0
    t0 = time.perf_counter()
    while True:  # repeat the step (same row, same position) until min_seconds have passed
        oracle.quantize_append(pool, k16[n_cached:n_sample], v16[n_cached:n_sample], [0, 1],
                               [n_cached], table[None])
        oracle.decode(pool, q16[None], table[None], [n_sample], 1.0)
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    threads = min(oracle.max_threads(), hkv)  # the decode loop has one task per KV head
    return {"value": n_sample * steps / dt, "unit": "KV positions/s/layer", "cores": threads,
            "kind": "oracle", "seconds": dt, "steps": steps, "host_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": _cpu_model(),
            "sample": "decode steps (quantize-append 1 row + fp64 attention of 32 q heads) "
                      "over the first %d positions of the 262,144-position window, repeated "
                      "for at least %.0f s, as positions/s" % (n_sample, min_seconds)}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


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


MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 / bf16 matrix peak


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


def bench_prefill(args):
    """Chunked prefill: a 2,048-row chunk (32 q / 8 KV heads, d 128) attends
    to a 65,536-position 4-bit prefix in 256 shuffled pages plus itself
    (causal), then the chunk is appended as 8 pages.  MFMA roofline over the
    attention kernel: FLOP = 4 d Hq sum_i (p0 + i + 1)."""
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
    table = torch.tensor(pp.export([s], (p0 + T) // P)[0], dtype=torch.int32, device=dev)
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
    print(json.dumps({
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
                     "kernel": "prefill_kernel", "algorithmic_flop": flop},
        "cpu_baseline": None}), flush=True)


def bench_quantize_bulk(args):
    """Bulk quantize-append of 262,143 rows x 8 KV heads (the cache of the
    256K decode workload) into 1,024 shuffled pages; HBM roofline over the
    kernel: 2 x 256 B read and 2 x (64 + 8) B written per (row, KV head)."""
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
    table = torch.tensor(pp.export([s], (L + 1) // P)[0], dtype=torch.int32, device=dev)
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
    print(json.dumps({
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
                     "kernel": "quantize_rows_kernel", "algorithmic_bytes": nbytes},
        "cpu_baseline": None}), flush=True)


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
    rng = np.random.default_rng(4)
    table = torch.tensor(rng.permutation(NP)[:L // P + 1][None].astype(np.int32), device=dev)
    g = torch.Generator(device=dev).manual_seed(4)
    x = torch.randn((L, hkv, d), generator=g, device=dev, dtype=torch.float32).half()
    # signs and centroids are inputs of the kernel: any +-1 vector and any
    # ascending 16 values time the same; these are fixed stand-ins
    signs = torch.tensor(np.where(rng.random(d) < 0.5, -1.0, 1.0), dtype=torch.float32,
                         device=dev)
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
    print(json.dumps({
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
                     "kernel": "tq4_encode_kernel", "algorithmic_bytes": nbytes},
        "cpu_baseline": None}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--layers", type=int, default=8, help="pools rotated across steps")
    ap.add_argument("--max-splits", type=int, default=64)
    ap.add_argument("--two-calls", action="store_true",
                    help="decode_256k: append and attend as two launches "
                         "(jf_kv_quantize_append + jf_decode_attn_q4) instead of jf_decode_step_q4")
    ap.add_argument("--cpu-sample", type=int, default=262144,
                    help="positions in the CPU oracle sample (0 = skip)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="repeat the CPU oracle step for at least this long")
    ap.add_argument("--positions", type=int, default=0,
                    help="decode: context length in positions, a multiple of the page size "
                         "(0 = the 262,144-position window of decode_256k); other lengths "
                         "print a decode_<positions> line without the counter traffic")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes (counter calibration)")
    ap.add_argument("--workload", default="decode_256k",
                    choices=["decode_256k", "prefill_chunk", "quantize_bulk", "tq4_encode_bulk"],
                    help="decode_256k (the headline line); prefill_chunk and quantize_bulk "
                         "print their own lines")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, max(1, args.steps))
        return
    if args.workload == "prefill_chunk":
        bench_prefill(args)
        return
    if args.workload == "quantize_bulk":
        bench_quantize_bulk(args)
        return
    if args.workload == "tq4_encode_bulk":
        bench_tq4_encode(args)
        return

    import numpy as np
    import torch

    from paper_2609_17475_amd import jfkv, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = workloads.WORKLOADS["decode_256k"]
    P, hkv, hq, d, G = wl.page_size, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.group_size
    L = args.positions or wl.seq_lens[0]
    if L < P or L % P:
        print("--positions must be a positive multiple of the page size (%d)" % P, file=sys.stderr)
        sys.exit(2)
    window = L == wl.seq_lens[0]
    n_cached = L - 1
    n_steps_total = args.warmup + args.steps
    NP = L // P + (wl.pool_pages - wl.seq_lens[0] // P)  # the window's pages + spare pages
    lay = jfkv.layout(P, hkv, d, G, NP)

    # ---- page table: one request holding the full window (shuffled pages)
    pp = jfkv.PagePool(NP, P, shuffle_seed=wl.seed)
    seq = pp.create()
    pp.reserve(seq, L)
    pp.set_length(seq, n_cached)
    table_rows, _ = pp.export([seq], L // P)
    table = np.array(table_rows, np.int32)
    t_table = torch.from_numpy(table).to(dev)

    # ---- inputs (seeded, drawn on the device)
    t0 = time.perf_counter()
    k, v = workloads.gen_kv_device(wl.seed, n_cached + n_steps_total, hkv, d, wl.n_outlier, dev)
    q = workloads.gen_q_device(wl.seed + 1, n_steps_total, hq, d, dev)
    log("inputs drawn in %.1fs" % (time.perf_counter() - t0))

    # ---- layer 0 cache built by the library's quantize-append, copied to the others
    pools = [jfkv.KVPool(lay, device=dev) for _ in range(args.layers)]
    t0 = time.perf_counter()
    jfkv.jf_kv_quantize_append(pools[0], k[:n_cached], v[:n_cached],
                               torch.tensor([0, n_cached], dtype=torch.int32, device=dev),
                               torch.tensor([0], dtype=torch.int32, device=dev), t_table)
    torch.cuda.synchronize()
    log("bulk quantize of %d rows: %.1f ms (incl. launch)" % (n_cached, 1e3 * (time.perf_counter() - t0)))
    for p in pools[1:]:
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            getattr(p, n).copy_(getattr(pools[0], n))
    torch.cuda.synchronize()

    # ---- per-step bound calls: append row n_cached + s at position n_cached, attend L
    cu = torch.tensor([0, 1], dtype=torch.int32, device=dev)
    start = torch.tensor([n_cached], dtype=torch.int32, device=dev)
    lens = torch.tensor([L], dtype=torch.int32, device=dev)
    ws = torch.zeros(jfkv.jf_decode_workspace_bytes(1, hq, d, args.max_splits), dtype=torch.uint8,
                     device=dev)
    out = torch.empty((n_steps_total, 1, hq, d), dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    appends, decodes = [], []
    for s in range(n_steps_total):
        pool = pools[s % args.layers]
        row = slice(n_cached + s, n_cached + s + 1)
        qs = q[s:s + 1].view(1, hq, d)
        if args.two_calls:
            appends.append(jfkv.bind_quantize_append(pool, k[row], v[row], cu, start, t_table,
                                                     stream))
            decodes.append(jfkv.bind_decode(pool, qs, t_table, lens, 1.0, args.max_splits, ws,
                                            out[s], stream))
        else:  # one launch: the row is appended at position L - 1, then attended to
            appends.append(lambda: None)
            decodes.append(jfkv.bind_decode_step(pool, k[row], v[row], qs, t_table, lens, 1.0,
                                                 args.max_splits, ws, out[s], stream))

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(n_steps_total)]

    def step(s, timed_events=False):
        pp.reserve(seq, L)  # host page reservation (already satisfied at the window)
        if timed_events:
            if args.two_calls:
                ev[s][0].record(stream)
                appends[s]()
            ev[s][1].record(stream)
            decodes[s]()
            ev[s][2].record(stream)
        else:
            appends[s]()
            decodes[s]()

    for s in range(args.warmup):
        step(s)
    torch.cuda.synchronize()
    # the timed steps, back to back between two synchronizations; one HIP
    # event pair on the kernels' stream brackets them (the kernel's average
    # duration for the roofline: the GPU time per step, launch gaps included)
    ev_all = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    t0 = time.perf_counter()
    ev_all[0].record(stream)
    for s in range(args.warmup, n_steps_total):
        step(s)
    ev_all[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms_per_step = ev_all[0].elapsed_time(ev_all[1]) / args.steps
    if args.two_calls:
        # the same steps again with events around each kernel, to split the
        # step between the append and the decode kernels
        for s in range(args.warmup, n_steps_total):
            step(s, timed_events=True)
        torch.cuda.synchronize()

    timed = range(args.warmup, n_steps_total)
    if args.two_calls:
        t_app = [ev[s][0].elapsed_time(ev[s][1]) for s in timed]
        t_dec = [ev[s][1].elapsed_time(ev[s][2]) for s in timed]
    else:  # one kernel per step: its average is the bracketed GPU time per step
        t_app = [0.0]
        t_dec = [gpu_ms_per_step]
    ms_per_step = 1e3 * wall / args.steps
    dec_ms = float(np.mean(t_dec))
    # the step kernel's algorithmic bytes: the window's codes and (scale,
    # bias) words, plus, when fused, the new row's fp16 K/V read and its
    # codes and meta written
    dec_bytes = L * BYTES_PER_POSITION + (0 if args.two_calls else 2 * hkv * d * 2 + BYTES_PER_POSITION)
    achieved = dec_bytes / (dec_ms * 1e-3) / 1e9
    log("append %.2f us  decode %.2f us  gpu/step %.2f us  wall/step %.2f us" % (
        1e3 * np.mean(t_app), 1e3 * dec_ms, 1e3 * gpu_ms_per_step, 1e3 * ms_per_step))

    # sanity: the timed steps produced finite outputs
    assert torch.isfinite(out.float()).all().item(), "non-finite decode output"

    result = {
        "metric": METRIC,
        "value": L / (ms_per_step * 1e-3),
        "unit": "KV positions/s/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u4 codes x f16 -> f32",
        "data": "synthetic",
        "config": {"workload": "decode_256k" if window else "decode_%d" % L, "positions": L, "batch": 1, "num_q_heads": hq,
                   "num_kv_heads": hkv, "head_dim": d, "page_size": P, "group_size": G,
                   "pages": L // P, "max_splits": args.max_splits,
                   "splits_used": min(args.max_splits, L // P, -(-torch.cuda.get_device_properties(
                       0).multi_processor_count // hkv)),
                   "layers_rotated": args.layers,
                   "step": ("jf_kv_quantize_append + jf_decode_attn_q4" if args.two_calls
                            else "jf_decode_step_q4 (append + attend, one kernel)")},
        "hbm_GBs": achieved,
        "hbm_pct_of_peak": 100.0 * achieved / HBM_PEAK_GBS,
        "us_per_step": {"append": (1e3 * float(np.mean(t_app)) if args.two_calls else None),
                        "decode" if args.two_calls else "step_kernel": 1e3 * dec_ms,
                        "gpu": 1e3 * gpu_ms_per_step,
                        "wall": 1e3 * ms_per_step},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic() if window else None,
                     "kernel": ("decode_kernel (split-K partials and the in-kernel combine)"
                                if args.two_calls else
                                "decode_kernel, fused step (row append, split-K partials, "
                                "in-kernel combine)"),
                     "algorithmic_bytes": dec_bytes},
    }
    if args.cpu_sample > 0:
        try:
            n_s = min(args.cpu_sample, L)
            rows = n_s
            kh = k[:rows].cpu().numpy()
            vh = v[:rows].cpu().numpy()
            qh = q[args.warmup].cpu().numpy()
            result["cpu_baseline"] = cpu_baseline(kh, vh, qh, table[0], n_s, args.cpu_seconds)
        except Exception as e:  # the baseline is a report, not the product
            log("cpu baseline failed: %r" % (e,))
            result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
