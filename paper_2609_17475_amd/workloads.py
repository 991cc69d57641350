"""Seeded synthetic inputs shaped like the paper's attention workloads.

This module only draws inputs: it holds none of the quantizer's or the
attention's arithmetic, so the HIP path and the CPU oracle can both consume
its tensors without sharing any of the method's code.

The paper measures a 27B model's real activations on repetitive-word capacity
prompts (Appendix A, controlled capacity protocol); neither the model nor its
data exist here, so Gaussian K/V with a few large "outlier" channels stand in
for them.  Shapes follow the paper's page geometry (256-token pages, Background
"Compact histories ..."), and the five workloads below:

  decode_4k        4 q heads / 1 KV head, d=128, 4,096 cached positions in 16
                   shuffled pages of a 32-page pool, 4 outlier channels x8,
                   one appended row per step.
  decode_32k_loop  32/8 heads, d=128, 32,768 cached positions + 6,144 decode
                   steps (append + attend), 160-page shuffled pool, 2%
                   outlier channels.
  decode_256k      32/8 heads, d=128, 262,144 positions in 1,024 shuffled
                   pages; 64 split-K partials at most.
  ragged_2req      32/8 heads, requests of 196,608 and 131,072 positions whose
                   first 32,768 positions share physical pages.
  prefill_chunk    2,048-row chunk over a 65,536-position prefix (256 shuffled
                   pages), 32/8 heads, then appended as 8 new pages.
  tq4_decode_256k  the paper's geometry and codec: 24/4 heads, d=256, 262,144
                   positions in 1,024 shuffled pages of TQ4 vectors.
  verify_256k      decode_256k's cache with 3 query tokens per request (the
                   paper's verification width: two proposed tokens and a
                   bonus position), causal among them.

Recipe (fixed draw order, numpy PCG64 ``default_rng(seed)``):
  1. K then V: float32 N(0,1), shape [n_rows][Hkv][d];
  2. outlier channels: for K then for V, for each KV head, ``n_out`` distinct
     channels drawn without replacement; those channels are multiplied by 8
     for every row; then K and V are rounded to fp16;
  3. q: float32 N(0,1) * (1/sqrt(d)) rounded to fp16 (pre-scaled: the
     workloads call attention with softmax_scale = 1);
  4. page permutation of the pool.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

PAGE_SIZE = 256
GROUP_SIZE = 64


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_lens: tuple          # cached positions per request before the step
    pool_pages: int
    n_outlier: int           # outlier channels per (K|V, KV head)
    seed: int
    shared_prefix: int = 0   # positions whose pages are shared by all requests
    chunk: int = 0           # prefill chunk rows (prefill workloads)
    steps: int = 0           # sequential decode steps (loop workloads)
    max_splits: int = 64
    queries: int = 1         # query tokens per request (the short verifier: 2..4)
    page_size: int = PAGE_SIZE
    group_size: int = GROUP_SIZE


WORKLOADS = {
    "decode_4k": Workload("decode_4k", 4, 1, 128, (4096,), 32, 4, seed=1),
    "decode_32k_loop": Workload("decode_32k_loop", 32, 8, 128, (32768,), 160, 3, seed=2,
                                steps=6144),
    "decode_256k": Workload("decode_256k", 32, 8, 128, (262144,), 1024 + 8, 3, seed=3),
    "ragged_2req": Workload("ragged_2req", 32, 8, 128, (196608, 131072), 1152 + 16, 3,
                            seed=4, shared_prefix=32768),
    "prefill_chunk": Workload("prefill_chunk", 32, 8, 128, (65536,), 256 + 16, 3, seed=5,
                              chunk=2048),
    # the paper's own geometry and format (24 query heads over 4 KV heads,
    # d = 256, TQ4 pages) at its full native window
    "tq4_decode_256k": Workload("tq4_decode_256k", 24, 4, 256, (262144,), 1024 + 8, 5, seed=6),
    "verify_256k": Workload("verify_256k", 32, 8, 128, (262144,), 1024 + 8, 3, seed=7, queries=3),
}


def outlier_count(head_dim: int, fraction: float = 0.02) -> int:
    """'2% outlier channels' read as round(0.02 * d) channels (3 at d=128)."""
    return int(round(fraction * head_dim))


def to_f16(x: np.ndarray) -> np.ndarray:
    """Round float32 to fp16 (IEEE round-to-nearest-even), vectorized."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.float16).numpy()


def _kv(rng, n_rows, hkv, d, n_out):
    k = rng.standard_normal((n_rows, hkv, d), dtype=np.float32)
    v = rng.standard_normal((n_rows, hkv, d), dtype=np.float32)
    for x in (k, v):
        for h in range(hkv):
            ch = rng.choice(d, size=n_out, replace=False) if n_out else []
            for c in ch:
                x[:, h, c] *= 8.0
    return to_f16(k), to_f16(v)


def gen_kv(seed: int, n_rows: int, hkv: int, d: int, n_out: int):
    """K, V fp16 [n_rows][hkv][d] (steps 1-2 of the recipe)."""
    rng = np.random.default_rng(seed)
    return _kv(rng, n_rows, hkv, d, n_out)


def gen_all(seed: int, n_rows: int, hkv: int, d: int, n_out: int, n_q_rows: int, hq: int,
            n_pages: int):
    """Full draw in recipe order: K, V, q fp16 [n_q_rows][hq][d], page permutation."""
    rng = np.random.default_rng(seed)
    k, v = _kv(rng, n_rows, hkv, d, n_out)
    q = to_f16(rng.standard_normal((n_q_rows, hq, d), dtype=np.float32)
               * np.float32(1.0 / math.sqrt(d)))
    perm = rng.permutation(n_pages).astype(np.int32)
    return k, v, q, perm


def needle_queries(k16: np.ndarray, hq: int, seed: int, gap: float = 12.0,
                   valid_len: int | None = None):
    """Needle variant (parity only): for each q head h (KV head h // (hq/hkv))
    pick a position t* and point q_h along K16[t*, kv] so that t*'s logit
    exceeds the typical maximum of the others by about ``gap``.

    Returns (q fp16 [hq][d], t_star int [hq])."""
    n, hkv, d = k16.shape
    n = n if valid_len is None else valid_len
    rng = np.random.default_rng(seed)
    gq = hq // hkv
    q = np.zeros((hq, d), np.float32)
    t_star = rng.integers(0, n, size=hq)
    for h in range(hq):
        kv = h // gq
        kstar = k16[t_star[h], kv].astype(np.float64)
        norm = float(np.linalg.norm(kstar))
        # others project onto the unit vector as ~N(0,1); their max over n
        # positions is about sqrt(2 ln n)
        typical_max = math.sqrt(2.0 * math.log(max(n, 2)))
        gamma = gap / max(norm - typical_max, 1.0)
        q[h] = gamma * kstar / norm
    return q.astype(np.float16), t_star


def page_order(seed: int, n_pages_pool: int) -> np.ndarray:
    """A seeded permutation of a pool's page IDs."""
    return np.random.default_rng(seed).permutation(n_pages_pool).astype(np.int32)


def gen_kv_device(seed: int, n_rows: int, hkv: int, d: int, n_out: int, device="cuda"):
    """Device-side draw for the large workloads (same recipe, torch's seeded
    generator on `device` instead of numpy PCG64): K, V fp16 [n_rows][hkv][d].
    Outlier channels: for K then V, for each KV head, the first n_out entries of
    a seeded permutation of the channels, scaled by 8."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = []
    for _ in range(2):
        x = torch.randn((n_rows, hkv, d), generator=g, device=device, dtype=torch.float32)
        out.append(x)
    for x in out:
        for h in range(hkv):
            ch = torch.randperm(d, generator=g, device=device)[:n_out]
            x[:, h, ch] *= 8.0
    return out[0].to(torch.float16), out[1].to(torch.float16)


def gen_q_device(seed: int, n_rows: int, hq: int, d: int, device="cuda"):
    """Queries fp16 [n_rows][hq][d] ~ N(0,1)/sqrt(d), torch's seeded generator."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    x = torch.randn((n_rows, hq, d), generator=g, device=device, dtype=torch.float32)
    return (x * (1.0 / math.sqrt(d))).to(torch.float16)
