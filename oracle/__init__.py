"""CPU oracle for attention over a group-wise 4-bit paged KV cache.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the HIP library: the C source here (``jf_oracle.c``) is built with gcc and
implements the same written definitions independently.

Paper: "JustFit: Just-in-Time State Management for Local LLM Serving", KVExec.
  * paged pool + page table: Background, "Compact histories need reusable
    storage" (eq. kvbytes);
  * affine 4-bit codes with per-group scale and offset: the Introduction's
    paragraph on four-bit weights; eight codes per 32-bit word: Appendix A, Table codec;
  * exact softmax attention over dequantized pages, heads independent:
    Sec. 3.1 (eq. groupattention).

All fp16 tensors are passed as numpy ``float16`` arrays (bit patterns cross the
C boundary as uint16).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "jf_oracle.c")
_LIB = os.path.join(_HERE, "libjforacle.so")
_lock = threading.Lock()
_lib = None

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (host only) into ``oracle/libjforacle.so``."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class Layout(ctypes.Structure):
    _fields_ = [("page_size", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int32)]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build(force=False)
            L = ctypes.CDLL(_LIB)
            P = ctypes.c_void_p
            i32 = ctypes.c_int32
            L.jfo_half_to_double.argtypes = [ctypes.c_uint16]
            L.jfo_half_to_double.restype = ctypes.c_double
            L.jfo_float_to_half.argtypes = [ctypes.c_float, ctypes.c_int]
            L.jfo_float_to_half.restype = ctypes.c_uint16
            L.jfo_double_to_half.argtypes = [ctypes.c_double, ctypes.c_int]
            L.jfo_double_to_half.restype = ctypes.c_uint16
            L.jfo_reconstruct.argtypes = [P, P, P, ctypes.c_int, P, i32, i32, i32, i32, P]
            L.jfo_reconstruct.restype = ctypes.c_int
            L.jfo_quantize_group.argtypes = [P, i32, P, P, P]
            L.jfo_quantize_group.restype = None
            L.jfo_quantize_groups.argtypes = [P, ctypes.c_int64, i32, P, P, P]
            L.jfo_quantize_groups.restype = None
            L.jfo_codes_bytes.argtypes = [P]
            L.jfo_codes_bytes.restype = ctypes.c_size_t
            L.jfo_meta_elems.argtypes = [P]
            L.jfo_meta_elems.restype = ctypes.c_size_t
            L.jfo_quantize_append.argtypes = [P, P, P, P, P, P, P, P, P, P, i32, i32]
            L.jfo_quantize_append.restype = ctypes.c_int
            L.jfo_dequant_vector.argtypes = [P, P, P, ctypes.c_int, i32, i32, i32, P]
            L.jfo_dequant_vector.restype = None
            L.jfo_decode.argtypes = [P, P, P, P, P, P, i32, i32, P, i32, P,
                                     ctypes.c_double, P]
            L.jfo_decode.restype = ctypes.c_int
            L.jfo_prefill.argtypes = [P, P, P, P, P, P, P, P, i32, i32, P, i32, i32,
                                      ctypes.c_double, ctypes.c_int, P, i32, P]
            L.jfo_prefill.restype = ctypes.c_int
            L.jfo_max_threads.argtypes = []
            L.jfo_max_threads.restype = ctypes.c_int
            L.jfo_set_threads.argtypes = [ctypes.c_int]
            L.jfo_set_threads.restype = None
            _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _u16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    assert a.dtype in (np.float16, np.uint16), a.dtype
    return a.view(np.uint16)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def layout(page_size, num_kv_heads, head_dim, group_size, num_pages) -> Layout:
    return Layout(page_size, num_kv_heads, head_dim, group_size, num_pages)


# ---------------------------------------------------------------- fp16 helpers
def half_to_double(bits: int) -> float:
    return lib().jfo_half_to_double(int(bits))


def float_to_half(f: float, mode: int) -> int:
    """mode 0 = nearest-even, 1 = toward -inf, 2 = toward +inf; returns bits."""
    return lib().jfo_float_to_half(float(np.float32(f)), int(mode))


def double_to_half(x: float, mode: int = 0) -> int:
    """The same rounding of a binary64 value; returns bits."""
    return lib().jfo_double_to_half(float(x), int(mode))


# ---------------------------------------------------------------- quantizer
def quantize_group(x: np.ndarray):
    """x: fp16[G] -> (codes uint8[G], scale fp16, bias fp16)."""
    x = _u16(x)
    G = x.shape[0]
    codes = np.zeros(G, np.uint8)
    s = np.zeros(1, np.uint16)
    b = np.zeros(1, np.uint16)
    lib().jfo_quantize_group(_ptr(x), G, _ptr(codes), _ptr(s), _ptr(b))
    return codes, s.view(np.float16)[0], b.view(np.float16)[0]


def quantize_groups(x: np.ndarray):
    """x: fp16 [n][G] -> (codes uint8 [n][G], scales fp16 [n], biases fp16 [n])."""
    x = _u16(x)
    n, G = x.shape
    codes = np.zeros((n, G), np.uint8)
    s = np.zeros(n, np.uint16)
    b = np.zeros(n, np.uint16)
    lib().jfo_quantize_groups(_ptr(x), n, G, _ptr(codes), _ptr(s), _ptr(b))
    return codes, s.view(np.float16), b.view(np.float16)


class Pool:
    """Host copy of one layer's K and V pools in the library's byte layout."""

    def __init__(self, lay: Layout, fill: int = 0xA5):
        self.layout = lay
        nb = lib().jfo_codes_bytes(ctypes.byref(lay))
        nm = lib().jfo_meta_elems(ctypes.byref(lay))
        self.k_codes = np.full(nb, fill, np.uint8)
        self.v_codes = np.full(nb, fill, np.uint8)
        self.k_meta = np.full(nm, fill | (fill << 8), np.uint16)
        self.v_meta = np.full(nm, fill | (fill << 8), np.uint16)

    def copy(self) -> "Pool":
        p = Pool.__new__(Pool)
        p.layout = self.layout
        for n in ("k_codes", "v_codes", "k_meta", "v_meta"):
            setattr(p, n, getattr(self, n).copy())
        return p

    def args(self):
        return (_ptr(self.k_codes), _ptr(self.k_meta), _ptr(self.v_codes), _ptr(self.v_meta))


def quantize_append(pool: Pool, k_new, v_new, cu_tok, start_pos, block_tables):
    k = _u16(k_new)
    v = _u16(v_new)
    cu = _i32(cu_tok)
    sp = _i32(start_pos)
    bt = _i32(block_tables)
    B = sp.shape[0]
    rc = lib().jfo_quantize_append(ctypes.byref(pool.layout), *pool.args(), _ptr(k), _ptr(v),
                                   _ptr(cu), _ptr(sp), _ptr(bt), B, bt.shape[-1])
    if rc != 0:
        raise ValueError("oracle quantize_append: invalid page reference")


def dequant_vector(pool: Pool, is_v: bool, page: int, kv: int, slot: int) -> np.ndarray:
    out = np.zeros(pool.layout.head_dim, np.float64)
    codes, meta = (pool.v_codes, pool.v_meta) if is_v else (pool.k_codes, pool.k_meta)
    lib().jfo_dequant_vector(ctypes.byref(pool.layout), _ptr(codes), _ptr(meta), int(is_v),
                             page, kv, slot, _ptr(out))
    return out


def decode(pool: Pool, q, block_tables, seq_lens, alpha: float) -> np.ndarray:
    """q fp16 [B][Hq][d] -> fp64 [B][Hq][d]."""
    qq = _u16(q)
    B, Hq, d = qq.shape
    bt = _i32(block_tables)
    sl = _i32(seq_lens)
    out = np.zeros((B, Hq, d), np.float64)
    rc = lib().jfo_decode(ctypes.byref(pool.layout), *pool.args(), _ptr(qq), B, Hq, _ptr(bt),
                          bt.shape[-1], _ptr(sl), float(alpha), _ptr(out))
    if rc != 0:
        raise ValueError("oracle decode: invalid arguments")
    return out


def reconstruct(pool: Pool, block_table, n_pos: int, kv0: int, g: int):
    """Page -> operand reconstruction of one head group (Background, eq.
    layerbytes; Sec. 3.1, eq. groupattention): (K, V) fp16 [g][n_pos][d], the
    dequantized vectors of KV heads kv0 .. kv0+g-1 at logical positions
    0 .. n_pos-1 of one request (block_table [max_pages]), each element the
    exact value rounded once to fp16 (nearest even); pages outside the pool
    give zeros."""
    bt = _i32(block_table).reshape(-1)
    d = pool.layout.head_dim
    res = []
    for is_v, (codes, meta) in enumerate(((pool.k_codes, pool.k_meta),
                                          (pool.v_codes, pool.v_meta))):
        out = np.zeros((g, n_pos, d), np.uint16)
        rc = lib().jfo_reconstruct(ctypes.byref(pool.layout), _ptr(codes), _ptr(meta), is_v,
                                   _ptr(bt), bt.shape[0], int(n_pos), int(kv0), int(g),
                                   _ptr(out))
        if rc != 0:
            raise ValueError("oracle reconstruct: invalid arguments")
        res.append(out.view(np.float16))
    return res[0], res[1]


def verify(pool: Pool, q, block_tables, seq_lens, alpha: float) -> np.ndarray:
    """Short packed verification (Sec. 3.1, speculative verification; Appendix
    A, causal string masks over 2 to 4 queries).  q fp16 [B][Sq][Hq][d] ->
    fp64 [B][Sq][Hq][d].  The last Sq cached positions of request b are its
    query tokens; token k attends to positions 0 .. L_b - Sq + k, i.e. the
    plain decode definition over the first L_b - Sq + k + 1 positions (an
    all-zero row when that count is <= 0)."""
    q = np.asarray(q)
    B, Sq = q.shape[:2]
    lens = [int(x) for x in np.asarray(seq_lens).reshape(-1)]
    bt = _i32(block_tables)
    out = np.zeros(q.shape, np.float64)
    for k in range(Sq):
        vis = [L - Sq + 1 + k for L in lens]
        live = [b for b in range(B) if vis[b] > 0]
        if live:
            out[live, k] = decode(pool, q[live, k], bt[live], [vis[b] for b in live], alpha)
    return out


def prefill(pool: Pool, q, k_chunk, v_chunk, block_table, prefix_len: int, alpha: float,
            chunk_quantized: bool = False, rows=None) -> np.ndarray:
    """q fp16 [T][Hq][d], k/v fp16 [T][Hkv][d] -> fp64 [len(rows) or T][Hq][d]."""
    qq = _u16(q)
    kk = _u16(k_chunk)
    vv = _u16(v_chunk)
    T, Hq, d = qq.shape
    bt = _i32(block_table)
    if rows is None:
        r_arr, n_rows, r_ptr = None, T, None
    else:
        r_arr = _i32(rows)
        n_rows = r_arr.shape[0]
        r_ptr = _ptr(r_arr)
    out = np.zeros((n_rows, Hq, d), np.float64)
    rc = lib().jfo_prefill(ctypes.byref(pool.layout), *pool.args(), _ptr(qq), _ptr(kk), _ptr(vv),
                           T, Hq, _ptr(bt), bt.shape[-1], int(prefix_len), float(alpha),
                           int(bool(chunk_quantized)), r_ptr, n_rows, _ptr(out))
    if rc != 0:
        raise ValueError("oracle prefill: invalid arguments")
    return out


def max_threads() -> int:
    return lib().jfo_max_threads()


def set_threads(n: int):
    """Threads of the oracle's OpenMP loops (for timing it on 1 or all cores)."""
    lib().jfo_set_threads(int(n))
