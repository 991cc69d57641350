"""ctypes binding of libjfkv.so (include/jfkv.h).

Argument marshalling only: every step of quantize-append, decode and prefill
runs in the library's HIP kernels.  Device buffers are torch tensors on the
GPU; the stream is torch's current stream unless one is given.  Errors raise
``JfError`` with the library's message.  If the shared library is missing the
import of this module fails loudly: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("JFKV_LIB") or os.path.join(HERE, "libjfkv.so")  # JFKV_LIB: another build

JF_OK, JF_ERR_INVALID, JF_ERR_NO_PAGES, JF_ERR_DEVICE, JF_ERR_UNSUPPORTED, JF_ERR_STATE, JF_ERR_IO = \
    range(7)
STATUS_NAMES = {0: "JF_OK", 1: "JF_ERR_INVALID", 2: "JF_ERR_NO_PAGES", 3: "JF_ERR_DEVICE",
                4: "JF_ERR_UNSUPPORTED", 5: "JF_ERR_STATE", 6: "JF_ERR_IO"}

# every symbol include/jfkv.h declares
EXPORTS = [
    "jf_last_error", "jf_version", "jf_kv_pool_bytes",
    "jf_page_table_pool_create", "jf_page_table_pool_destroy", "jf_page_table_create",
    "jf_page_table_fork", "jf_page_table_assign", "jf_page_table_reserve",
    "jf_page_table_set_length", "jf_page_table_release", "jf_page_table_export",
    "jf_page_table_stats", "jf_page_table_info",
    "jf_kv_quantize_append", "jf_decode_workspace_bytes", "jf_decode_attn_q4",
    "jf_verify_attn_q4", "jf_decode_step_q4", "jf_decode_step_q4_static", "jf_prefill_attn_q4",
    "jf_reconstruct_q4", "jf_tq4_pool_bytes", "jf_tq4_encode_append", "jf_tq4_decode_attn",
    "jf_tq4_reconstruct", "jf_kv_page_bytes", "jf_kv_pack_pages", "jf_kv_unpack_pages",
    "jf_snapshot_save", "jf_snapshot_restore", "jf_calib_read_stream",
]


class JfError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, str(status)), message))
        self.status = status


class Layout(ctypes.Structure):
    _fields_ = [("page_size", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int32)]


class PoolPtrs(ctypes.Structure):
    _fields_ = [("k_codes", ctypes.c_void_p), ("k_meta", ctypes.c_void_p),
                ("v_codes", ctypes.c_void_p), ("v_meta", ctypes.c_void_p)]


def _load():
    # Load torch first: its wheel ships its own HIP runtime (same SONAME as
    # /opt/rocm's), and the library must bind to that one, which owns the
    # streams and allocations it receives.  Loading libjfkv.so first would
    # map a second runtime version into the process.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError("libjfkv.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    P, i32, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    pi32 = ctypes.POINTER(ctypes.c_int32)
    st = ctypes.c_int
    sig = {
        "jf_last_error": (ctypes.c_char_p, []),
        "jf_version": (ctypes.c_char_p, []),
        "jf_kv_pool_bytes": (st, [P, ctypes.POINTER(sz), ctypes.POINTER(sz)]),
        "jf_page_table_pool_create": (st, [i32, i32, u64, ctypes.POINTER(P)]),
        "jf_page_table_pool_destroy": (st, [P]),
        "jf_page_table_create": (st, [P, pi32]),
        "jf_page_table_fork": (st, [P, i32, i32, pi32]),
        "jf_page_table_assign": (st, [P, i32, P, i32]),
        "jf_page_table_reserve": (st, [P, i32, i32]),
        "jf_page_table_set_length": (st, [P, i32, i32]),
        "jf_page_table_release": (st, [P, i32]),
        "jf_page_table_export": (st, [P, P, i32, i32, P, P]),
        "jf_page_table_stats": (st, [P, pi32, pi32, pi32]),
        "jf_page_table_info": (st, [P, i32, pi32, pi32]),
        "jf_kv_quantize_append": (st, [P, P, P, P, P, P, P, i32, i32, i32, P]),
        "jf_decode_workspace_bytes": (st, [i32, i32, i32, i32, ctypes.POINTER(sz)]),
        "jf_decode_attn_q4": (st, [P, P, P, i32, i32, P, i32, P, ctypes.c_float, i32, P, sz, P,
                                   P]),
        "jf_verify_attn_q4": (st, [P, P, P, i32, i32, i32, P, i32, P, ctypes.c_float, i32, P, sz,
                                   P, P]),
        "jf_decode_step_q4": (st, [P, P, P, P, P, i32, i32, P, i32, P, ctypes.c_float, i32, P, sz,
                                   P, P]),
        "jf_decode_step_q4_static": (st, [P, P, P, P, P, i32, i32, P, i32, P, ctypes.c_float,
                                          i32, P, P]),
        "jf_prefill_attn_q4": (st, [P, P, P, P, P, i32, i32, P, i32, i32, ctypes.c_float, P, P]),
        "jf_reconstruct_q4": (st, [P, P, P, i32, i32, i32, i32, P, P, P]),
        "jf_tq4_reconstruct": (st, [P, P, P, P, P, P, P, P, P, i32, i32, i32, i32, P, P, P]),
        "jf_kv_page_bytes": (st, [P, ctypes.POINTER(sz)]),
        "jf_kv_pack_pages": (st, [P, P, P, i32, i32, P, P]),
        "jf_kv_unpack_pages": (st, [P, P, P, i32, i32, P, P]),
        "jf_calib_read_stream": (st, [P, sz, i32, P, P]),
        "jf_snapshot_save": (st, [ctypes.c_char_p, P, P, i32, P, P, i32, i32, P, P, sz, P]),
        "jf_snapshot_restore": (st, [ctypes.c_char_p, P, P, i32, P, P, i32, P, P, sz, pi32, P]),
        "jf_tq4_pool_bytes": (st, [P, ctypes.POINTER(sz), ctypes.POINTER(sz)]),
        "jf_tq4_encode_append": (st, [P, P, P, P, P, P, P, P, P, i32, i32, i32, P]),
        "jf_tq4_decode_attn": (st, [P, P, P, P, P, P, P, P, P, i32, i32, P, i32, P,
                                    ctypes.c_float, i32, P, sz, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


lib = _load()


def _check(status: int):
    if status != JF_OK:
        raise JfError(status, lib.jf_last_error().decode())


def version() -> str:
    return lib.jf_version().decode()


def layout(page_size: int, num_kv_heads: int, head_dim: int, group_size: int,
           num_pages: int) -> Layout:
    return Layout(page_size, num_kv_heads, head_dim, group_size, num_pages)


def kv_pool_bytes(lay: Layout):
    cb, mb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib.jf_kv_pool_bytes(ctypes.byref(lay), ctypes.byref(cb), ctypes.byref(mb)))
    return cb.value, mb.value


# ------------------------------------------------------------ page tables
class PagePool:
    """Host page allocator with per-request page tables (owned by the library)."""

    def __init__(self, num_pages: int, page_size: int, shuffle_seed: int = 0):
        h = ctypes.c_void_p()
        _check(lib.jf_page_table_pool_create(num_pages, page_size, shuffle_seed, ctypes.byref(h)))
        self._h = h
        self.num_pages = num_pages
        self.page_size = page_size

    def close(self):
        if self._h:
            _check(lib.jf_page_table_pool_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def create(self) -> int:
        s = ctypes.c_int32()
        _check(lib.jf_page_table_create(self._h, ctypes.byref(s)))
        return s.value

    def fork(self, src: int, prefix_len: int) -> int:
        s = ctypes.c_int32()
        _check(lib.jf_page_table_fork(self._h, src, prefix_len, ctypes.byref(s)))
        return s.value

    def assign(self, seq: int, page_ids: Sequence[int]):
        arr = (ctypes.c_int32 * len(page_ids))(*[int(p) for p in page_ids])
        _check(lib.jf_page_table_assign(self._h, seq, arr, len(page_ids)))

    def reserve(self, seq: int, new_len: int):
        _check(lib.jf_page_table_reserve(self._h, seq, new_len))

    def set_length(self, seq: int, length: int):
        _check(lib.jf_page_table_set_length(self._h, seq, length))

    def release(self, seq: int):
        _check(lib.jf_page_table_release(self._h, seq))

    def export(self, seqs: Sequence[int], max_pages: int):
        """-> (block_table list[list[int]] padded with -1, lens list[int])."""
        n = len(seqs)
        s = (ctypes.c_int32 * max(n, 1))(*seqs)
        bt = (ctypes.c_int32 * max(n * max_pages, 1))()
        ln = (ctypes.c_int32 * max(n, 1))()
        _check(lib.jf_page_table_export(self._h, s, n, max_pages, bt, ln))
        table = [list(bt[i * max_pages:(i + 1) * max_pages]) for i in range(n)]
        return table, list(ln[:n])

    def stats(self):
        f, u, h = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib.jf_page_table_stats(self._h, ctypes.byref(f), ctypes.byref(u), ctypes.byref(h)))
        return {"free": f.value, "used": u.value, "high_water": h.value}

    def info(self, seq: int):
        n, ln = ctypes.c_int32(), ctypes.c_int32()
        _check(lib.jf_page_table_info(self._h, seq, ctypes.byref(n), ctypes.byref(ln)))
        return n.value, ln.value


# ------------------------------------------------------------ device work
def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


class KVPool:
    """One layer's K and V pools in device memory (uint8 codes, fp16 meta)."""

    def __init__(self, lay: Layout, device="cuda", fill: Optional[int] = None):
        import torch
        self.layout = lay
        cb, mb = kv_pool_bytes(lay)

        def buf(n):
            t = torch.empty(n, dtype=torch.uint8, device=device)
            if fill is not None:
                t.fill_(fill)
            return t

        self.k_codes = buf(cb)
        self.v_codes = buf(cb)
        self.k_meta = buf(mb).view(torch.float16)
        self.v_meta = buf(mb).view(torch.float16)

    def ptrs(self) -> PoolPtrs:
        return PoolPtrs(self.k_codes.data_ptr(), self.k_meta.data_ptr(),
                        self.v_codes.data_ptr(), self.v_meta.data_ptr())


def _dev_check(t, name, dtype=None):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))


def _check_append_args(pool: KVPool, k_new, v_new, cu_tok, start_pos, block_tables):
    import torch
    for t, n, dt in ((k_new, "k_new", torch.float16), (v_new, "v_new", torch.float16),
                     (cu_tok, "cu_tok", torch.int32), (start_pos, "start_pos", torch.int32),
                     (block_tables, "block_tables", torch.int32)):
        _dev_check(t, n, dt)
    lay = pool.layout
    total = k_new.shape[0]
    if tuple(k_new.shape) != (total, lay.num_kv_heads, lay.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [total_tok][Hkv][d]")
    B = start_pos.shape[0]
    if cu_tok.shape[0] != B + 1 or block_tables.dim() != 2 or block_tables.shape[0] != B:
        raise ValueError("cu_tok [B+1], start_pos [B], block_tables [B][max_pages]")


def jf_kv_quantize_append(pool: KVPool, k_new, v_new, cu_tok, start_pos, block_tables,
                          stream=None):
    _check_append_args(pool, k_new, v_new, cu_tok, start_pos, block_tables)
    lay = pool.layout
    total = k_new.shape[0]
    B = start_pos.shape[0]
    ptrs = pool.ptrs()
    _check(lib.jf_kv_quantize_append(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(k_new),
                                     _ptr(v_new), _ptr(cu_tok), _ptr(start_pos),
                                     _ptr(block_tables), B, block_tables.shape[1], total,
                                     _stream(stream)))


def decode_head_chunk(head_dim: int, group_size: int, gq: int) -> int:
    """Query heads one decode block serves (a head chunk; the split cap of
    jf_decode_attn_q4 divides the compute units by num_kv_heads * ceil(Gq /
    this)).  A column set holds 4 heads for 32-dim groups or head_dim 256,
    else 8; blocks take two sets when Gq (query heads per KV head, times
    tokens for the verifier) exceeds one set and head_dim <= 128."""
    hs = 4 if group_size == 32 or head_dim == 256 else 8
    return 2 * hs if head_dim <= 128 and gq > hs else hs


def jf_decode_workspace_bytes(B: int, num_q_heads: int, head_dim: int, max_splits: int) -> int:
    n = ctypes.c_size_t()
    _check(lib.jf_decode_workspace_bytes(B, num_q_heads, head_dim, max_splits, ctypes.byref(n)))
    return n.value


def _check_decode_args(pool: KVPool, q, block_tables, seq_lens, workspace, out):
    import torch
    _dev_check(q, "q", torch.float16)
    _dev_check(block_tables, "block_tables", torch.int32)
    _dev_check(seq_lens, "seq_lens", torch.int32)
    _dev_check(workspace, "workspace")
    _dev_check(out, "out", torch.float16)
    B, Hq, d = q.shape
    if d != pool.layout.head_dim or out.shape != q.shape:
        raise ValueError("q/out must be [B][Hq][head_dim]")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_tables [B][max_pages], seq_lens [B]")


def _check_step_args(pool: KVPool, k_new, v_new, q, block_tables, seq_lens, workspace, out):
    import torch
    _dev_check(k_new, "k_new", torch.float16)
    _dev_check(v_new, "v_new", torch.float16)
    lay = pool.layout
    B = q.shape[0]
    if tuple(k_new.shape) != (B, lay.num_kv_heads, lay.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [B][Hkv][head_dim]")
    _check_decode_args(pool, q, block_tables, seq_lens, workspace, out)


def jf_decode_attn_q4(pool: KVPool, q, block_tables, seq_lens, softmax_scale: float,
                      max_splits: int, workspace, out, stream=None):
    _check_decode_args(pool, q, block_tables, seq_lens, workspace, out)
    lay = pool.layout
    B, Hq, d = q.shape
    ptrs = pool.ptrs()
    _check(lib.jf_decode_attn_q4(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(q), B, Hq,
                                 _ptr(block_tables), block_tables.shape[1], _ptr(seq_lens),
                                 float(softmax_scale), int(max_splits), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _ptr(out),
                                 _stream(stream)))


def jf_verify_attn_q4(pool: KVPool, q, block_tables, seq_lens, softmax_scale: float,
                      max_splits: int, workspace, out, stream=None):
    """Short packed verification: q, out fp16 [B][Sq][Hq][d] (Sq = 1..4); token
    k of request b sees positions 0 .. seq_lens[b] - Sq + k."""
    import torch
    _dev_check(q, "q", torch.float16)
    _dev_check(block_tables, "block_tables", torch.int32)
    _dev_check(seq_lens, "seq_lens", torch.int32)
    _dev_check(workspace, "workspace")
    _dev_check(out, "out", torch.float16)
    if q.dim() != 4 or q.shape[3] != pool.layout.head_dim or out.shape != q.shape:
        raise ValueError("q/out must be [B][Sq][Hq][head_dim]")
    B, Sq, Hq, _ = q.shape
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_tables [B][max_pages], seq_lens [B]")
    lay = pool.layout
    ptrs = pool.ptrs()
    _check(lib.jf_verify_attn_q4(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(q), B, Sq, Hq,
                                 _ptr(block_tables), block_tables.shape[1], _ptr(seq_lens),
                                 float(softmax_scale), int(max_splits), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _ptr(out),
                                 _stream(stream)))


def jf_decode_step_q4(pool: KVPool, k_new, v_new, q, block_tables, seq_lens,
                      softmax_scale: float, max_splits: int, workspace, out, stream=None):
    """Append request b's row (k_new/v_new fp16 [B][Hkv][d]) at position
    seq_lens[b] - 1, then attend over seq_lens[b] positions; one kernel."""
    _check_step_args(pool, k_new, v_new, q, block_tables, seq_lens, workspace, out)
    lay = pool.layout
    B = q.shape[0]
    ptrs = pool.ptrs()
    _check(lib.jf_decode_step_q4(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(k_new), _ptr(v_new),
                                 _ptr(q), B, q.shape[1], _ptr(block_tables), block_tables.shape[1],
                                 _ptr(seq_lens), float(softmax_scale), int(max_splits),
                                 _ptr(workspace), workspace.numel() * workspace.element_size(),
                                 _ptr(out), _stream(stream)))


def jf_decode_step_q4_static(pool: KVPool, k_new, v_new, q, block_tables, seq_lens,
                             softmax_scale: float, max_splits: int, out, stream=None):
    """jf_decode_step_q4 with the library's static device scratch in place of a
    workspace (for callers that cannot allocate); see include/jfkv.h."""
    import torch
    _dev_check(k_new, "k_new", torch.float16)
    _dev_check(v_new, "v_new", torch.float16)
    _dev_check(q, "q", torch.float16)
    _dev_check(block_tables, "block_tables", torch.int32)
    _dev_check(seq_lens, "seq_lens", torch.int32)
    _dev_check(out, "out", torch.float16)
    lay = pool.layout
    B, Hq, d = q.shape
    if d != lay.head_dim or out.shape != q.shape:
        raise ValueError("q/out must be [B][Hq][head_dim]")
    if tuple(k_new.shape) != (B, lay.num_kv_heads, d) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [B][Hkv][head_dim]")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_tables [B][max_pages], seq_lens [B]")
    ptrs = pool.ptrs()
    _check(lib.jf_decode_step_q4_static(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(k_new),
                                        _ptr(v_new), _ptr(q), B, Hq, _ptr(block_tables),
                                        block_tables.shape[1], _ptr(seq_lens),
                                        float(softmax_scale), int(max_splits), _ptr(out),
                                        _stream(stream)))


def _check_prefill_args(pool: KVPool, q, k_chunk, v_chunk, block_table, out):
    import torch
    _dev_check(q, "q", torch.float16)
    _dev_check(k_chunk, "k_chunk", torch.float16)
    _dev_check(v_chunk, "v_chunk", torch.float16)
    _dev_check(block_table, "block_table", torch.int32)
    _dev_check(out, "out", torch.float16)
    lay = pool.layout
    T, Hq, d = q.shape
    if d != lay.head_dim or out.shape != q.shape:
        raise ValueError("q/out must be [T][Hq][head_dim]")
    if tuple(k_chunk.shape) != (T, lay.num_kv_heads, d) or v_chunk.shape != k_chunk.shape:
        raise ValueError("k_chunk/v_chunk must be [T][Hkv][head_dim]")


def jf_prefill_attn_q4(pool: KVPool, q, k_chunk, v_chunk, block_table, prefix_len: int,
                       softmax_scale: float, out, stream=None):
    _check_prefill_args(pool, q, k_chunk, v_chunk, block_table, out)
    lay = pool.layout
    T, Hq, d = q.shape
    ptrs = pool.ptrs()
    _check(lib.jf_prefill_attn_q4(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(q), _ptr(k_chunk),
                                  _ptr(v_chunk), T, Hq, _ptr(block_table), block_table.shape[-1],
                                  int(prefix_len), float(softmax_scale), _ptr(out),
                                  _stream(stream)))


# ------------------------------------------------------------ pre-bound calls
class BoundCall:
    """A library call with its ctypes arguments marshalled once (for timing
    loops and graph capture, where per-call Python work would dominate)."""

    def __init__(self, fn, args, keep):
        self._fn = fn
        self._args = args
        self._keep = keep  # owners of the pointers (tensors, structs)

    def __call__(self):
        _check(self._fn(*self._args))


def bind_quantize_append(pool: KVPool, k_new, v_new, cu_tok, start_pos, block_tables,
                         stream=None) -> BoundCall:
    _check_append_args(pool, k_new, v_new, cu_tok, start_pos, block_tables)
    lay, ptrs = pool.layout, pool.ptrs()
    B = start_pos.shape[0]
    args = (ctypes.byref(lay), ctypes.byref(ptrs), _ptr(k_new), _ptr(v_new), _ptr(cu_tok),
            _ptr(start_pos), _ptr(block_tables), B, block_tables.shape[1], k_new.shape[0],
            _stream(stream))
    return BoundCall(lib.jf_kv_quantize_append, args,
                     (lay, ptrs, pool, k_new, v_new, cu_tok, start_pos, block_tables))


def bind_decode(pool: KVPool, q, block_tables, seq_lens, softmax_scale, max_splits, workspace,
                out, stream=None) -> BoundCall:
    _check_decode_args(pool, q, block_tables, seq_lens, workspace, out)
    lay, ptrs = pool.layout, pool.ptrs()
    B, Hq, _ = q.shape
    args = (ctypes.byref(lay), ctypes.byref(ptrs), _ptr(q), B, Hq, _ptr(block_tables),
            block_tables.shape[1], _ptr(seq_lens), float(softmax_scale), int(max_splits),
            _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(out),
            _stream(stream))
    return BoundCall(lib.jf_decode_attn_q4, args,
                     (lay, ptrs, pool, q, block_tables, seq_lens, workspace, out))


def bind_decode_step(pool: KVPool, k_new, v_new, q, block_tables, seq_lens, softmax_scale,
                     max_splits, workspace, out, stream=None) -> BoundCall:
    _check_step_args(pool, k_new, v_new, q, block_tables, seq_lens, workspace, out)
    lay, ptrs = pool.layout, pool.ptrs()
    B, Hq, _ = q.shape
    args = (ctypes.byref(lay), ctypes.byref(ptrs), _ptr(k_new), _ptr(v_new), _ptr(q), B, Hq,
            _ptr(block_tables), block_tables.shape[1], _ptr(seq_lens), float(softmax_scale),
            int(max_splits), _ptr(workspace), workspace.numel() * workspace.element_size(),
            _ptr(out), _stream(stream))
    return BoundCall(lib.jf_decode_step_q4, args,
                     (lay, ptrs, pool, k_new, v_new, q, block_tables, seq_lens, workspace, out))


def bind_verify(pool: KVPool, q, block_tables, seq_lens, softmax_scale, max_splits, workspace,
                out, stream=None) -> BoundCall:
    """jf_verify_attn_q4 with its arguments marshalled once (q, out [B][Sq][Hq][d])."""
    lay, ptrs = pool.layout, pool.ptrs()
    if q.dim() != 4 or out.shape != q.shape or q.shape[3] != lay.head_dim:
        raise ValueError("q/out must be [B][Sq][Hq][head_dim]")
    B, Sq, Hq, _ = q.shape
    args = (ctypes.byref(lay), ctypes.byref(ptrs), _ptr(q), B, Sq, Hq, _ptr(block_tables),
            block_tables.shape[1], _ptr(seq_lens), float(softmax_scale), int(max_splits),
            _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(out),
            _stream(stream))
    return BoundCall(lib.jf_verify_attn_q4, args,
                     (lay, ptrs, pool, q, block_tables, seq_lens, workspace, out))


def bind_prefill(pool: KVPool, q, k_chunk, v_chunk, block_table, prefix_len, softmax_scale, out,
                 stream=None) -> BoundCall:
    _check_prefill_args(pool, q, k_chunk, v_chunk, block_table, out)
    lay, ptrs = pool.layout, pool.ptrs()
    T, Hq, _ = q.shape
    args = (ctypes.byref(lay), ctypes.byref(ptrs), _ptr(q), _ptr(k_chunk), _ptr(v_chunk), T, Hq,
            _ptr(block_table), block_table.shape[-1], int(prefix_len), float(softmax_scale),
            _ptr(out), _stream(stream))
    return BoundCall(lib.jf_prefill_attn_q4, args,
                     (lay, ptrs, pool, q, k_chunk, v_chunk, block_table, out))


def jf_reconstruct_q4(pool: KVPool, block_table, n_pos: int, kv0: int, num_heads: int, k_out,
                      v_out, stream=None):
    """K, V of KV heads kv0 .. kv0+num_heads-1 at positions 0..n_pos-1 as fp16
    k_out, v_out [num_heads][n_pos][d] (block_table int32 [max_pages])."""
    import torch
    _dev_check(block_table, "block_table", torch.int32)
    _dev_check(k_out, "k_out", torch.float16)
    _dev_check(v_out, "v_out", torch.float16)
    lay = pool.layout
    shape = (num_heads, n_pos, lay.head_dim)
    if tuple(k_out.shape) != shape or tuple(v_out.shape) != shape:
        raise ValueError("k_out/v_out must be [num_heads][n_pos][head_dim]")
    ptrs = pool.ptrs()
    _check(lib.jf_reconstruct_q4(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(block_table),
                                 block_table.shape[-1], int(n_pos), int(kv0), int(num_heads),
                                 _ptr(k_out), _ptr(v_out), _stream(stream)))


# ---------------------------------------------------------------- TQ4 format
def tq4_pool_bytes(lay: Layout):
    w, n = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib.jf_tq4_pool_bytes(ctypes.byref(lay), ctypes.byref(w), ctypes.byref(n)))
    return w.value, n.value


class TQ4Pool:
    """One layer's TQ4 pool for K or V in device memory: index words (u32 bit
    patterns held as int32) [num_pages][num_kv_heads][page_size][head_dim/8]
    and fp16 norms [num_pages][num_kv_heads][page_size]."""

    def __init__(self, lay: Layout, device="cuda", fill: Optional[int] = None):
        import torch
        self.layout = lay
        wb, nb = tq4_pool_bytes(lay)
        w = torch.empty(wb, dtype=torch.uint8, device=device)
        n = torch.empty(nb, dtype=torch.uint8, device=device)
        if fill is not None:
            w.fill_(fill)
            n.fill_(fill)
        shape = (lay.num_pages, lay.num_kv_heads, lay.page_size)
        self.words = w.view(torch.int32).view(*shape, lay.head_dim // 8)
        self.norms = n.view(torch.float16).view(*shape)


def _check_tq4_args(pool: TQ4Pool, x, signs, centroids, cu_tok, start_pos, block_tables):
    import torch
    for t, n, dt in ((x, "x", torch.float16), (signs, "signs", torch.float32),
                     (centroids, "centroids", torch.float32), (cu_tok, "cu_tok", torch.int32),
                     (start_pos, "start_pos", torch.int32),
                     (block_tables, "block_tables", torch.int32)):
        _dev_check(t, n, dt)
    lay = pool.layout
    if x.dim() != 3 or tuple(x.shape[1:]) != (lay.num_kv_heads, lay.head_dim):
        raise ValueError("x must be [total_tok][Hkv][head_dim]")
    if signs.numel() != lay.head_dim or centroids.numel() != 16:
        raise ValueError("signs [head_dim], centroids [16]")
    B = start_pos.shape[0]
    if cu_tok.shape[0] != B + 1 or block_tables.dim() != 2 or block_tables.shape[0] != B:
        raise ValueError("cu_tok [B+1], start_pos [B], block_tables [B][max_pages]")


def jf_tq4_encode_append(pool: TQ4Pool, x, signs, centroids, cu_tok, start_pos, block_tables,
                         stream=None):
    """Encode rows x [total_tok][Hkv][256] (fp16) into a TQ4 pool at their
    logical positions (see include/jfkv.h)."""
    _check_tq4_args(pool, x, signs, centroids, cu_tok, start_pos, block_tables)
    _check(lib.jf_tq4_encode_append(ctypes.byref(pool.layout), _ptr(pool.words), _ptr(pool.norms),
                                    _ptr(x), _ptr(signs), _ptr(centroids), _ptr(cu_tok),
                                    _ptr(start_pos), _ptr(block_tables), start_pos.shape[0],
                                    block_tables.shape[1], x.shape[0], _stream(stream)))


def bind_tq4_encode_append(pool: TQ4Pool, x, signs, centroids, cu_tok, start_pos, block_tables,
                           stream=None) -> "BoundCall":
    """jf_tq4_encode_append with its arguments checked and marshalled once."""
    _check_tq4_args(pool, x, signs, centroids, cu_tok, start_pos, block_tables)
    lay = pool.layout
    args = (ctypes.byref(lay), _ptr(pool.words), _ptr(pool.norms), _ptr(x), _ptr(signs),
            _ptr(centroids), _ptr(cu_tok), _ptr(start_pos), _ptr(block_tables),
            start_pos.shape[0], block_tables.shape[1], x.shape[0], _stream(stream))
    return BoundCall(lib.jf_tq4_encode_append, args,
                     (lay, pool, x, signs, centroids, cu_tok, start_pos, block_tables))


def _tq4_decode_args(k_pool: TQ4Pool, v_pool: TQ4Pool, k_signs, v_signs, centroids, q,
                     block_tables, seq_lens, softmax_scale, max_splits, workspace, out, stream):
    import torch
    lay = k_pool.layout
    for t, n, dt in ((k_signs, "k_signs", torch.float32), (v_signs, "v_signs", torch.float32),
                     (centroids, "centroids", torch.float32), (q, "q", torch.float16),
                     (block_tables, "block_tables", torch.int32),
                     (seq_lens, "seq_lens", torch.int32), (out, "out", torch.float16)):
        _dev_check(t, n, dt)
    _dev_check(workspace, "workspace")
    if tuple(v_pool.words.shape) != tuple(k_pool.words.shape):
        raise ValueError("K and V pools must have the same layout")
    B, Hq, d = q.shape
    if d != lay.head_dim or out.shape != q.shape:
        raise ValueError("q/out must be [B][Hq][head_dim]")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_tables [B][max_pages], seq_lens [B]")
    return (ctypes.byref(lay), _ptr(k_pool.words), _ptr(k_pool.norms), _ptr(v_pool.words),
            _ptr(v_pool.norms), _ptr(k_signs), _ptr(v_signs), _ptr(centroids), _ptr(q), B, Hq,
            _ptr(block_tables), block_tables.shape[1], _ptr(seq_lens), float(softmax_scale),
            int(max_splits), _ptr(workspace), workspace.numel() * workspace.element_size(),
            _ptr(out), _stream(stream))


def jf_tq4_decode_attn(k_pool: TQ4Pool, v_pool: TQ4Pool, k_signs, v_signs, centroids, q,
                       block_tables, seq_lens, softmax_scale: float, max_splits: int, workspace,
                       out, stream=None):
    """Decode attention of q [B][Hq][256] (fp16) over TQ4 K/V pools through the
    page tables (see include/jfkv.h); the workspace is sized by
    jf_decode_workspace_bytes(B, Hq, 256, max_splits) and zero-filled once."""
    _check(lib.jf_tq4_decode_attn(*_tq4_decode_args(k_pool, v_pool, k_signs, v_signs, centroids,
                                                    q, block_tables, seq_lens, softmax_scale,
                                                    max_splits, workspace, out, stream)))


def bind_tq4_decode(k_pool: TQ4Pool, v_pool: TQ4Pool, k_signs, v_signs, centroids, q,
                    block_tables, seq_lens, softmax_scale, max_splits, workspace, out,
                    stream=None) -> "BoundCall":
    """jf_tq4_decode_attn with its arguments checked and marshalled once."""
    args = _tq4_decode_args(k_pool, v_pool, k_signs, v_signs, centroids, q, block_tables,
                            seq_lens, softmax_scale, max_splits, workspace, out, stream)
    return BoundCall(lib.jf_tq4_decode_attn, args,
                     (k_pool, v_pool, k_signs, v_signs, centroids, q, block_tables, seq_lens,
                      workspace, out))


def jf_tq4_reconstruct(k_pool: TQ4Pool, v_pool: TQ4Pool, k_signs, v_signs, centroids,
                       block_table, n_pos: int, kv0: int, num_heads: int, k_out, v_out,
                       stream=None):
    """x_hat = norm * S H c[z] / 16 of KV heads kv0 .. kv0+num_heads-1 at
    positions 0..n_pos-1 as fp16 k_out, v_out [num_heads][n_pos][256]."""
    import torch
    for t, n, dt in ((k_signs, "k_signs", torch.float32), (v_signs, "v_signs", torch.float32),
                     (centroids, "centroids", torch.float32),
                     (block_table, "block_table", torch.int32), (k_out, "k_out", torch.float16),
                     (v_out, "v_out", torch.float16)):
        _dev_check(t, n, dt)
    lay = k_pool.layout
    if tuple(v_pool.words.shape) != tuple(k_pool.words.shape):
        raise ValueError("K and V pools must have the same layout")
    shape = (num_heads, n_pos, lay.head_dim)
    if tuple(k_out.shape) != shape or tuple(v_out.shape) != shape:
        raise ValueError("k_out/v_out must be [num_heads][n_pos][head_dim]")
    _check(lib.jf_tq4_reconstruct(ctypes.byref(lay), _ptr(k_pool.words), _ptr(k_pool.norms),
                                  _ptr(v_pool.words), _ptr(v_pool.norms), _ptr(k_signs),
                                  _ptr(v_signs), _ptr(centroids), _ptr(block_table),
                                  block_table.shape[-1], int(n_pos), int(kv0), int(num_heads),
                                  _ptr(k_out), _ptr(v_out), _stream(stream)))


# ---------------------------------------------------------------- snapshots
def kv_page_bytes(lay: Layout) -> int:
    n = ctypes.c_size_t()
    _check(lib.jf_kv_page_bytes(ctypes.byref(lay), ctypes.byref(n)))
    return n.value


def jf_calib_read_stream(buf, blocks: int, sink, stream=None):
    """One read of buf (device, 16-byte multiple) with the kernels' load type
    (read-rate calibration)."""
    import torch
    if not buf.is_cuda or not sink.is_cuda or buf.numel() * buf.element_size() % 16:
        raise ValueError("buf and sink must be device tensors, buf a multiple of 16 bytes")
    _check(lib.jf_calib_read_stream(_ptr(buf), buf.numel() * buf.element_size(), int(blocks),
                                    _ptr(sink), _stream(stream)))


def jf_kv_pack_pages(pool: KVPool, block_table, first: int, count: int, buf, stream=None):
    """Pages block_table[first .. first+count-1] -> buf (device uint8)."""
    import torch
    _dev_check(block_table, "block_table", torch.int32)
    if buf.dtype != torch.uint8 or buf.numel() < count * kv_page_bytes(pool.layout):
        raise ValueError("buf must be uint8 with count * page_bytes bytes")
    lay, ptrs = pool.layout, pool.ptrs()
    _check(lib.jf_kv_pack_pages(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(block_table),
                                int(first), int(count), _ptr(buf), _stream(stream)))


def jf_kv_unpack_pages(pool: KVPool, block_table, first: int, count: int, buf, stream=None):
    """buf (device uint8) -> pages block_table[first .. first+count-1]."""
    import torch
    _dev_check(block_table, "block_table", torch.int32)
    if buf.dtype != torch.uint8 or buf.numel() < count * kv_page_bytes(pool.layout):
        raise ValueError("buf must be uint8 with count * page_bytes bytes")
    lay, ptrs = pool.layout, pool.ptrs()
    _check(lib.jf_kv_unpack_pages(ctypes.byref(lay), ctypes.byref(ptrs), _ptr(block_table),
                                  int(first), int(count), _ptr(buf), _stream(stream)))


def _snapshot_args(pools, block_table, block_table_host, staging_dev, staging):
    import numpy as np
    import torch
    lay = pools[0].layout
    for p in pools:
        if tuple(getattr(p.layout, f) for f, _ in Layout._fields_) != \
                tuple(getattr(lay, f) for f, _ in Layout._fields_):
            raise ValueError("every layer's pool must have the same layout")
    _dev_check(block_table, "block_table", torch.int32)
    _dev_check(staging_dev, "staging_dev", torch.uint8)
    if staging.dtype != torch.uint8 or staging.device.type != "cpu" or not staging.is_pinned():
        raise ValueError("staging must be a pinned host uint8 tensor")
    if staging.numel() != staging_dev.numel():
        raise ValueError("staging and staging_dev must have the same size")
    host = np.ascontiguousarray(np.asarray(block_table_host, np.int32).reshape(-1))
    if host.shape[0] != block_table.reshape(-1).shape[0]:
        raise ValueError("block_table and block_table_host must have the same length")
    arr = (PoolPtrs * len(pools))(*[p.ptrs() for p in pools])
    return lay, arr, host


def snapshot_save(path: str, pools, block_table, block_table_host, n_pos: int, staging_dev,
                  staging, stream=None):
    """Save positions 0..n_pos-1 of one request, every layer in `pools`, to
    `path` (safetensors; see include/jfkv.h), through staging_dev (device) and
    staging (pinned host), uint8 buffers of equal size."""
    lay, arr, host = _snapshot_args(pools, block_table, block_table_host, staging_dev, staging)
    _check(lib.jf_snapshot_save(os.fsencode(path), ctypes.byref(lay), arr, len(pools),
                                _ptr(block_table), host.ctypes.data, host.shape[0], int(n_pos),
                                _ptr(staging_dev), _ptr(staging), staging.numel(),
                                _stream(stream)))


def snapshot_restore(path: str, pools, block_table, block_table_host, staging_dev, staging,
                     stream=None) -> int:
    """Restore a snapshot into the request pages listed in block_table; returns n_pos."""
    lay, arr, host = _snapshot_args(pools, block_table, block_table_host, staging_dev, staging)
    n = ctypes.c_int32()
    _check(lib.jf_snapshot_restore(os.fsencode(path), ctypes.byref(lay), arr, len(pools),
                                   _ptr(block_table), host.ctypes.data, host.shape[0],
                                   _ptr(staging_dev), _ptr(staging), staging.numel(),
                                   ctypes.byref(n), _stream(stream)))
    return n.value
