"""ctypes binding of libherald.so (the C ABI in include/herald.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels. Device buffers are torch tensors on a ROCm device (their
``data_ptr()`` is passed through), streams are ``torch.cuda.Stream`` objects
or raw ``hipStream_t`` integers. Loading fails loudly when the library has not
been built (``python -m paper_2606_21633_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libherald.so")

F32, BF16 = 0, 1
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)

c_i32, c_i64, c_p, c_sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t


class Heads(ctypes.Structure):
    _fields_ = [("num_q_heads", c_i32), ("num_kv_heads", c_i32), ("head_dim", c_i32),
                ("dtype", ctypes.c_int)]


class KV(ctypes.Structure):
    _fields_ = [("k", c_p), ("v", c_p), ("stride_b", c_i64), ("stride_h", c_i64),
                ("stride_s", c_i64), ("page_table", c_p), ("page_size", c_i32),
                ("max_pages", c_i32), ("stride_page", c_i64), ("seq_lens", c_p),
                ("max_seq_len", c_i64)]


class Pool(ctypes.Structure):
    _fields_ = [("k", c_p), ("v", c_p), ("stride_b", c_i64), ("stride_h", c_i64),
                ("stride_s", c_i64), ("capacity", c_i32)]


class Layer(ctypes.Structure):
    _fields_ = [("cache", Pool), ("active", Pool), ("idle", Pool), ("q_steps", c_p),
                ("blk_k", c_p), ("blk_v", c_p), ("done_k", c_p), ("done_v", c_p),
                ("q_next", c_p), ("out", c_p), ("out_step_stride", c_i64),
                ("dense", c_i32), ("q_draft", c_p), ("draft_k", c_p), ("draft_v", c_p),
                ("out_draft", c_p), ("select_x", c_i32)]


class HeraldError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = _lib_or_none().herald_status_string(status).decode() if _lib_or_none() else ""
        super().__init__(f"{fn}: status {status} ({msg})")


_lib = None


def _lib_or_none():
    return _lib


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libherald.so not built at {LIB_PATH}; run "
                           "`python -m paper_2606_21633_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    L.herald_status_string.restype = ctypes.c_char_p
    L.herald_status_string.argtypes = [ctypes.c_int]
    L.herald_budget_tokens.restype = c_i32
    L.herald_budget_tokens.argtypes = [c_i64, c_i32, c_i32]
    L.herald_select_workspace.restype = c_sz
    L.herald_select_workspace.argtypes = [ctypes.POINTER(Heads), c_i32, c_i64]
    L.herald_select.restype = ctypes.c_int
    L.herald_select.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_p, ctypes.POINTER(KV),
                                c_p, c_i32, c_p, c_p, c_sz, c_p]
    L.herald_select_xq_workspace.restype = c_sz
    L.herald_select_xq_workspace.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i64]
    L.herald_select_xq.restype = ctypes.c_int
    L.herald_select_xq.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i32, c_p,
                                   ctypes.POINTER(KV), c_p, c_i32, c_p, c_p, c_sz, c_p]
    L.herald_select_draft.restype = ctypes.c_int
    L.herald_select_draft.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i32, c_p,
                                      ctypes.POINTER(KV), c_p, c_i32, c_p, c_i32, c_p, c_p,
                                      c_sz, c_p]
    L.herald_select_attn.restype = ctypes.c_int
    L.herald_select_attn.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i32, c_p,
                                     ctypes.POINTER(KV), c_p, c_p, c_i32, c_p, c_i32, c_p, c_p,
                                     c_p, c_sz, c_p]
    L.herald_gather.restype = ctypes.c_int
    L.herald_gather.argtypes = [ctypes.POINTER(Heads), c_i32, ctypes.POINTER(KV), c_p, c_p,
                                c_i32, ctypes.POINTER(Pool), c_i32, c_p]
    L.herald_block_attn_workspace.restype = c_sz
    L.herald_block_attn_workspace.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i64]
    L.herald_block_attn.restype = ctypes.c_int
    L.herald_block_attn.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_p,
                                    ctypes.POINTER(KV), c_p, c_p, c_p, c_p, c_sz, c_p]
    L.herald_block_attn_groups.restype = ctypes.c_int
    L.herald_block_attn_groups.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i32, c_p,
                                           ctypes.POINTER(KV), c_p, c_p, c_p, c_p, c_sz, c_p]
    L.herald_decode_block_workspace.restype = c_sz
    L.herald_decode_block_workspace.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i64,
                                                c_i32]
    L.herald_decode_block.restype = ctypes.c_int
    L.herald_decode_block.argtypes = [ctypes.POINTER(Heads), c_i32, c_i32, c_i32, c_i32,
                                      ctypes.POINTER(Layer), c_p, c_i64, c_p, c_i64, c_p, c_p,
                                      c_i32, c_i32, c_p, c_sz, c_p, c_p]
    _lib = L
    return L


EXPORTS = ("herald_status_string", "herald_budget_tokens", "herald_select_workspace",
           "herald_select", "herald_select_xq_workspace", "herald_select_xq",
           "herald_select_draft", "herald_select_attn",
           "herald_gather", "herald_block_attn_workspace",
           "herald_block_attn", "herald_block_attn_groups", "herald_decode_block_workspace",
           "herald_decode_block")


# ------------------------------------------------------------------ helpers


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> int | None:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(fn: str, st: int):
    if st != OK:
        raise HeraldError(fn, st)


def heads(num_q_heads: int, num_kv_heads: int, head_dim: int, dtype) -> Heads:
    """dtype: "bf16"/"f32", a torch dtype, or the enum value."""
    if not isinstance(dtype, int):
        name = str(dtype)
        dtype = BF16 if ("bf16" in name or "bfloat16" in name) else F32
    return Heads(num_q_heads, num_kv_heads, head_dim, dtype)


def kv_view(k, v, seq_lens, max_seq_len: int, page_table=None) -> KV:
    """KV view of torch tensors.

    Contiguous: k, v are [batch][Hkv][S_cap][d] (any tensor whose last three
    strides describe head/row/element; batch stride from dim 0).
    Paged: k, v are [n_pages][Hkv][page_size][d] and page_table is
    [batch][max_pages] int32.
    """
    kv = KV()
    kv.k, kv.v = _ptr(k), _ptr(v)
    kv.seq_lens = _ptr(seq_lens)
    kv.max_seq_len = int(max_seq_len)
    if page_table is None:
        kv.stride_b, kv.stride_h, kv.stride_s = k.stride(0), k.stride(1), k.stride(2)
        kv.page_table, kv.page_size, kv.max_pages, kv.stride_page = None, 0, 0, 0
    else:
        kv.stride_page, kv.stride_h, kv.stride_s = k.stride(0), k.stride(1), k.stride(2)
        kv.stride_b = 0
        kv.page_table = _ptr(page_table)
        kv.page_size = k.shape[2]
        kv.max_pages = page_table.shape[1]
    # the view holds raw device pointers: keep the tensors alive with it
    kv._refs = (k, v, seq_lens, page_table)
    return kv


def pool_view(k, v) -> Pool:
    """Writable view of [batch][Hkv][capacity][d] tensors."""
    pool = Pool(_ptr(k), _ptr(v), k.stride(0), k.stride(1), k.stride(2), k.shape[2])
    pool._refs = (k, v)  # keep the tensors alive with the view
    return pool


# ------------------------------------------------------------------ entry points


def budget_tokens(S: int, num: int = 1, den: int = 20) -> int:
    return int(lib().herald_budget_tokens(int(S), int(num), int(den)))


def select_workspace(hd: Heads, batch: int, max_seq_len: int) -> int:
    return int(lib().herald_select_workspace(ctypes.byref(hd), batch, max_seq_len))


def select(hd: Heads, batch: int, block: int, q_sel, kv: KV, k_per_seq, k_max: int,
           idx_out, ws, ws_bytes: int | None = None, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().herald_select(ctypes.byref(hd), batch, block, _ptr(q_sel), ctypes.byref(kv),
                             _ptr(k_per_seq), k_max, _ptr(idx_out), _ptr(ws), nbytes,
                             _stream(stream))
    _check("herald_select", st)


def select_xq_workspace(hd: Heads, batch: int, x: int, max_seq_len: int) -> int:
    return int(lib().herald_select_xq_workspace(ctypes.byref(hd), batch, x, max_seq_len))


def select_xq(hd: Heads, batch: int, block: int, x: int, q_sel, kv: KV, k_per_seq, k_max: int,
              idx_out, ws, ws_bytes: int | None = None, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().herald_select_xq(ctypes.byref(hd), batch, block, x, _ptr(q_sel),
                                ctypes.byref(kv), _ptr(k_per_seq), k_max, _ptr(idx_out),
                                _ptr(ws), nbytes, _stream(stream))
    _check("herald_select_xq", st)


def select_draft(hd: Heads, batch: int, block: int, x: int, q_sel, kv: KV, draft_k, n_draft: int,
                 k_per_seq, k_max: int, idx_out, ws, ws_bytes: int | None = None, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().herald_select_draft(ctypes.byref(hd), batch, block, x, _ptr(q_sel),
                                   ctypes.byref(kv), _ptr(draft_k), n_draft, _ptr(k_per_seq),
                                   k_max, _ptr(idx_out), _ptr(ws), nbytes, _stream(stream))
    _check("herald_select_draft", st)


def select_attn(hd: Heads, batch: int, block: int, x: int, q_sel, kv: KV, draft_k, draft_v,
                n_draft: int, k_per_seq, k_max: int, idx_out, o_out, ws,
                ws_bytes: int | None = None, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().herald_select_attn(ctypes.byref(hd), batch, block, x, _ptr(q_sel),
                                  ctypes.byref(kv), _ptr(draft_k), _ptr(draft_v), n_draft,
                                  _ptr(k_per_seq), k_max, _ptr(idx_out), _ptr(o_out), _ptr(ws),
                                  nbytes, _stream(stream))
    _check("herald_select_attn", st)


def gather(hd: Heads, batch: int, kv: KV, idx, k_per_seq, k_max: int, dst: Pool,
           dst_row0: int = 0, stream=None):
    st = lib().herald_gather(ctypes.byref(hd), batch, ctypes.byref(kv), _ptr(idx),
                             _ptr(k_per_seq), k_max, ctypes.byref(dst), dst_row0,
                             _stream(stream))
    _check("herald_gather", st)


def block_attn_workspace(hd: Heads, batch: int, block: int, max_ctx: int) -> int:
    return int(lib().herald_block_attn_workspace(ctypes.byref(hd), batch, block, max_ctx))


def block_attn(hd: Heads, batch: int, block: int, q, ctx: KV, blk_k, blk_v, out, ws,
               ws_bytes: int | None = None, stream=None):
    nbytes = (ws.numel() * ws.element_size() if ws is not None else 0) \
        if ws_bytes is None else ws_bytes
    st = lib().herald_block_attn(ctypes.byref(hd), batch, block, _ptr(q), ctypes.byref(ctx),
                                 _ptr(blk_k), _ptr(blk_v), _ptr(out), _ptr(ws), nbytes,
                                 _stream(stream))
    _check("herald_block_attn", st)


def block_attn_groups(hd: Heads, batch: int, block: int, groups: int, q, ctx: KV, blk_k, blk_v,
                      out, ws, ws_bytes: int | None = None, stream=None):
    nbytes = (ws.numel() * ws.element_size() if ws is not None else 0) \
        if ws_bytes is None else ws_bytes
    st = lib().herald_block_attn_groups(ctypes.byref(hd), batch, block, groups, _ptr(q),
                                        ctypes.byref(ctx), _ptr(blk_k), _ptr(blk_v), _ptr(out),
                                        _ptr(ws), nbytes, _stream(stream))
    _check("herald_block_attn_groups", st)


def decode_block_workspace(hd: Heads, batch: int, block: int, max_seq_len: int,
                           k_max: int) -> int:
    return int(lib().herald_decode_block_workspace(ctypes.byref(hd), batch, block,
                                                   max_seq_len, k_max))


def decode_block(hd: Heads, layers, batch: int, block: int, steps: int, seq_lens,
                 max_seq_len: int, n_active, max_active: int, n_idle, k_next, k_max: int,
                 dense: bool, ws, s_main=None, s_retr=None, ws_bytes: int | None = None):
    arr = (Layer * len(layers))(*layers)
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().herald_decode_block(ctypes.byref(hd), len(layers), batch, block, steps, arr,
                                   _ptr(seq_lens), max_seq_len, _ptr(n_active), max_active,
                                   _ptr(n_idle), _ptr(k_next), k_max, int(bool(dense)),
                                   _ptr(ws), nbytes, _stream(s_main), _stream(s_retr))
    _check("herald_decode_block", st)


def workspace(nbytes: int, device):
    """A 256-byte aligned device workspace of at least nbytes (torch-owned)."""
    import torch
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
