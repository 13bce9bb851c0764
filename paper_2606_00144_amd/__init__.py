"""Python binding of libbd: the BudgetDraft sparse-drafter / full-verifier hot path on MI355X.

Argument marshalling only.  Every step runs in the gfx950 HIP kernels of
``libbd.so`` (built in-tree by ``python -m paper_2606_00144_amd.build``);
torch provides device memory and the current HIP stream.  There is no CPU
fallback: if the library is missing or a call is rejected, a ``BdError`` is
raised.

Functions carry the names of the C entry points:

    bd_select_kv, bd_select_kv_chunks, bd_sparse_decode_attn,
    bd_multiview_attn, bd_multiview_attn_bwd, bd_verify_attn, bd_verify_attn_noalloc, bd_accept_len,
    bd_cache_append, bd_cache_rollback, bd_top1_ce, bd_sample_budgets

KV caches are bf16 tensors, either contiguous ``[S][Hkv][L][128]`` or paged
``[num_pages][Hkv][page_size][128]`` together with an int32 ``page_table``
``[S][max_pages]``.  ``seq_lens`` is an int32 device tensor ``[S]``.
"""
from __future__ import annotations

import ctypes
import math
import os
import threading
from typing import Optional

import torch

__all__ = [
    "BdError", "lib", "library_path", "kv_desc", "Workspace",
    "bd_select_kv", "bd_select_kv_chunks", "bd_sparse_decode_attn", "bd_multiview_attn", "bd_multiview_attn_bwd", "bd_verify_attn",
    "bd_verify_attn_noalloc", "bd_accept_len",
    "bd_cache_append", "bd_cache_rollback", "bd_top1_ce", "bd_sample_budgets",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.environ.get("BD_LIBRARY") or os.path.join(_HERE, "libbd.so")

BD_OK, BD_ERR_INVALID_ARG, BD_ERR_UNSUPPORTED, BD_ERR_WORKSPACE, BD_ERR_DEVICE = range(5)
HEAD_DIM = 128


class BdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libbd status {status}: {msg}")
        self.status = status


class KvDesc(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("num_seqs", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32), ("seq_lens", ctypes.c_void_p),
        ("stride_seq", ctypes.c_int64), ("stride_head", ctypes.c_int64), ("stride_tok", ctypes.c_int64),
        ("page_table", ctypes.c_void_p), ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int32), ("stride_page", ctypes.c_int64),
    ]


_P = ctypes.c_void_p
_I32, _I64, _F32, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
_KV = ctypes.POINTER(KvDesc)

_SIGNATURES = {
    "bd_status_string": (ctypes.c_char_p, [_I32]),
    "bd_last_error": (ctypes.c_char_p, []),
    "bd_abi_version": (_I32, []),
    "bd_select_kv_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, _I32]),
    "bd_select_kv": (_I32, [_KV, _P, _I32, _I32, _I32, _I32, _F32, _P, _P, _P, _P, _P, _SZ, _P]),
    "bd_select_kv_chunks": (_I32, [_KV, _P, _I32, _I32, _I32, _I32, _I32, _F32, _P, _P, _P, _P, _P, _SZ, _P]),
    "bd_cache_append": (_I32, [_KV, _P, _P, _I32, _P, _I32, _P, _P]),
    "bd_cache_rollback": (_I32, [_P, _P, _P, _I32, _I32, _P, _P, _P]),
    "bd_top1_ce_workspace_bytes": (_SZ, [_I32, _I32]),
    "bd_top1_ce": (_I32, [_P, ctypes.c_int64, _P, ctypes.c_int64, _P, _I32, _I32, _P, _P, _P, _P, _SZ, _P]),
    "bd_sample_budgets": (_I32, [_P, _I32, _P, _P, _I32, _P, _P]),
    "bd_sparse_decode_attn_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32]),
    "bd_sparse_decode_attn": (_I32, [_KV, _P, _I32, _P, _I32, _P, _F32, _P, _P, _P, _SZ, _P]),
    "bd_multiview_attn_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, _I32, _I32, _I32, _I32]),
    "bd_multiview_attn": (_I32, [_KV, _P, _I32, _I32, _I32, _P, _I32, _P, _F32, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "bd_multiview_attn_bwd_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, _I32, _I32, _I32, _I32]),
    "bd_multiview_attn_bwd": (_I32, [_KV, _P, _I32, _I32, _I32, _P, _I32, _P, _F32, _P, _P, _P, _P, _P, _P,
                                     _P, _P, _P, _P, _SZ, _P]),
    "bd_verify_attn_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, _I32]),
    "bd_verify_attn": (_I32, [_KV, _P, _I32, _I32, _F32, _P, _P, _P, _SZ, _P]),
    "bd_verify_attn_noalloc": (_I32, [_KV, _P, _I32, _I32, _F32, _P, _P, _P]),
    "bd_accept_len_workspace_bytes": (_SZ, [_I32, _I32, _I32]),
    "bd_accept_len": (_I32, [_P, _I64, _P, _I32, _I32, _I32, _P, _P, _P, _P, _SZ, _P]),
}

_lib = None
_lib_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """The loaded libbd.so with argument types set.  Raises if it is not built."""
    global _lib
    with _lib_lock:
        if _lib is None:
            if not os.path.exists(library_path):
                raise BdError(BD_ERR_DEVICE, f"{library_path} is not built; run `python -m paper_2606_00144_amd.build`")
            handle = ctypes.CDLL(library_path)
            for name, (res, args) in _SIGNATURES.items():
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            _lib = handle
    return _lib


def _check(status: int) -> None:
    if status != BD_OK:
        raise BdError(status, lib().bd_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _scale(scale: Optional[float]) -> float:
    return 1.0 / math.sqrt(HEAD_DIM) if scale is None else float(scale)


def _require(cond: bool, msg: str) -> None:
    if not cond:
        raise BdError(BD_ERR_INVALID_ARG, msg)


def kv_desc(k: torch.Tensor, v: Optional[torch.Tensor], seq_lens: torch.Tensor,
            page_table: Optional[torch.Tensor] = None, max_seq_len: Optional[int] = None) -> KvDesc:
    """Describe a KV cache for the C ABI (tensors must outlive the call)."""
    _require(k.dtype == torch.bfloat16 and k.dim() == 4 and k.shape[3] == HEAD_DIM and k.stride(3) == 1,
             "k must be bf16 [*, Hkv, *, 128] with a contiguous last dimension")
    if v is not None:
        _require(v.dtype == torch.bfloat16 and v.shape == k.shape and v.stride() == k.stride(),
                 "v must match k in shape and strides")
    _require(seq_lens.dtype == torch.int32 and seq_lens.dim() == 1, "seq_lens must be int32 [S]")
    d = KvDesc()
    d.k, d.v = k.data_ptr(), (v.data_ptr() if v is not None else None)
    d.num_seqs = seq_lens.shape[0]
    d.num_kv_heads = k.shape[1]
    d.head_dim = k.shape[3]
    d.seq_lens = seq_lens.data_ptr()
    d.stride_head, d.stride_tok = k.stride(1), k.stride(2)
    if page_table is None:
        _require(k.shape[0] == seq_lens.shape[0], "contiguous k must be [S, Hkv, L, 128]")
        d.max_seq_len = k.shape[2] if max_seq_len is None else int(max_seq_len)
        d.stride_seq = k.stride(0)
    else:
        _require(page_table.dtype == torch.int32 and page_table.dim() == 2 and page_table.shape[0] == seq_lens.shape[0],
                 "page_table must be int32 [S, max_pages]")
        d.page_table = page_table.data_ptr()
        d.page_size = k.shape[2]
        d.max_pages_per_seq = page_table.shape[1]
        d.num_pages = k.shape[0]
        d.stride_page = k.stride(0)
        d.max_seq_len = page_table.shape[1] * k.shape[2] if max_seq_len is None else int(max_seq_len)
    return d


class Workspace:
    """Zero-initialised device scratch, reused across calls.

    Every completed call leaves the leading counter region at zero and writes
    its other scratch only past it, so reuse on one stream needs no clearing.
    One instance must not serve calls that overlap in time.
    """

    def __init__(self):
        self.buf: Optional[torch.Tensor] = None

    def get(self, nbytes: int, device) -> Optional[torch.Tensor]:
        if nbytes == 0:
            return None
        if self.buf is None or self.buf.numel() < nbytes + 256 or self.buf.device != torch.device(device):
            self.buf = torch.zeros(nbytes + 256, dtype=torch.uint8, device=device)
        return self.buf


_default_ws = {}


def _ws(op: str, nbytes: int, device, workspace: Optional[Workspace]):
    if workspace is None:
        key = (op, torch.device(device).index, _stream())
        workspace = _default_ws.setdefault(key, Workspace())
    buf = workspace.get(nbytes, device)
    if buf is None:
        return None, 0
    base = buf.data_ptr()
    aligned = (base + 255) & ~255
    return aligned, buf.numel() - (aligned - base)


# --------------------------------------------------------------------- operations

def bd_select_kv(k: torch.Tensor, q_win: torch.Tensor, seq_lens: torch.Tensor, budget: int, *,
                 pool_kernel: int = 7, scale: Optional[float] = None, lse_win: Optional[torch.Tensor] = None,
                 return_scores: bool = False, page_table: Optional[torch.Tensor] = None,
                 max_seq_len: Optional[int] = None, workspace: Optional[Workspace] = None, outputs=None):
    """Budgeted KV selection.  q_win: bf16 [S, W, Hq, 128].  Returns (idx [S,Hkv,B], nsel [S][, scores]).
    outputs: optional preallocated (idx, nsel[, scores])."""
    return _select("bd_select_kv", (pool_kernel,), budget, k, q_win, seq_lens, budget, scale, lse_win,
                   return_scores, page_table, max_seq_len, workspace, outputs)


def bd_select_kv_chunks(k: torch.Tensor, q_win: torch.Tensor, seq_lens: torch.Tensor, budget: int, *,
                        chunk: int = 8, budget_counts_window: bool = False, scale: Optional[float] = None,
                        lse_win: Optional[torch.Tensor] = None, return_scores: bool = False,
                        page_table: Optional[torch.Tensor] = None, max_seq_len: Optional[int] = None,
                        workspace: Optional[Workspace] = None, outputs=None):
    """Chunk-level selection (TopKChunks): the top floor(B/chunk) prefix chunks, then the window
    (budget_counts_window=True: floor((B-W)/chunk) chunks).  Returns (idx [S,Hkv,ld], nsel [S][, scores])
    with ld = B + W (or B); a head's unused idx slots hold -1."""
    W = q_win.shape[1]
    ld = budget if budget_counts_window else budget + W
    return _select("bd_select_kv_chunks", (chunk, int(bool(budget_counts_window))), ld, k, q_win, seq_lens, budget,
                   scale, lse_win, return_scores, page_table, max_seq_len, workspace, outputs)


def _out(given, shape, dtype, dev, what):
    """A caller-given output (checked) or a new one."""
    if given is None:
        return torch.empty(shape, dtype=dtype, device=dev)
    _require(given.dtype == dtype and tuple(given.shape) == tuple(shape) and given.is_contiguous(),
             f"{what} must be contiguous {dtype} {tuple(shape)}")
    return given


def _select(entry, mode_args, ld, k, q_win, seq_lens, budget, scale, lse_win, return_scores, page_table, max_seq_len,
            workspace, outputs=None):
    _require(q_win.dtype == torch.bfloat16 and q_win.dim() == 4 and q_win.is_contiguous(), "q_win must be contiguous bf16 [S,W,Hq,128]")
    kv = kv_desc(k, None, seq_lens, page_table, max_seq_len)
    S, W, Hq = q_win.shape[0], q_win.shape[1], q_win.shape[2]
    dev = q_win.device
    given = tuple(outputs) + (None,) * 3 if outputs is not None else (None,) * 3
    idx = _out(given[0], (S, kv.num_kv_heads, ld), torch.int32, dev, "idx")
    nsel = _out(given[1], (S,), torch.int32, dev, "nsel")
    scores = None
    if return_scores:
        scores = given[2] if given[2] is not None else torch.zeros((S, kv.num_kv_heads, kv.max_seq_len),
                                                                    dtype=torch.float32, device=dev)
        _require(scores.dtype == torch.float32 and tuple(scores.shape) == (S, kv.num_kv_heads, kv.max_seq_len)
                 and scores.is_contiguous(), "scores must be contiguous fp32 [S,Hkv,max_seq_len]")
    if lse_win is not None:
        _require(lse_win.dtype == torch.float32 and lse_win.is_contiguous() and lse_win.shape == (S, W, Hq), "lse_win must be fp32 [S,W,Hq]")
    L = lib()
    nb = L.bd_select_kv_workspace_bytes(S, kv.num_kv_heads, Hq, W, kv.max_seq_len)
    wp, wb = _ws("select", nb, dev, workspace)
    _check(getattr(L, entry)(ctypes.byref(kv), q_win.data_ptr(), Hq, W, budget, *mode_args, _scale(scale),
                             _ptr(lse_win), idx.data_ptr(), nsel.data_ptr(), _ptr(scores), wp, wb, _stream()))
    return (idx, nsel, scores) if return_scores else (idx, nsel)


def bd_sparse_decode_attn(k: torch.Tensor, v: torch.Tensor, q: torch.Tensor, idx: torch.Tensor, nsel: torch.Tensor,
                          seq_lens: torch.Tensor, *, scale: Optional[float] = None, return_lse: bool = False,
                          page_table: Optional[torch.Tensor] = None, max_seq_len: Optional[int] = None,
                          out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                          workspace: Optional[Workspace] = None):
    """Drafter decode attention over selected entries.  q: bf16 [S, Hq, 128]; idx int32 [S, Hkv, ld].
    out / lse: optional preallocated outputs."""
    _require(q.dtype == torch.bfloat16 and q.dim() == 3 and q.is_contiguous(), "q must be contiguous bf16 [S,Hq,128]")
    _require(idx.dtype == torch.int32 and idx.dim() == 3 and idx.is_contiguous(), "idx must be contiguous int32 [S,Hkv,ld]")
    _require(nsel.dtype == torch.int32 and nsel.is_contiguous(), "nsel must be int32 [S]")
    kv = kv_desc(k, v, seq_lens, page_table, max_seq_len)
    S, Hq = q.shape[0], q.shape[1]
    out = _out(out, q.shape, torch.bfloat16, q.device, "out")
    lse = _out(lse, (S, Hq), torch.float32, q.device, "lse") if return_lse else None
    L = lib()
    nb = L.bd_sparse_decode_attn_workspace_bytes(S, kv.num_kv_heads, Hq, idx.shape[2])
    wp, wb = _ws("decode", nb, q.device, workspace)
    _check(L.bd_sparse_decode_attn(ctypes.byref(kv), q.data_ptr(), Hq, idx.data_ptr(), idx.shape[2], nsel.data_ptr(),
                                   _scale(scale), out.data_ptr(), _ptr(lse), wp, wb, _stream()))
    return (out, lse) if return_lse else out


def bd_multiview_attn(k: torch.Tensor, v: torch.Tensor, q_blk: torch.Tensor, idx_views: Optional[torch.Tensor],
                      nsel_views: Optional[torch.Tensor], seq_lens: torch.Tensor, *, scale: Optional[float] = None,
                      full: bool = True, train: bool = False, page_table: Optional[torch.Tensor] = None,
                      max_seq_len: Optional[int] = None, workspace: Optional[Workspace] = None, outputs=None):
    """Block attention under views and the full cache.  q_blk: bf16 [S, C, Hq, 128]; idx_views int32 [V, S, Hkv, ld].

    Returns (out_views, out_full).  With train=True also the training outputs the backward takes:
    (out_views, out_full, out32_views, lse_views, out32_full, lse_full).  outputs: optional
    preallocated tensors in that order (None entries are allocated).
    """
    _require(q_blk.dtype == torch.bfloat16 and q_blk.dim() == 4 and q_blk.is_contiguous(), "q_blk must be contiguous bf16 [S,C,Hq,128]")
    kv = kv_desc(k, v, seq_lens, page_table, max_seq_len)
    S, C, Hq = q_blk.shape[0], q_blk.shape[1], q_blk.shape[2]
    V = 0 if idx_views is None else idx_views.shape[0]
    ld = 0 if idx_views is None else idx_views.shape[3]
    if V:
        _require(idx_views.dtype == torch.int32 and idx_views.is_contiguous(), "idx_views must be contiguous int32 [V,S,Hkv,ld]")
        _require(nsel_views is not None and nsel_views.dtype == torch.int32 and nsel_views.shape == (V, S), "nsel_views must be int32 [V,S]")
    dev = q_blk.device
    given = tuple(outputs) + (None,) * 6 if outputs is not None else (None,) * 6
    out_v = _out(given[0], (V, S, C, Hq, HEAD_DIM), torch.bfloat16, dev, "out_views") if V else None
    out_f = _out(given[1], (S, C, Hq, HEAD_DIM), torch.bfloat16, dev, "out_full") if full else None
    o32_v = _out(given[2], (V, S, C, Hq, HEAD_DIM), torch.float32, dev, "out32_views") if (V and train) else None
    lse_v = _out(given[3], (V, S, C, Hq), torch.float32, dev, "lse_views") if (V and train) else None
    o32_f = _out(given[4], (S, C, Hq, HEAD_DIM), torch.float32, dev, "out32_full") if (full and train) else None
    lse_f = _out(given[5], (S, C, Hq), torch.float32, dev, "lse_full") if (full and train) else None
    L = lib()
    nb = L.bd_multiview_attn_workspace_bytes(S, kv.num_kv_heads, Hq, C, V, ld, kv.max_seq_len, int(full))
    wp, wb = _ws("multiview", nb, dev, workspace)
    _check(L.bd_multiview_attn(ctypes.byref(kv), q_blk.data_ptr(), Hq, C, V, _ptr(idx_views), ld, _ptr(nsel_views),
                               _scale(scale), _ptr(out_v), _ptr(lse_v), _ptr(o32_v), _ptr(out_f), _ptr(lse_f),
                               _ptr(o32_f), wp, wb, _stream()))
    return (out_v, out_f, o32_v, lse_v, o32_f, lse_f) if train else (out_v, out_f)


def bd_multiview_attn_bwd(k: torch.Tensor, v: torch.Tensor, q_blk: torch.Tensor, idx_views: Optional[torch.Tensor],
                          nsel_views: Optional[torch.Tensor], seq_lens: torch.Tensor,
                          out32_views: Optional[torch.Tensor], lse_views: Optional[torch.Tensor],
                          dout_views: Optional[torch.Tensor], out32_full: Optional[torch.Tensor] = None,
                          lse_full: Optional[torch.Tensor] = None, dout_full: Optional[torch.Tensor] = None, *,
                          scale: Optional[float] = None, with_dkv: bool = True,
                          page_table: Optional[torch.Tensor] = None, max_seq_len: Optional[int] = None,
                          workspace: Optional[Workspace] = None, grads=None):
    """Gradients of bd_multiview_attn (grads: optional preallocated (dq, dk, dv)).  out32/lse are the forward's training outputs (train=True), dout
    the upstream gradients (bf16, shaped like the outputs).  Returns (dq [S,C,Hq,128], dk_blk, dv_blk [S,C,Hkv,128]) in fp32;
    dk_blk and dv_blk are None unless with_dkv."""
    _require(q_blk.dtype == torch.bfloat16 and q_blk.dim() == 4 and q_blk.is_contiguous(), "q_blk must be contiguous bf16 [S,C,Hq,128]")
    kv = kv_desc(k, v, seq_lens, page_table, max_seq_len)
    S, C, Hq = q_blk.shape[0], q_blk.shape[1], q_blk.shape[2]
    V = 0 if idx_views is None else idx_views.shape[0]
    ld = 0 if idx_views is None else idx_views.shape[3]
    if V:
        _require(idx_views.dtype == torch.int32 and idx_views.is_contiguous(), "idx_views must be contiguous int32 [V,S,Hkv,ld]")
        _require(nsel_views is not None and nsel_views.dtype == torch.int32 and nsel_views.shape == (V, S), "nsel_views must be int32 [V,S]")
        for t, shp, dt in ((out32_views, (V, S, C, Hq, HEAD_DIM), torch.float32), (dout_views, (V, S, C, Hq, HEAD_DIM), torch.bfloat16),
                           (lse_views, (V, S, C, Hq), torch.float32)):
            _require(t is not None and t.dtype == dt and tuple(t.shape) == shp and t.is_contiguous(),
                     f"view tensors must be contiguous {dt} {shp}")
    full = dout_full is not None
    if full:
        for t, shp, dt in ((out32_full, (S, C, Hq, HEAD_DIM), torch.float32), (dout_full, (S, C, Hq, HEAD_DIM), torch.bfloat16),
                           (lse_full, (S, C, Hq), torch.float32)):
            _require(t is not None and t.dtype == dt and tuple(t.shape) == shp and t.is_contiguous(),
                     f"full-branch tensors must be contiguous {dt} {shp}")
    dev = q_blk.device
    given = tuple(grads) + (None,) * 3 if grads is not None else (None,) * 3
    dq = _out(given[0], (S, C, Hq, HEAD_DIM), torch.float32, dev, "dq")
    dk = _out(given[1], (S, C, kv.num_kv_heads, HEAD_DIM), torch.float32, dev, "dk") if with_dkv else None
    dv = _out(given[2], (S, C, kv.num_kv_heads, HEAD_DIM), torch.float32, dev, "dv") if with_dkv else None
    L = lib()
    nb = L.bd_multiview_attn_bwd_workspace_bytes(S, kv.num_kv_heads, Hq, C, V, ld, kv.max_seq_len, int(full))
    wp, wb = _ws("multiview_bwd", nb, dev, workspace)
    _check(L.bd_multiview_attn_bwd(ctypes.byref(kv), q_blk.data_ptr(), Hq, C, V, _ptr(idx_views), ld,
                                   _ptr(nsel_views), _scale(scale), _ptr(out32_views), _ptr(lse_views),
                                   _ptr(dout_views), _ptr(out32_full), _ptr(lse_full), _ptr(dout_full),
                                   dq.data_ptr(), _ptr(dk), _ptr(dv), wp, wb, _stream()))
    return dq, dk, dv


def bd_verify_attn(k: torch.Tensor, v: torch.Tensor, q: torch.Tensor, seq_lens: torch.Tensor, *,
                   scale: Optional[float] = None, return_lse: bool = False, page_table: Optional[torch.Tensor] = None,
                   max_seq_len: Optional[int] = None, out: Optional[torch.Tensor] = None,
                   lse: Optional[torch.Tensor] = None, workspace: Optional[Workspace] = None):
    """Verifier attention at the gamma+1 draft positions.  q: bf16 [S, gamma+1, Hq, 128].
    out / lse: optional preallocated outputs."""
    _require(q.dtype == torch.bfloat16 and q.dim() == 4 and q.is_contiguous(), "q must be contiguous bf16 [S,gamma+1,Hq,128]")
    kv = kv_desc(k, v, seq_lens, page_table, max_seq_len)
    S, R, Hq = q.shape[0], q.shape[1], q.shape[2]
    gamma = R - 1
    out = _out(out, q.shape, torch.bfloat16, q.device, "out")
    lse = _out(lse, (S, R, Hq), torch.float32, q.device, "lse") if return_lse else None
    L = lib()
    nb = L.bd_verify_attn_workspace_bytes(S, kv.num_kv_heads, Hq, gamma, kv.max_seq_len)
    wp, wb = _ws("verify", nb, q.device, workspace)
    _check(L.bd_verify_attn(ctypes.byref(kv), q.data_ptr(), Hq, gamma, _scale(scale), out.data_ptr(), _ptr(lse),
                            wp, wb, _stream()))
    return (out, lse) if return_lse else out


def bd_verify_attn_noalloc(k: torch.Tensor, v: torch.Tensor, q: torch.Tensor, seq_lens: torch.Tensor, *,
                           out: torch.Tensor, lse: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                           page_table: Optional[torch.Tensor] = None, max_seq_len: Optional[int] = None) -> None:
    """bd_verify_attn into caller-given outputs (out bf16 [S, gamma+1, Hq, 128], lse fp32 [S, gamma+1, Hq] or
    None) with the library's fixed scratch: nothing is allocated, here or in the library."""
    _require(q.dtype == torch.bfloat16 and q.dim() == 4 and q.is_contiguous(), "q must be contiguous bf16 [S,gamma+1,Hq,128]")
    _require(out.dtype == torch.bfloat16 and out.shape == q.shape and out.is_contiguous(), "out must be shaped like q")
    if lse is not None:
        _require(lse.dtype == torch.float32 and lse.shape == q.shape[:3] and lse.is_contiguous(), "lse must be fp32 [S,gamma+1,Hq]")
    kv = kv_desc(k, v, seq_lens, page_table, max_seq_len)
    _check(lib().bd_verify_attn_noalloc(ctypes.byref(kv), q.data_ptr(), q.shape[2], q.shape[1] - 1, _scale(scale),
                                        out.data_ptr(), _ptr(lse), _stream()))


def bd_accept_len(logits: torch.Tensor, draft: torch.Tensor, *, return_argmax: bool = False,
                  workspace: Optional[Workspace] = None, outputs=None):
    """Greedy acceptance.  logits fp32 [S, gamma+1, V] (last dim contiguous); draft int32 [S, gamma]."""
    _require(logits.dtype == torch.float32 and logits.dim() == 3 and logits.stride(2) == 1
             and (logits.shape[0] == 1 or logits.stride(0) == logits.shape[1] * logits.stride(1)),
             "logits must be fp32 [S,gamma+1,V] with evenly spaced rows")
    S, R, V = logits.shape
    gamma = R - 1
    _require(draft.dtype == torch.int32 and draft.shape == (S, gamma) and draft.is_contiguous(), "draft must be int32 [S,gamma]")
    dev = logits.device
    if outputs is None:
        acc = torch.empty((S,), dtype=torch.int32, device=dev)
        bonus = torch.empty((S,), dtype=torch.int32, device=dev)
        am = torch.empty((S, R), dtype=torch.int32, device=dev) if return_argmax else None
    else:
        acc, bonus, am = outputs
    L = lib()
    nb = L.bd_accept_len_workspace_bytes(S, gamma, V)
    wp, wb = _ws("accept", nb, dev, workspace)
    _check(L.bd_accept_len(logits.data_ptr(), logits.stride(1), draft.data_ptr(), S, gamma, V, acc.data_ptr(),
                           bonus.data_ptr(), _ptr(am), wp, wb, _stream()))
    return (acc, bonus, am) if return_argmax else (acc, bonus)


def bd_cache_append(k: torch.Tensor, v: torch.Tensor, seq_lens: torch.Tensor, k_new: torch.Tensor,
                    v_new: torch.Tensor, *, idx: Optional[torch.Tensor] = None, nsel: Optional[torch.Tensor] = None,
                    page_table: Optional[torch.Tensor] = None, max_seq_len: Optional[int] = None) -> None:
    """Append rows in place: k_new, v_new bf16 [S, n, Hkv, 128] go to positions seq_lens[s] ..; seq_lens
    (and, with the sparse list idx [S, Hkv, ld] / nsel [S], the list) advance in place."""
    _require(k_new.dtype == torch.bfloat16 and k_new.dim() == 4 and k_new.is_contiguous() and k_new.shape == v_new.shape
             and v_new.is_contiguous() and v_new.dtype == torch.bfloat16, "k_new and v_new must be contiguous bf16 [S,n,Hkv,128]")
    _require(seq_lens.dtype == torch.int32 and seq_lens.is_contiguous(), "seq_lens must be int32 [S]")
    if idx is not None:
        _require(idx.dtype == torch.int32 and idx.dim() == 3 and idx.is_contiguous(), "idx must be contiguous int32 [S,Hkv,ld]")
        _require(nsel is not None and nsel.dtype == torch.int32 and nsel.is_contiguous(), "nsel must be int32 [S]")
    kv = kv_desc(k, v, seq_lens, page_table, max_seq_len)
    _require(k_new.shape[0] == kv.num_seqs and k_new.shape[2] == kv.num_kv_heads, "k_new must be [S,n,Hkv,128]")
    _check(lib().bd_cache_append(ctypes.byref(kv), k_new.data_ptr(), v_new.data_ptr(), k_new.shape[1], _ptr(idx),
                                 idx.shape[2] if idx is not None else 0, _ptr(nsel), _stream()))


def bd_cache_rollback(seq_lens: torch.Tensor, accept: torch.Tensor, spec: int, *,
                      nsel: Optional[torch.Tensor] = None, base_lens: Optional[torch.Tensor] = None,
                      base_nsel: Optional[torch.Tensor] = None) -> None:
    """Keep the accepted speculative rows in place: with base_lens (and base_nsel), the lengths before the
    speculative appends, seq_lens = min(seq_lens, base + accept); without, spec - accept is subtracted."""
    _require(seq_lens.dtype == torch.int32 and seq_lens.is_contiguous(), "seq_lens must be int32 [S]")
    _require(accept.dtype == torch.int32 and accept.shape == seq_lens.shape, "accept must be int32 [S]")
    for t, n in ((nsel, "nsel"), (base_lens, "base_lens"), (base_nsel, "base_nsel")):
        if t is not None:
            _require(t.dtype == torch.int32 and t.shape == seq_lens.shape and t.is_contiguous(), f"{n} must be int32 [S]")
    _check(lib().bd_cache_rollback(seq_lens.data_ptr(), _ptr(nsel), accept.data_ptr(), seq_lens.shape[0], int(spec),
                                   _ptr(base_lens), _ptr(base_nsel), _stream()))


def bd_top1_ce(student: torch.Tensor, *, teacher: Optional[torch.Tensor] = None, targets: Optional[torch.Tensor] = None,
               return_targets: bool = False, return_lse: bool = False, workspace: Optional[Workspace] = None):
    """Top-1 CE per row: student fp32 [R, V]; teacher fp32 [R, V] (targets = its argmax) or targets int32 [R]."""
    _require(student.dtype == torch.float32 and student.dim() == 2 and student.stride(1) == 1, "student must be fp32 [R,V]")
    R, V = student.shape
    if teacher is not None:
        _require(teacher.dtype == torch.float32 and teacher.shape == student.shape and teacher.stride(1) == 1,
                 "teacher must be fp32 [R,V]")
    if targets is not None:
        _require(targets.dtype == torch.int32 and targets.shape == (R,) and targets.is_contiguous(), "targets must be int32 [R]")
    dev = student.device
    loss = torch.empty((R,), dtype=torch.float32, device=dev)
    tgt = torch.empty((R,), dtype=torch.int32, device=dev) if return_targets else None
    lse = torch.empty((R,), dtype=torch.float32, device=dev) if return_lse else None
    L = lib()
    wp, wb = _ws("ce", L.bd_top1_ce_workspace_bytes(R, V), dev, workspace)
    _check(L.bd_top1_ce(student.data_ptr(), student.stride(0), _ptr(teacher), teacher.stride(0) if teacher is not None else 0,
                        _ptr(targets), R, V, loss.data_ptr(), _ptr(tgt), _ptr(lse), wp, wb, _stream()))
    out = [loss] + ([tgt] if return_targets else []) + ([lse] if return_lse else [])
    return out[0] if len(out) == 1 else tuple(out)


def bd_sample_budgets(u: torch.Tensor, budgets, weights) -> torch.Tensor:
    """B ~ Cat(budgets, weights) for every uniform draw in u (fp32 device tensor)."""
    _require(u.dtype == torch.float32 and u.is_contiguous(), "u must be contiguous fp32")
    n = len(budgets)
    _require(n == len(weights) and n >= 1, "budgets and weights must have the same length")
    b = (ctypes.c_int32 * n)(*[int(x) for x in budgets])
    w = (ctypes.c_float * n)(*[float(x) for x in weights])
    out = torch.empty(u.shape, dtype=torch.int32, device=u.device)
    _check(lib().bd_sample_budgets(u.data_ptr(), u.numel(), ctypes.cast(b, ctypes.c_void_p),
                                   ctypes.cast(w, ctypes.c_void_p), n, out.data_ptr(), _stream()))
    return out
