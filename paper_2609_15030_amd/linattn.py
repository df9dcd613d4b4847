"""Python binding of the C ABI in include/linattn.h.

Argument marshalling only: torch tensors become device pointers, NumPy
arrays become host pointers, the current torch stream becomes the hipStream_t.
Every step of the computation runs in the gfx950 library; if the library is
missing this module raises on import rather than falling back to anything.

Function names and argument order follow the C entry points.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblinattn.so")

LA_OK = 0
LA_ERR_INVALID_ARG = 1
LA_ERR_UNSUPPORTED = 2
LA_ERR_EMPTY_SUFFIX = 3
LA_ERR_MISALIGNED_STATE = 4
LA_ERR_HIP = 5
LA_ERR_WORKSPACE = 6

LA_F32 = 0
LA_BF16 = 1
LA_GDR_LITERAL = 0
LA_GDR_DECAYED_DELTA = 1

EXPORTED = ("strict_prefix_boundary", "la_prefill_workspace_bytes", "la_prefill",
            "la_prefill_resume", "la_checkpoint_rows", "la_prefill_form", "la_prefill_scan_columns",
            "la_prefill_paged", "la_prefill_paged_noalloc", "la_decode_step", "la_state_save_paged",
            "la_state_restore_paged",
            "la_state_save_host", "la_state_restore_host", "la_hybrid_boundary", "la_hybrid_restore",
            "la_status_string", "la_last_error_message", "la_trace_set_events")


class LaShape(ctypes.Structure):
    _fields_ = [("n_seqs", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("ckpt_interval", ctypes.c_int32),
                ("io_dtype", ctypes.c_int32), ("variant", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class LaPages(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("n_pages", ctypes.c_int64),
                ("ckpt_page_ids", ctypes.c_void_p), ("state_page_ids", ctypes.c_void_p),
                ("err_count", ctypes.c_void_p)]


class LaKvBlocks(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("n_pool_blocks", ctypes.c_int64),
                ("cache", ctypes.c_void_p), ("n_cache_blocks", ctypes.c_int64),
                ("block_bytes", ctypes.c_int64), ("block_tokens", ctypes.c_int64),
                ("src_ids", ctypes.c_void_p), ("dst_ids", ctypes.c_void_p), ("max_blocks", ctypes.c_int64)]


def make_shape(n_seqs, n_heads, dk, dv, ckpt_interval, io_dtype=LA_BF16,
               variant=LA_GDR_LITERAL, scale=1.0, chunk=64) -> LaShape:
    return LaShape(n_seqs, n_heads, dk, dv, chunk, ckpt_interval, io_dtype, variant, scale)


class LinAttnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_15030_amd.build` (hipcc, gfx950)")
    # The library must share one HIP runtime with torch (which owns device
    # memory and streams).  torch ships its own libamdhip64.so.7; loading
    # torch first makes the dynamic linker bind our dependency to that copy
    # instead of loading a second runtime from the ROCm install.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    SH = ctypes.POINTER(LaShape)
    sig = {
        "strict_prefix_boundary": ([I64, I64, I64, ctypes.POINTER(I64)], I32),
        "la_prefill_workspace_bytes": ([SH, I64], SZ),
        "la_prefill": ([SH, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
        "la_prefill_resume": ([SH, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
        "la_checkpoint_rows": ([I32, P, P, I64, P, ctypes.POINTER(I64)], I32),
        "la_prefill_form": ([SH], I32),
        "la_prefill_scan_columns": ([SH, P, ctypes.POINTER(I64)], I32),
        "la_prefill_paged": ([SH, ctypes.POINTER(LaPages), P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
        "la_prefill_paged_noalloc": ([SH, ctypes.POINTER(LaPages), P, P, P, P, P, P, P, P, P, P, P, P, P, P], I32),
        "la_decode_step": ([SH, P, P, P, P, P, P, P, P], I32),
        "la_state_save_paged": ([P, I64, I64, P, I64, P, P, P], I32),
        "la_state_restore_paged": ([P, I64, P, P, I64, I64, P, P], I32),
        "la_state_save_host": ([P, I64, I64, P, I64, P, P, P, P], I32),
        "la_state_restore_host": ([P, I64, P, P, I64, I64, P, P, P], I32),
        "la_hybrid_boundary": ([I64, I64, I64, I64, I64, ctypes.POINTER(I64), ctypes.POINTER(I64)], I32),
        "la_hybrid_restore": ([ctypes.POINTER(LaKvBlocks), I32, I32, I64, P, P, P, I64, P, P, P, P], I32),
        "la_status_string": ([I32], ctypes.c_char_p),
        "la_last_error_message": ([], ctypes.c_char_p),
        "la_trace_set_events": ([ctypes.POINTER(P), I32], None),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


_lib = _load()


def library() -> ctypes.CDLL:
    return _lib


def status_string(status: int) -> str:
    return _lib.la_status_string(status).decode()


def last_error_message() -> str:
    return _lib.la_last_error_message().decode()


def _check(status: int):
    if status != LA_OK:
        raise LinAttnError(status, last_error_message())


def _dptr(t) -> Optional[int]:
    """Device pointer of a torch tensor (None stays NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _hptr(a, dtype) -> Optional[ctypes.c_void_p]:
    """Host pointer of a NumPy array (converted to ``dtype``, kept alive by the caller)."""
    if a is None:
        return None
    assert a.dtype == dtype and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def strict_prefix_boundary(n_tokens: int, interval: int, available_tokens: int) -> int:
    out = ctypes.c_int64(-1)
    _check(_lib.strict_prefix_boundary(int(n_tokens), int(interval), int(available_tokens),
                                       ctypes.byref(out)))
    return out.value


def strict_prefix_boundary_status(n_tokens: int, interval: int, available_tokens: int):
    """(status, B) without raising; B is -1 when nothing was written."""
    out = ctypes.c_int64(-1)
    st = _lib.strict_prefix_boundary(int(n_tokens), int(interval), int(available_tokens),
                                     ctypes.byref(out))
    return st, out.value


def la_prefill_workspace_bytes(shape: LaShape, total_tokens: int) -> int:
    return _lib.la_prefill_workspace_bytes(ctypes.byref(shape), int(total_tokens))


def la_prefill(shape: LaShape, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host: np.ndarray,
               o, final_state=None, ckpt_out=None, ckpt_offsets_dev=None,
               ckpt_offsets_host: Optional[np.ndarray] = None, workspace=None, stream=None,
               check: bool = True) -> int:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.la_prefill(ctypes.byref(shape), _dptr(q), _dptr(k), _dptr(v), _dptr(g), _dptr(beta),
                         _dptr(cu_seqlens_dev), _hptr(cu_seqlens_host, np.int32), _dptr(o),
                         _dptr(final_state), _dptr(ckpt_out), _dptr(ckpt_offsets_dev),
                         _hptr(ckpt_offsets_host, np.int32), _dptr(workspace), ws_bytes,
                         _stream(stream))
    if check:
        _check(st)
    return st


def la_prefill_resume(shape: LaShape, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host: np.ndarray,
                      start_pos_dev, start_pos_host: np.ndarray, state_in, o, final_state=None,
                      ckpt_out=None, ckpt_offsets_dev=None,
                      ckpt_offsets_host: Optional[np.ndarray] = None, workspace=None, stream=None,
                      check: bool = True) -> int:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.la_prefill_resume(ctypes.byref(shape), _dptr(q), _dptr(k), _dptr(v), _dptr(g),
                                _dptr(beta), _dptr(cu_seqlens_dev), _hptr(cu_seqlens_host, np.int32),
                                _dptr(start_pos_dev), _hptr(start_pos_host, np.int64),
                                _dptr(state_in), _dptr(o), _dptr(final_state), _dptr(ckpt_out),
                                _dptr(ckpt_offsets_dev), _hptr(ckpt_offsets_host, np.int32),
                                _dptr(workspace), ws_bytes, _stream(stream))
    if check:
        _check(st)
    return st


def la_state_save_paged(states, pool, page_ids_dev, err_count_dev=None, stream=None,
                        check: bool = True) -> int:
    n_pages = pool.shape[0]
    page_elems = pool[0].numel() if n_pages else states[0].numel()
    n_items = page_ids_dev.numel()
    st = _lib.la_state_save_paged(_dptr(states), n_items, page_elems, _dptr(pool), n_pages,
                                  _dptr(page_ids_dev), _dptr(err_count_dev), _stream(stream))
    if check:
        _check(st)
    return st


def la_state_restore_paged(pool, page_ids_dev, states, err_count_dev=None, stream=None,
                           check: bool = True) -> int:
    n_pages = pool.shape[0]
    page_elems = pool[0].numel() if n_pages else states[0].numel()
    n_items = page_ids_dev.numel()
    st = _lib.la_state_restore_paged(_dptr(pool), n_pages, _dptr(page_ids_dev), _dptr(states),
                                     n_items, page_elems, _dptr(err_count_dev), _stream(stream))
    if check:
        _check(st)
    return st


LA_FORM_NONE, LA_FORM_FUSED_SCAN, LA_FORM_FUSED_TWO_LEVEL, LA_FORM_TILE_SCAN_OUT, LA_FORM_SPLIT_DK_SCAN = 0, 1, 2, 3, 4


def la_prefill_form(shape: LaShape) -> int:
    """Which kernels a prefill of this shape runs (LA_FORM_*)."""
    return _lib.la_prefill_form(ctypes.byref(shape))


def la_prefill_scan_columns(shape: LaShape, cu_seqlens_host):
    """(columns, narrow chains): the fused scan's workgroup width for a bf16
    call of this shape and these lengths (32, 64 or 128; 64 for a mix of 32
    and 64; 0 when it runs none) and how many chains, the longest, run at 32
    columns."""
    cu = np.ascontiguousarray(cu_seqlens_host, dtype=np.int32)
    narrow = ctypes.c_int64(0)
    w = _lib.la_prefill_scan_columns(ctypes.byref(shape), cu.ctypes.data, ctypes.byref(narrow))
    return w, int(narrow.value)


def la_checkpoint_rows(cu_seqlens_host, start_pos_host, interval: int):
    """Checkpoint row offsets per sequence and the total row count, as the
    library numbers them (start_pos_host None: a cold call)."""
    cu = np.ascontiguousarray(cu_seqlens_host, dtype=np.int32)
    n = len(cu) - 1
    sp = None if start_pos_host is None else np.ascontiguousarray(start_pos_host, dtype=np.int64)
    offs = np.zeros(max(n, 0), np.int32)
    total = ctypes.c_int64(-1)
    _check(_lib.la_checkpoint_rows(n, _hptr(cu, np.int32), _hptr(sp, np.int64), int(interval),
                                   _hptr(offs, np.int32), ctypes.byref(total)))
    return offs, total.value


def make_pages(pool, ckpt_page_ids=None, state_page_ids=None, err_count=None, n_pages=None) -> LaPages:
    """la_pages for a device pool ([n_pages, dk * dv] fp32) and device int32 page tables."""
    n = pool.shape[0] if n_pages is None else n_pages
    pages = LaPages(_dptr(pool), int(n), _dptr(ckpt_page_ids), _dptr(state_page_ids), _dptr(err_count))
    pages._keep = (pool, ckpt_page_ids, state_page_ids, err_count)   # the struct holds raw addresses only
    return pages


def la_prefill_paged(shape: LaShape, pages: Optional[LaPages], q, k, v, g, beta, cu_dev, cu_host, start_dev,
                     start_host, o, final_state, ckpt_off_dev, ckpt_off_host, workspace, stream=None,
                     check: bool = True) -> int:
    """A prefill whose checkpoints go to pool pages and whose starting states
    come from pool pages; start_dev / start_host None make it a cold call."""
    cu_host = np.ascontiguousarray(cu_host, dtype=np.int32)
    sh = None if start_host is None else np.ascontiguousarray(start_host, dtype=np.int64)
    oh = None if ckpt_off_host is None else np.ascontiguousarray(ckpt_off_host, dtype=np.int32)
    st = _lib.la_prefill_paged(ctypes.byref(shape), None if pages is None else ctypes.byref(pages), _dptr(q),
                               _dptr(k), _dptr(v), _dptr(g), _dptr(beta), _dptr(cu_dev), _hptr(cu_host, np.int32),
                               _dptr(start_dev), _hptr(sh, np.int64), _dptr(o), _dptr(final_state),
                               _dptr(ckpt_off_dev), _hptr(oh, np.int32), _dptr(workspace),
                               workspace.numel() * workspace.element_size(), _stream(stream))
    if check:
        _check(st)
    return st


def la_prefill_paged_noalloc(shape: LaShape, pages: Optional[LaPages], q, k, v, g, beta, cu_dev, cu_host, start_dev,
                             start_host, o, final_state, ckpt_off_dev, ckpt_off_host, stream=None,
                             check: bool = True) -> int:
    """la_prefill_paged on the library's static workspace (no allocation)."""
    cu_host = np.ascontiguousarray(cu_host, dtype=np.int32)
    sh = None if start_host is None else np.ascontiguousarray(start_host, dtype=np.int64)
    oh = None if ckpt_off_host is None else np.ascontiguousarray(ckpt_off_host, dtype=np.int32)
    st = _lib.la_prefill_paged_noalloc(ctypes.byref(shape), None if pages is None else ctypes.byref(pages),
                                       _dptr(q), _dptr(k), _dptr(v), _dptr(g), _dptr(beta), _dptr(cu_dev),
                                       _hptr(cu_host, np.int32), _dptr(start_dev), _hptr(sh, np.int64), _dptr(o),
                                       _dptr(final_state), _dptr(ckpt_off_dev), _hptr(oh, np.int32),
                                       _stream(stream))
    if check:
        _check(st)
    return st


def la_decode_step(shape: LaShape, q, k, v, g, beta, state, o, stream=None, check: bool = True) -> int:
    """One decode token per (sequence, head): state [n_seqs, H, dk, dv] fp32 is
    updated in place, o [n_seqs, H, dv] receives the output."""
    st = _lib.la_decode_step(ctypes.byref(shape), _dptr(q), _dptr(k), _dptr(v), _dptr(g), _dptr(beta),
                             _dptr(state), _dptr(o), _stream(stream))
    if check:
        _check(st)
    return st


def _hostptr(t) -> int:
    """Address of a pinned host tensor (the library checks it is device-mapped)."""
    if t.is_cuda:
        raise ValueError("expected a host tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def la_state_save_host(states, host_pool, page_ids_dev, err_count_dev=None, stream=None, done_event=None,
                       check: bool = True) -> int:
    """Scatter device states into a pinned host pool ([n_pages, page_elems] fp32)."""
    n_pages = host_pool.shape[0]
    page_elems = host_pool[0].numel() if n_pages else states[0].numel()
    n_items = page_ids_dev.numel()
    st = _lib.la_state_save_host(_dptr(states), n_items, page_elems, _hostptr(host_pool), n_pages,
                                 _dptr(page_ids_dev), _dptr(err_count_dev), _stream(stream), done_event)
    if check:
        _check(st)
    return st


def la_state_restore_host(host_pool, page_ids_dev, states, err_count_dev=None, stream=None, done_event=None,
                          check: bool = True) -> int:
    """Gather pages of a pinned host pool into device states."""
    n_pages = host_pool.shape[0]
    page_elems = host_pool[0].numel() if n_pages else states[0].numel()
    n_items = page_ids_dev.numel()
    st = _lib.la_state_restore_host(_hostptr(host_pool), n_pages, _dptr(page_ids_dev), _dptr(states), n_items,
                                    page_elems, _dptr(err_count_dev), _stream(stream), done_event)
    if check:
        _check(st)
    return st


def la_hybrid_boundary(n_tokens: int, interval: int, kv_block_tokens: int, kv_cached_tokens: int,
                       state_cached_tokens: int):
    """(B, KV blocks covering [0, B)) for a hybrid cache."""
    b, nb = ctypes.c_int64(-1), ctypes.c_int64(-1)
    _check(_lib.la_hybrid_boundary(int(n_tokens), int(interval), int(kv_block_tokens), int(kv_cached_tokens),
                                   int(state_cached_tokens), ctypes.byref(b), ctypes.byref(nb)))
    return b.value, nb.value


def _anyptr(t) -> Optional[int]:
    """Address of a device tensor or of a pinned host tensor (the library checks which)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def make_kv_blocks(pool, cache, src_ids, dst_ids, block_tokens: int) -> LaKvBlocks:
    """la_kv_blocks for byte pools [n_blocks, block_bytes] (uint8 tensors; the pool
    may be pinned host memory) and device int32 tables [n_seqs, max_blocks]."""
    kv = LaKvBlocks(_anyptr(pool), int(pool.shape[0]), _dptr(cache), int(cache.shape[0]),
                    int(cache.shape[1] if cache.dim() > 1 else pool.shape[1]), int(block_tokens),
                    _dptr(src_ids), _dptr(dst_ids), int(src_ids.shape[1]))
    kv._keep = (pool, cache, src_ids, dst_ids)     # the struct holds raw addresses only
    return kv


def la_hybrid_restore(kv: LaKvBlocks, boundary_dev, boundary_host, state_pool, state_page_ids_dev, states,
                      n_heads: int, err_count_dev=None, stream=None, check: bool = True) -> int:
    """Joint restore: KV blocks of every prefix [0, B_i) and the state pages of the
    checkpoint at B_i.  states: [n_seqs * n_heads, page_elems] device fp32."""
    bh = np.ascontiguousarray(boundary_host, dtype=np.int64)
    n_seqs = len(bh)
    page_elems = states.shape[-1] if states is not None else 0
    n_state_pages = state_pool.shape[0] if state_pool is not None else 0
    st = _lib.la_hybrid_restore(ctypes.byref(kv), n_seqs, int(n_heads), int(page_elems), _dptr(boundary_dev),
                                _hptr(bh, np.int64), _anyptr(state_pool), int(n_state_pages),
                                _dptr(state_page_ids_dev), _dptr(states), _dptr(err_count_dev), _stream(stream))
    if check:
        _check(st)
    return st


def la_trace_set_events(events: Sequence[int]):
    """events: hipEvent_t handles (ints); an empty sequence switches tracing off."""
    if not events:
        _lib.la_trace_set_events(None, 0)
        return
    arr = (ctypes.c_void_p * len(events))(*events)
    _lib.la_trace_set_events(arr, len(events))
