"""Thin ctypes binding of libcsr (include/csr.h).

Argument marshalling only: tensors are passed as raw device pointers, host
integers by value, and the stream is torch's current HIP stream.  Every step of
the computation runs in the library's HIP kernels.  The library must have been
built (``python -m paper_2605_07325_amd.build``); there is no fallback.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional

import torch

# CSR_LIBRARY points at an alternative build (A/B tuning); default: the in-tree library.
_LIB_PATH = os.environ.get("CSR_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcsr.so")

CSR_OK, CSR_E_INVAL, CSR_E_UNSUPPORTED, CSR_E_WORKSPACE, CSR_E_HIP = 0, 1, 2, 3, 4
CSR_F32, CSR_BF16 = 0, 1
CSR_APPEND = 1
CSR_ROPE_NONE, CSR_ROPE_NEOX, CSR_ROPE_INTERLEAVED = 0, 1, 2
CSR_KV_SAME, CSR_KV_FP8_E4M3 = 0, 1
CSR_NOALLOC_SCRATCH_BYTES = 64 << 20  # include/csr.h

# Every function include/csr.h declares.
EXPORTS = ("csr_kv_append", "csr_extend_workspace_size", "csr_extend_attention", "csr_prefill_workspace_size",
           "csr_extend_attention_noalloc", "csr_prefill", "csr_set_attention_events", "csr_set_workgroup_clock",
           "csr_set_plan_overrides",
           "csr_status_string", "csr_last_error")


class AttnDesc(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("rope_style", ctypes.c_int32), ("rope_dim", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("kv_dtype", ctypes.c_int32), ("k_scale", ctypes.c_float), ("v_scale", ctypes.c_float),
                ("q_scale", ctypes.c_float)]


class CsrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with `python -m paper_2605_07325_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        p, i32, u32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
        D = ctypes.POINTER(AttnDesc)
        L.csr_kv_append.argtypes = [D, i32, p, p, p, p, i32, p, i32, p, p, i32, p]
        L.csr_kv_append.restype = ctypes.c_int
        L.csr_extend_workspace_size.argtypes = [D, i32, i32, i32, i32]
        L.csr_extend_workspace_size.restype = sz
        L.csr_extend_attention.argtypes = [D, i32, p, p, p, p, p, i32, p, i32, p, p, i32, i32, i32, u32, p, p, p, sz, p]
        L.csr_extend_attention.restype = ctypes.c_int
        L.csr_extend_attention_noalloc.argtypes = [D, i32, p, p, p, p, p, i32, p, i32, p, p, i32, i32, i32, u32, p, p,
                                                   p]
        L.csr_extend_attention_noalloc.restype = ctypes.c_int
        L.csr_prefill_workspace_size.argtypes = [D, i32, i32, i32]
        L.csr_prefill_workspace_size.restype = sz
        L.csr_prefill.argtypes = [D, i32, p, p, p, p, p, i32, p, i32, p, i32, i32, p, p, p, sz, p]
        L.csr_prefill.restype = ctypes.c_int
        L.csr_set_attention_events.argtypes = [p, p]
        L.csr_set_attention_events.restype = ctypes.c_int
        L.csr_set_workgroup_clock.argtypes = [p, i32]
        L.csr_set_workgroup_clock.restype = ctypes.c_int
        L.csr_set_plan_overrides.argtypes = [i32, i32, i32]
        L.csr_set_plan_overrides.restype = ctypes.c_int
        L.csr_status_string.argtypes = [ctypes.c_int]
        L.csr_status_string.restype = ctypes.c_char_p
        L.csr_last_error.argtypes = []
        L.csr_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _status_name(st: int) -> str:
    try:
        return lib().csr_status_string(st).decode()
    except Exception:  # library not loadable: still report the number
        return f"status {st}"


def _check(st: int) -> None:
    if st != CSR_OK:
        raise CsrError(st, lib().csr_last_error().decode())


def set_attention_events(begin_event, end_event) -> None:
    """csr_set_attention_events: raw hipEvent_t handles (ints) or None to disable."""
    _check(lib().csr_set_attention_events(None if begin_event is None else ctypes.c_void_p(begin_event),
                                          None if end_event is None else ctypes.c_void_p(end_event)))


def set_workgroup_clock(stamps=None) -> None:
    """csr_set_workgroup_clock: an int64 device tensor of shape [capacity, 4], or None to disable."""
    if stamps is None:
        _check(lib().csr_set_workgroup_clock(None, 0))
        return
    if stamps.dtype != torch.int64 or stamps.dim() != 2 or stamps.shape[1] != 4 or not stamps.is_cuda \
            or not stamps.is_contiguous():
        raise ValueError("workgroup clock buffer: a contiguous int64 CUDA tensor of shape [capacity, 4]")
    _check(lib().csr_set_workgroup_clock(_ptr(stamps), int(stamps.shape[0])))


def workgroup_clock_table(stamps) -> "dict":
    """Decode a filled [capacity, 4] buffer (copied to the host) into arrays: start and end in
    microseconds from the first start, first / end key tile, sequence, split, kv head, XCD."""
    import numpy as np
    w = stamps.cpu().numpy().view(np.uint64)
    used = w[:, 1] > 0
    w = w[used]
    t0 = w[:, 0].min() if len(w) else 0
    return {"start_us": (w[:, 0] - t0).astype(np.float64) * 0.01, "end_us": (w[:, 1] - t0).astype(np.float64) * 0.01,
            "tb": (w[:, 2] >> np.uint64(32)).astype(np.int64), "te": (w[:, 2] & np.uint64(0xffffffff)).astype(np.int64),
            "seq": (w[:, 3] >> np.uint64(32)).astype(np.int64), "split": ((w[:, 3] >> np.uint64(16)) & np.uint64(0xffff)).astype(np.int64),
            "kv_head": ((w[:, 3] >> np.uint64(8)) & np.uint64(0xff)).astype(np.int64), "xcd": (w[:, 3] & np.uint64(0xff)).astype(np.int64)}


def set_plan_overrides(nsplit: int = 0, fixed_order: bool = False, dma_all_waves: bool = False) -> None:
    """csr_set_plan_overrides (testing and A/B measurement, this thread): all defaults restore the planner."""
    _check(lib().csr_set_plan_overrides(int(nsplit), int(bool(fixed_order)), int(bool(dma_all_waves))))


@contextlib.contextmanager
def plan_overrides(nsplit: int = 0, fixed_order: bool = False, dma_all_waves: bool = False):
    """Plan overrides for the calls inside the block; the planner's choice again afterwards."""
    set_plan_overrides(nsplit, fixed_order, dma_all_waves)
    try:
        yield
    finally:
        set_plan_overrides()


def make_desc(num_q_heads: int, num_kv_heads: int, head_dim: int, page_size: int = 16, dtype=torch.bfloat16,
              softmax_scale: float = 0.0, rope_style: int = CSR_ROPE_NONE, rope_dim: int = 0,
              rope_theta: float = 0.0, kv_dtype: int = CSR_KV_SAME, k_scale: float = 0.0,
              v_scale: float = 0.0, q_scale: float = 0.0) -> AttnDesc:
    """csr_attn_desc.  ``rope_style`` != CSR_ROPE_NONE makes the library rotate q
    and k_new at their absolute positions (``rope_dim`` dims, 0 = all; base
    ``rope_theta``); ``kv_dtype`` = CSR_KV_FP8_E4M3 keeps the cache as e4m3
    codes (uint8 pools) with dequantisation scales ``k_scale``, ``v_scale``;
    with it, ``q_scale`` > 0 selects fp8 score products (q quantised too)."""
    dt = {torch.bfloat16: CSR_BF16, torch.float32: CSR_F32}.get(dtype, dtype)
    return AttnDesc(num_q_heads, num_kv_heads, head_dim, page_size, softmax_scale, int(dt), int(rope_style),
                    int(rope_dim), float(rope_theta), int(kv_dtype), float(k_scale), float(v_scale),
                    float(q_scale))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _pages(desc: AttnDesc, pool: Optional[torch.Tensor]) -> int:
    """num_pages of a [num_pages][P][Hkv][d] pool, after checking that the tensor has exactly that
    layout: num_pages bounds every page id the kernels dereference, so a pool of another shape
    (say flattened to slots) must not reach the library."""
    if pool is None:
        return 0
    want = (desc.page_size, desc.num_kv_heads, desc.head_dim)
    if pool.dim() != 4 or tuple(pool.shape[1:]) != want:
        raise ValueError(f"pool must be [num_pages, {want[0]}, {want[1]}, {want[2]}], got {tuple(pool.shape)}")
    if desc.kv_dtype == CSR_KV_FP8_E4M3:
        dt = torch.uint8
    else:
        dt = torch.bfloat16 if desc.dtype == CSR_BF16 else torch.float32
    if pool.dtype != dt:
        raise ValueError(f"pool dtype {pool.dtype}, expected {dt}")
    if not pool.is_contiguous() or not pool.is_cuda:
        raise ValueError("pool must be a contiguous device tensor")
    return int(pool.shape[0])


def _pool_pages(desc: AttnDesc, k_pool: Optional[torch.Tensor], v_pool: Optional[torch.Tensor]) -> int:
    n = _pages(desc, k_pool)
    if (k_pool is None) != (v_pool is None) or _pages(desc, v_pool) != n:
        raise ValueError("k_pool and v_pool must both be given, with the same shape, or both be None")
    return n


def kv_append(desc: AttnDesc, k_new, v_new, k_pool, v_pool, block_table, bt_stride: int, cu_seqlens_q,
              cache_seqlens, stream=None) -> None:
    """csr_kv_append: copy chunk K/V rows to cache positions L_b + i."""
    batch = int(cu_seqlens_q.shape[0]) - 1
    _check(lib().csr_kv_append(ctypes.byref(desc), batch, _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool),
                               _pool_pages(desc, k_pool, v_pool), _ptr(block_table), bt_stride, _ptr(cu_seqlens_q), _ptr(cache_seqlens),
                               int(k_new.shape[0]), _stream(stream)))


def extend_workspace_size(desc: AttnDesc, batch: int, total_q: int, max_seqlen_q: int, max_cache_len: int) -> int:
    return int(lib().csr_extend_workspace_size(ctypes.byref(desc), batch, total_q, max_seqlen_q, max_cache_len))


def prefill_workspace_size(desc: AttnDesc, batch: int, total: int, max_seqlen: int) -> int:
    return int(lib().csr_prefill_workspace_size(ctypes.byref(desc), batch, total, max_seqlen))


def _workspace(nbytes: int, device, workspace):
    if nbytes == 0:
        return workspace
    if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return workspace


def extend_attention(desc: AttnDesc, q, k_new, v_new, k_pool, v_pool, block_table, bt_stride: int, cu_seqlens_q,
                     cache_seqlens, max_seqlen_q: int, max_cache_len: int, append: bool = False, out=None,
                     lse: Optional[torch.Tensor] = None, want_lse: bool = True, workspace=None, stream=None):
    """csr_extend_attention.  Returns ``(out, lse)``; buffers are allocated with
    torch when not supplied (lse only if ``want_lse``)."""
    batch = int(cu_seqlens_q.shape[0]) - 1
    total_q = int(q.shape[0])
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((total_q, desc.num_q_heads), dtype=torch.float32, device=q.device)
    ws_bytes = extend_workspace_size(desc, batch, total_q, max_seqlen_q, max_cache_len) if total_q else 0
    workspace = _workspace(ws_bytes, q.device, workspace)
    ws_cap = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().csr_extend_attention(
        ctypes.byref(desc), batch, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool), _pool_pages(desc, k_pool, v_pool),
        _ptr(block_table), bt_stride, _ptr(cu_seqlens_q), _ptr(cache_seqlens), total_q, max_seqlen_q, max_cache_len,
        CSR_APPEND if append else 0, _ptr(out), _ptr(lse), _ptr(workspace), ws_cap, _stream(stream)))
    return out, lse


def extend_attention_noalloc(desc: AttnDesc, q, k_new, v_new, k_pool, v_pool, block_table, bt_stride: int,
                             cu_seqlens_q, cache_seqlens, max_seqlen_q: int, max_cache_len: int, append: bool = False,
                             out=None, lse: Optional[torch.Tensor] = None, want_lse: bool = True, stream=None):
    """csr_extend_attention_noalloc: as ``extend_attention`` with the library's own scratch array as the
    workspace (the binding still allocates ``out`` / ``lse`` when they are not supplied)."""
    batch = int(cu_seqlens_q.shape[0]) - 1
    total_q = int(q.shape[0])
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((total_q, desc.num_q_heads), dtype=torch.float32, device=q.device)
    _check(lib().csr_extend_attention_noalloc(
        ctypes.byref(desc), batch, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool),
        _pool_pages(desc, k_pool, v_pool), _ptr(block_table), bt_stride, _ptr(cu_seqlens_q), _ptr(cache_seqlens), total_q,
        max_seqlen_q, max_cache_len, CSR_APPEND if append else 0, _ptr(out), _ptr(lse), _stream(stream)))
    return out, lse


def prefill(desc: AttnDesc, q, k, v, cu_seqlens, max_seqlen: int, k_pool=None, v_pool=None, block_table=None,
            bt_stride: int = 1, out=None, lse=None, want_lse: bool = True, workspace=None, stream=None):
    """csr_prefill (L = 0 re-prefill; optional warm-up write of the cache)."""
    batch = int(cu_seqlens.shape[0]) - 1
    total = int(q.shape[0])
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((total, desc.num_q_heads), dtype=torch.float32, device=q.device)
    ws_bytes = prefill_workspace_size(desc, batch, total, max_seqlen) if total else 0
    workspace = _workspace(ws_bytes, q.device, workspace)
    ws_cap = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().csr_prefill(
        ctypes.byref(desc), batch, _ptr(q), _ptr(k), _ptr(v), _ptr(k_pool), _ptr(v_pool), _pool_pages(desc, k_pool, v_pool),
        _ptr(block_table), bt_stride, _ptr(cu_seqlens), total, max_seqlen, _ptr(out), _ptr(lse), _ptr(workspace),
        ws_cap, _stream(stream)))
    return out, lse
