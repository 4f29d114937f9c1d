"""Python binding of ``libkvt.so`` (argument marshalling only).

Every step of append and extend attention runs in the library's HIP
kernels; this module turns torch tensors into the C structs of
``include/kvt.h``, passes torch's current HIP stream, and raises on a
non-OK status.  torch supplies device memory and streams, nothing else.
There is no fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvt.so")

KVT_OK = 0
KVT_ERR_INVALID_ARG = 1
KVT_ERR_UNSUPPORTED = 2
KVT_ERR_OUT_OF_RANGE = 3
KVT_ERR_WORKSPACE = 4
KVT_ERR_DEVICE = 5
KVT_ERR_SCRATCH_LIMIT = 6
NOALLOC_SCRATCH_BYTES = 64 << 20    # KVT_NOALLOC_SCRATCH_BYTES
KVT_DTYPE_BF16 = 0
KVT_DTYPE_F32 = 1
BLOCK_SIZE = 16

MGR_EXPORTED = ("kvt_mgr_append", "kvt_mgr_begin_request", "kvt_mgr_create", "kvt_mgr_destroy", "kvt_mgr_end_request",
                "kvt_mgr_entry_tier", "kvt_mgr_fork", "kvt_mgr_free_pages", "kvt_mgr_live_entries",
                "kvt_mgr_message_pages", "kvt_mgr_message_state", "kvt_mgr_one_off", "kvt_mgr_pin",
                "kvt_mgr_prefill_done", "kvt_mgr_remove", "kvt_mgr_replace", "kvt_mgr_replay", "kvt_mgr_spawn",
                "kvt_mgr_start_prefill", "kvt_mgr_terminate", "kvt_mgr_unpin")
MGR_OPS = ("spawn", "fork", "append", "one_off", "pin", "unpin", "replace", "remove", "terminate", "begin_request",
           "start_prefill", "prefill_done", "end_request")   # KVT_MGR_OP_* in this order
EXPORTED = ("kvt_append_kv", "kvt_cascade_extend_attention", "kvt_cascade_extend_attention_ex",
            "kvt_cascade_uses_shared_pass", "kvt_cascade_workspace_bytes", "kvt_cascade_workspace_bytes_ex",
            "kvt_copy_blocks",
            "kvt_decode_attention", "kvt_decode_workspace_bytes", "kvt_extend_attention",
            "kvt_extend_attention_noalloc", "kvt_extend_workspace_bytes", "kvt_last_hip_error",
            "kvt_status_str") + MGR_EXPORTED
CASCADE_AUTO, CASCADE_SHARED_PASS, CASCADE_PLAIN = 0, 1, 2    # kvt_cascade_mode
KVT_COPY_TO_HOST = 0
KVT_COPY_TO_DEVICE = 1
KVT_PINNED, KVT_ACTIVE, KVT_SUSPENDED, KVT_EXPIRED, KVT_TEMPORARY = 0, 1, 2, 3, 4
KVT_TIER_PINNED, KVT_TIER_ACTIVE, KVT_TIER_SUSPENDED, KVT_TIER_DISCARDED = 0, 1, 2, 3


class KvtPool(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("num_blocks", ctypes.c_int64),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class KvtSeqs(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("prefix_len", ctypes.POINTER(ctypes.c_int32)),
                ("suffix_len", ctypes.POINTER(ctypes.c_int32)), ("block_table", ctypes.c_void_p),
                ("block_table_host", ctypes.POINTER(ctypes.c_int32)), ("max_blocks", ctypes.c_int32)]


class KvtMgrReport(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("admitted_entries", "admitted_pages", "bypassed_entries",
                                               "rejected_entries", "released_entries", "released_pages",
                                               "hit_tokens", "miss_tokens")]

    def as_dict(self) -> dict:
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


class KvtError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_str(status)} (status {status}"
                         + (f", hipError {lib().kvt_last_hip_error()}" if status == KVT_ERR_DEVICE else "") + ")")


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_39819_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.kvt_append_kv.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.kvt_append_kv.restype = ctypes.c_int
        L.kvt_extend_attention.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_void_p, ctypes.c_int32, ctypes.c_float,
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                           ctypes.c_void_p]
        L.kvt_extend_attention.restype = ctypes.c_int
        L.kvt_extend_attention_noalloc.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_void_p, ctypes.c_int32,
                                                   ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.kvt_extend_attention_noalloc.restype = ctypes.c_int
        L.kvt_extend_workspace_bytes.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_int32]
        L.kvt_extend_workspace_bytes.restype = ctypes.c_size_t
        L.kvt_cascade_extend_attention.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_int32, ctypes.c_void_p,
                                                   ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.kvt_cascade_extend_attention.restype = ctypes.c_int
        L.kvt_cascade_workspace_bytes.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_int32, ctypes.c_int32]
        L.kvt_cascade_workspace_bytes.restype = ctypes.c_size_t
        L.kvt_cascade_uses_shared_pass.argtypes = L.kvt_cascade_workspace_bytes.argtypes
        L.kvt_cascade_uses_shared_pass.restype = ctypes.c_int32
        L.kvt_cascade_extend_attention_ex.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_int32, ctypes.c_int32,
                                                      ctypes.c_void_p, ctypes.c_int32, ctypes.c_float,
                                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                      ctypes.c_size_t, ctypes.c_void_p]
        L.kvt_cascade_extend_attention_ex.restype = ctypes.c_int
        L.kvt_cascade_workspace_bytes_ex.argtypes = [P(KvtPool), P(KvtSeqs), ctypes.c_int32, ctypes.c_int32,
                                                     ctypes.c_int32]
        L.kvt_cascade_workspace_bytes_ex.restype = ctypes.c_size_t
        L.kvt_copy_blocks.argtypes = [P(KvtPool), ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_int64,
                                      ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        L.kvt_copy_blocks.restype = ctypes.c_int
        L.kvt_decode_attention.argtypes = L.kvt_extend_attention.argtypes
        L.kvt_decode_attention.restype = ctypes.c_int
        L.kvt_decode_workspace_bytes.argtypes = L.kvt_extend_workspace_bytes.argtypes
        L.kvt_decode_workspace_bytes.restype = ctypes.c_size_t
        M, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        L.kvt_mgr_create.argtypes, L.kvt_mgr_create.restype = [I64], M
        L.kvt_mgr_destroy.argtypes, L.kvt_mgr_destroy.restype = [M], None
        for name in ("kvt_mgr_free_pages", "kvt_mgr_live_entries"):
            getattr(L, name).argtypes, getattr(L, name).restype = [M], I64
        for name, args in (("kvt_mgr_spawn", [I64]), ("kvt_mgr_fork", [I64, I64]), ("kvt_mgr_append", [I64, I64]),
                           ("kvt_mgr_one_off", [I64]), ("kvt_mgr_pin", [I64, I64]), ("kvt_mgr_unpin", [I64, I64]),
                           ("kvt_mgr_replace", [I64, I64, I64]), ("kvt_mgr_remove", [I64, I64]),
                           ("kvt_mgr_terminate", [I64]), ("kvt_mgr_begin_request", [I64]),
                           ("kvt_mgr_start_prefill", [I64, P(KvtMgrReport)]),
                           ("kvt_mgr_prefill_done", [I64, P(KvtMgrReport)]), ("kvt_mgr_end_request", [I64])):
            getattr(L, name).argtypes, getattr(L, name).restype = [M] + args, ctypes.c_int
        for name in ("kvt_mgr_message_state", "kvt_mgr_entry_tier"):
            getattr(L, name).argtypes, getattr(L, name).restype = [M, I64, I64], I32
        L.kvt_mgr_replay.argtypes, L.kvt_mgr_replay.restype = [M, P(I64), I64, P(KvtMgrReport)], I64
        L.kvt_mgr_message_pages.argtypes = [M, I64, I64, P(I32), I64]
        L.kvt_mgr_message_pages.restype = I64
        L.kvt_status_str.argtypes = [ctypes.c_int]
        L.kvt_status_str.restype = ctypes.c_char_p
        L.kvt_last_hip_error.argtypes = []
        L.kvt_last_hip_error.restype = ctypes.c_int
        _lib = L
    return _lib


def status_str(s: int) -> str:
    return lib().kvt_status_str(int(s)).decode()


# ---------------------------------------------------------------------------
# raw structs (plain integers as pointers)
# ---------------------------------------------------------------------------

_I32_MIN, _I32_MAX = -(1 << 31), (1 << 31) - 1


def _i32_array(x) -> ctypes.Array:
    # short lists of Python ints (the common case: a few sequence lengths)
    # skip numpy's per-call overhead, and so do short 1-D integer arrays
    # (turned into such a list first); anything else goes through numpy,
    # which rejects values outside int32 instead of wrapping them
    if type(x) is np.ndarray and x.ndim == 1 and x.dtype.kind in "iu" and x.size <= 64:
        x = x.tolist()
    if type(x) in (list, tuple) and len(x) <= 64 and all(type(e) is int and _I32_MIN <= e <= _I32_MAX for e in x):
        return (ctypes.c_int32 * len(x))(*x)
    a = np.asarray(x)
    if a.dtype.kind not in "iu":
        a = np.asarray(x, dtype=np.int64)          # raises on ints beyond int64
    a = a.reshape(-1)
    if a.size and (int(a.min()) < _I32_MIN or int(a.max()) > _I32_MAX):
        raise OverflowError("length or block id outside the int32 range")
    a = np.ascontiguousarray(a.astype(np.int32))
    return (ctypes.c_int32 * a.size).from_buffer_copy(a)


def raw_pool(k: int, v: int, num_blocks: int, num_kv_heads: int, head_dim: int, dtype: int) -> KvtPool:
    return KvtPool(k, v, num_blocks, num_kv_heads, head_dim, dtype)


class RawSeqs:
    """kvt_seqs plus the host arrays it points at (kept alive with it)."""

    def __init__(self, prefix_len, suffix_len, block_table_ptr: int, max_blocks: int, block_table_host=None):
        self.prefix = _i32_array(prefix_len)
        self.suffix = _i32_array(suffix_len)
        self.host = _i32_array(block_table_host) if block_table_host is not None else None
        self.struct = KvtSeqs(len(self.prefix), self.prefix, self.suffix, block_table_ptr,
                              self.host if self.host is not None else None, max_blocks)


# ---------------------------------------------------------------------------
# torch-facing calls
# ---------------------------------------------------------------------------

def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return KVT_DTYPE_BF16
    if t.dtype == torch.float32:
        return KVT_DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream_handle(device, stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def _pool_struct(k_pool, v_pool) -> KvtPool:
    if k_pool.shape != v_pool.shape or k_pool.dtype != v_pool.dtype or k_pool.dim() != 4:
        raise ValueError("k_pool and v_pool must both be [num_blocks][num_kv_heads][16][head_dim] of one dtype")
    if k_pool.shape[2] != BLOCK_SIZE:
        raise ValueError("page size must be 16")
    if not (k_pool.is_contiguous() and v_pool.is_contiguous()):
        raise ValueError("pools must be contiguous")
    nb, hkv, _, d = k_pool.shape
    return KvtPool(k_pool.data_ptr(), v_pool.data_ptr(), nb, hkv, d, _dtype_code(k_pool))


def _seqs(prefix_len, suffix_len, block_table, checked: bool) -> RawSeqs:
    import torch
    if block_table.dtype != torch.int32 or block_table.dim() != 2 or not block_table.is_contiguous():
        raise ValueError("block_table must be a contiguous int32 [num_seqs][max_blocks] device tensor")
    host = block_table.cpu().numpy() if checked else None
    return RawSeqs(prefix_len, suffix_len, block_table.data_ptr(), block_table.shape[1], host)


def _check_tokens(t, name, rows, heads, d, dtype):
    if t.dtype != dtype or tuple(t.shape) != (rows, heads, d) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous [{rows}][{heads}][{d}] {dtype} tensor, got {tuple(t.shape)} {t.dtype}")


def append_kv(k_pool, v_pool, block_table, prefix_len: Sequence[int], suffix_len: Sequence[int], k_new, v_new,
              *, stream=None, checked: bool = False) -> None:
    """Scatter the new tokens' K/V into their pages (``kvt_append_kv``)."""
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, suffix_len, block_table, checked)
    T = sum(seqs.suffix)
    _check_tokens(k_new, "k_new", T, pool.num_kv_heads, pool.head_dim, k_pool.dtype)
    _check_tokens(v_new, "v_new", T, pool.num_kv_heads, pool.head_dim, k_pool.dtype)
    st = lib().kvt_append_kv(ctypes.byref(pool), ctypes.byref(seqs.struct), k_new.data_ptr(), v_new.data_ptr(),
                             _stream_handle(k_pool.device, stream))
    if st != KVT_OK:
        raise KvtError(st, "kvt_append_kv")


def extend_workspace_bytes(k_pool, v_pool, block_table, prefix_len, suffix_len, num_q_heads: int) -> int:
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, suffix_len, block_table, False)
    return int(lib().kvt_extend_workspace_bytes(ctypes.byref(pool), ctypes.byref(seqs.struct), int(num_q_heads)))


def extend_attention(q, k_pool, v_pool, block_table, prefix_len: Sequence[int], suffix_len: Sequence[int],
                     scale: Optional[float] = None, *, out=None, lse=None, return_lse: bool = False,
                     workspace=None, use_workspace: bool = True, stream=None, checked: bool = False):
    """Causal attention of the new tokens over prefix + suffix (``kvt_extend_attention``).

    Returns ``out`` ([T][Hq][D], pool dtype), or ``(out, lse)`` when an lse
    buffer is given or ``return_lse`` is set.  ``workspace``: a byte tensor
    of at least ``extend_workspace_bytes`` (allocated here when
    ``use_workspace`` and none is given).
    """
    return _attention("kvt_extend_attention", "kvt_extend_workspace_bytes", q, k_pool, v_pool, block_table,
                      prefix_len, suffix_len, scale, out, lse, return_lse, workspace, use_workspace, stream, checked)


def extend_attention_noalloc(q, k_pool, v_pool, block_table, prefix_len: Sequence[int], suffix_len: Sequence[int],
                             scale: Optional[float] = None, *, out, lse=None, stream=None, checked: bool = False):
    """``kvt_extend_attention_noalloc``: the extend call with its split partials
    in the library's static scratch; ``out`` (and ``lse`` if wanted) are the
    caller's, so neither this function nor the library allocates device memory.
    Raises ``KvtError`` (KVT_ERR_SCRATCH_LIMIT) when the split plan needs more
    than ``NOALLOC_SCRATCH_BYTES``."""
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, suffix_len, block_table, checked)
    T = sum(seqs.suffix)
    Hq = int(q.shape[1])
    _check_tokens(q, "q", T, Hq, pool.head_dim, k_pool.dtype)
    _check_tokens(out, "out", T, Hq, pool.head_dim, k_pool.dtype)
    if lse is not None and (str(lse.dtype) != "torch.float32" or tuple(lse.shape) != (T, Hq)
                            or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [T][Hq] tensor")
    if scale is None:
        scale = 1.0 / math.sqrt(pool.head_dim)
    st = lib().kvt_extend_attention_noalloc(ctypes.byref(pool), ctypes.byref(seqs.struct), q.data_ptr(), Hq,
                                            float(scale), out.data_ptr(),
                                            lse.data_ptr() if lse is not None else None,
                                            _stream_handle(q.device, stream))
    if st != KVT_OK:
        raise KvtError(st, "kvt_extend_attention_noalloc")
    return out if lse is None else (out, lse)


def cascade_workspace_bytes(k_pool, v_pool, block_table, prefix_len, suffix_len, shared_len: int,
                            num_q_heads: int, mode: int = CASCADE_AUTO) -> int:
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, suffix_len, block_table, False)
    return int(lib().kvt_cascade_workspace_bytes_ex(ctypes.byref(pool), ctypes.byref(seqs.struct), int(shared_len),
                                                    int(mode), int(num_q_heads)))


def cascade_uses_shared_pass(k_pool, v_pool, block_table, prefix_len, suffix_len, shared_len: int,
                             num_q_heads: int) -> bool:
    """Whether ``cascade_extend_attention`` (with a workspace) runs the shared
    pass or the plain extend plan (``kvt_cascade_uses_shared_pass``)."""
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, suffix_len, block_table, False)
    r = int(lib().kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(seqs.struct), int(shared_len),
                                               int(num_q_heads)))
    if r < 0:
        raise ValueError("invalid cascade arguments")
    return r == 1


def cascade_extend_attention(q, k_pool, v_pool, block_table, prefix_len, suffix_len, shared_len: int,
                             scale: Optional[float] = None, *, out=None, lse=None, return_lse: bool = False,
                             workspace=None, use_workspace: bool = True, stream=None, checked: bool = False,
                             mode: int = CASCADE_AUTO):
    """Extend attention for sequences that share their first ``shared_len``
    positions (``kvt_cascade_extend_attention_ex``); same result as
    ``extend_attention``.  ``mode``: CASCADE_AUTO (the library's estimate
    picks the shared pass or the plain plan), CASCADE_SHARED_PASS, CASCADE_PLAIN."""
    return _attention("kvt_cascade_extend_attention_ex", "kvt_cascade_workspace_bytes_ex", q, k_pool, v_pool,
                      block_table, prefix_len, suffix_len, scale, out, lse, return_lse, workspace, use_workspace,
                      stream, checked, shared=(int(shared_len), int(mode)))


def copy_blocks(k_pool, v_pool, block_ids, host, to_host: bool, *, stream=None, checked: bool = False):
    """Pages ``block_ids`` (device int32) of the pools to (``to_host``) or from a
    pinned host tensor [n][2][Hkv][16][D] of the pool dtype (``kvt_copy_blocks``)."""
    import torch
    pool = _pool_struct(k_pool, v_pool)
    if block_ids.dtype != torch.int32 or not block_ids.is_cuda or not block_ids.is_contiguous():
        raise ValueError("block_ids must be a contiguous int32 device tensor")
    n = int(block_ids.numel())
    want = (n, 2) + tuple(k_pool.shape[1:])
    if tuple(host.shape) != want or host.dtype != k_pool.dtype or not host.is_contiguous():
        raise ValueError(f"host must be a contiguous {k_pool.dtype} tensor of shape {want}")
    if n and not host.is_pinned():
        raise ValueError("host must be pinned memory")
    ids_host = None
    if checked:
        ids_np = np.ascontiguousarray(block_ids.cpu().numpy(), dtype=np.int32)
        ids_host = ids_np.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    st = lib().kvt_copy_blocks(ctypes.byref(pool), block_ids.data_ptr() if n else None, ids_host, n,
                               host.data_ptr() if n else None,
                               KVT_COPY_TO_HOST if to_host else KVT_COPY_TO_DEVICE,
                               _stream_handle(k_pool.device, stream))
    if st != KVT_OK:
        raise KvtError(st, "kvt_copy_blocks")


def decode_workspace_bytes(k_pool, v_pool, block_table, prefix_len, num_q_heads: int) -> int:
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, np.ones(len(prefix_len), dtype=np.int32), block_table, False)
    return int(lib().kvt_decode_workspace_bytes(ctypes.byref(pool), ctypes.byref(seqs.struct), int(num_q_heads)))


def decode_attention(q, k_pool, v_pool, block_table, prefix_len: Sequence[int], scale: Optional[float] = None, *,
                     out=None, lse=None, return_lse: bool = False, workspace=None, use_workspace: bool = True,
                     stream=None, checked: bool = False):
    """One decoding step (``kvt_decode_attention``): row b of ``q`` ([B][Hq][D])
    is the new token of sequence b at position ``prefix_len[b]``, whose K/V
    was appended first.  Returns ``out`` ([B][Hq][D]) or ``(out, lse)``."""
    ones = np.ones(len(prefix_len), dtype=np.int32)
    return _attention("kvt_decode_attention", "kvt_decode_workspace_bytes", q, k_pool, v_pool, block_table,
                      prefix_len, ones, scale, out, lse, return_lse, workspace, use_workspace, stream, checked)


def _attention(entry: str, ws_entry: str, q, k_pool, v_pool, block_table, prefix_len, suffix_len, scale, out, lse,
               return_lse, workspace, use_workspace, stream, checked, shared: Optional[int] = None):
    import torch
    if stream is not None:
        # buffers allocated here (out, lse, the split workspace) belong to the
        # stream the kernels run on: torch's caching allocator then hands a
        # freed workspace to the next allocation on that stream only, which is
        # ordered after these kernels
        with torch.cuda.stream(stream):
            return _attention(entry, ws_entry, q, k_pool, v_pool, block_table, prefix_len, suffix_len, scale, out,
                              lse, return_lse, workspace, use_workspace, None, checked, shared)
    lead = () if shared is None else shared     # the cascade entry points take (shared_len, mode) after seqs
    pool = _pool_struct(k_pool, v_pool)
    seqs = _seqs(prefix_len, suffix_len, block_table, checked)
    T = sum(seqs.suffix)
    Hq = int(q.shape[1])
    _check_tokens(q, "q", T, Hq, pool.head_dim, k_pool.dtype)
    if scale is None:
        scale = 1.0 / math.sqrt(pool.head_dim)
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_tokens(out, "out", T, Hq, pool.head_dim, k_pool.dtype)
    want_lse = return_lse or lse is not None
    if want_lse and lse is None:
        lse = torch.empty((T, Hq), dtype=torch.float32, device=q.device)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (T, Hq) or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [T][Hq] tensor")
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    elif use_workspace:
        need = int(getattr(lib(), ws_entry)(ctypes.byref(pool), ctypes.byref(seqs.struct), *lead, Hq))
        if need:
            workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
            ws_ptr, ws_bytes = workspace.data_ptr(), need
    st = getattr(lib(), entry)(ctypes.byref(pool), ctypes.byref(seqs.struct), *lead, q.data_ptr(), Hq, float(scale),
                               out.data_ptr(), lse.data_ptr() if lse is not None else None, ws_ptr, ws_bytes,
                               _stream_handle(q.device, stream))
    if st != KVT_OK:
        raise KvtError(st, entry)
    return (out, lse) if want_lse else out


# ---------------------------------------------------------------------------
# host block manager
# ---------------------------------------------------------------------------

class Manager:
    """The library's host block manager over ``num_pages`` KV pages.

    Each method is one ``kvt_mgr_*`` call; a non-OK status raises
    ``KvtError``.  Request-boundary calls return the report as a dict."""

    def __init__(self, num_pages: int):
        self._h = lib().kvt_mgr_create(int(num_pages))
        if not self._h:
            raise ValueError(f"kvt_mgr_create: bad page count {num_pages}")

    def close(self):
        if self._h:
            lib().kvt_mgr_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _call(self, name: str, *args):
        st = getattr(lib(), name)(self._h, *[int(a) for a in args])
        if st != KVT_OK:
            raise KvtError(st, name)

    def _report(self, name: str, ctx: int) -> dict:
        rep = KvtMgrReport()
        st = getattr(lib(), name)(self._h, int(ctx), ctypes.byref(rep))
        if st != KVT_OK:
            raise KvtError(st, name)
        return rep.as_dict()

    def spawn(self, ctx): self._call("kvt_mgr_spawn", ctx)
    def fork(self, parent, child): self._call("kvt_mgr_fork", parent, child)
    def append(self, ctx, tokens): self._call("kvt_mgr_append", ctx, tokens)
    def one_off(self, ctx): self._call("kvt_mgr_one_off", ctx)
    def pin(self, ctx, i): self._call("kvt_mgr_pin", ctx, i)
    def unpin(self, ctx, i): self._call("kvt_mgr_unpin", ctx, i)
    def replace(self, ctx, i, tokens): self._call("kvt_mgr_replace", ctx, i, tokens)
    def remove(self, ctx, i): self._call("kvt_mgr_remove", ctx, i)
    def terminate(self, ctx): self._call("kvt_mgr_terminate", ctx)
    def begin_request(self, ctx): self._call("kvt_mgr_begin_request", ctx)
    def end_request(self, ctx): self._call("kvt_mgr_end_request", ctx)

    def start_prefill(self, ctx) -> dict:
        return self._report("kvt_mgr_start_prefill", ctx)

    def prefill_done(self, ctx) -> dict:
        return self._report("kvt_mgr_prefill_done", ctx)

    @staticmethod
    def encode(events) -> np.ndarray:
        """(method name, args) pairs as the int64 [n][4] array replay takes."""
        arr = np.zeros((len(events), 4), dtype=np.int64)
        for i, (op, args) in enumerate(events):
            arr[i, 0] = MGR_OPS.index(op)
            arr[i, 1:1 + len(args)] = args
        return arr

    def replay(self, events) -> tuple:
        """Run an encoded event array natively; returns (calls that succeeded,
        summed start_prefill / prefill_done reports)."""
        arr = np.ascontiguousarray(events, dtype=np.int64).reshape(-1, 4)
        rep = KvtMgrReport()
        ok = int(lib().kvt_mgr_replay(self._h, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), arr.shape[0],
                                      ctypes.byref(rep)))
        if ok < 0:
            raise ValueError("kvt_mgr_replay rejected its arguments")
        return ok, rep.as_dict()

    def free_pages(self) -> int:
        return int(lib().kvt_mgr_free_pages(self._h))

    def live_entries(self) -> int:
        return int(lib().kvt_mgr_live_entries(self._h))

    def message_state(self, ctx, i) -> int:
        return int(lib().kvt_mgr_message_state(self._h, int(ctx), int(i)))

    def entry_tier(self, ctx, i) -> Optional[int]:
        t = int(lib().kvt_mgr_entry_tier(self._h, int(ctx), int(i)))
        return None if t < 0 else t

    def message_pages(self, ctx, i) -> Optional[list]:
        n = int(lib().kvt_mgr_message_pages(self._h, int(ctx), int(i), None, 0))
        if n < 0:
            return None
        buf = (ctypes.c_int32 * max(n, 1))()
        lib().kvt_mgr_message_pages(self._h, int(ctx), int(i), buf, n)
        return list(buf[:n])
