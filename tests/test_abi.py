"""C-ABI library: it loads, exports every declared symbol, and rejects bad
arguments on the host before any HIP call (CPU only).

The pointers used here are fake; each call is built to fail validation, so no
kernel is ever launched.  Every test that passes fake pointers is skipped
when a GPU is present, so that a validation bug could never launch a kernel
on them.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_39819_amd import kvt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvt.h")

FAKE_K, FAKE_V, FAKE_BT = 0x10000000, 0x20000000000, 0x30000000000
FAKE_Q, FAKE_OUT = 0x40000000000, 0x50000000000


def _gpu_present():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


no_gpu_only = pytest.mark.skipif(_gpu_present(), reason="fake-pointer late-validation test runs only without a GPU")


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kvt_[a-z_]+)\s*\(", src)))


def test_header_declares_the_expected_entry_points():
    assert declared_symbols() == sorted(kvt.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = kvt.lib()
    for name in declared_symbols():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", kvt.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (kvt_[a-z_]+)\b", out))
    assert set(declared_symbols()) <= exported


def test_status_strings():
    for code in range(7):
        assert kvt.status_str(code)
    assert kvt.status_str(99) == "unknown status"
    assert kvt.lib().kvt_last_hip_error() == 0


def _pool(nb=64, hkv=1, d=64, dtype=kvt.KVT_DTYPE_BF16, k=FAKE_K, v=FAKE_V):
    return kvt.raw_pool(k, v, nb, hkv, d, dtype)


def _extend(pool, seqs, hq=4, scale=0.125, q=FAKE_Q, out=FAKE_OUT, ws=None, ws_bytes=0):
    L = kvt.lib()
    return L.kvt_extend_attention(ctypes.byref(pool) if pool is not None else None,
                                  ctypes.byref(seqs.struct) if seqs is not None else None,
                                  q, hq, scale, out, None, ws, ws_bytes, None)


def _decode(pool, seqs, hq=4, scale=0.125, q=FAKE_Q, out=FAKE_OUT, ws=None, ws_bytes=0):
    L = kvt.lib()
    return L.kvt_decode_attention(ctypes.byref(pool) if pool is not None else None,
                                  ctypes.byref(seqs.struct) if seqs is not None else None,
                                  q, hq, scale, out, None, ws, ws_bytes, None)


def _append(pool, seqs, kn=FAKE_Q, vn=FAKE_OUT):
    L = kvt.lib()
    return L.kvt_append_kv(ctypes.byref(pool) if pool is not None else None,
                           ctypes.byref(seqs.struct) if seqs is not None else None, kn, vn, None)


def _seqs(P=(240,), S=(16,), bt=FAKE_BT, max_blocks=16, host=None):
    return kvt.RawSeqs(list(P), list(S), bt, max_blocks, host)


@no_gpu_only
@pytest.mark.parametrize("call", [_extend, _append])
def test_invalid_arguments_are_rejected(call):
    E = kvt.KVT_ERR_INVALID_ARG
    assert call(None, _seqs()) == E
    assert call(_pool(k=0), _seqs()) == E
    assert call(_pool(nb=0), _seqs()) == E
    assert call(_pool(hkv=0), _seqs()) == E
    assert call(_pool(), None) == E
    assert call(_pool(), _seqs(P=(), S=())) == E                    # no sequences
    assert call(_pool(), _seqs(S=(0,))) == E                         # empty suffix
    assert call(_pool(), _seqs(P=(-1,))) == E                        # negative prefix
    assert call(_pool(), _seqs(bt=0)) == E                           # no block table
    assert call(_pool(), _seqs(max_blocks=15)) == E                  # 256 tokens need 16 pages


@no_gpu_only
def test_unsupported_shapes_are_rejected():
    U = kvt.KVT_ERR_UNSUPPORTED
    for call in (_extend, _append):
        assert call(_pool(d=96), _seqs()) == U
        assert call(_pool(d=256), _seqs()) == U
        assert call(_pool(dtype=7), _seqs()) == U


@no_gpu_only
def test_extend_specific_checks():
    E = kvt.KVT_ERR_INVALID_ARG
    assert _extend(_pool(), _seqs(), q=0) == E
    assert _extend(_pool(), _seqs(), out=0) == E
    assert _extend(_pool(hkv=2), _seqs(), hq=3) == E                 # Hq not a multiple of Hkv
    assert _extend(_pool(), _seqs(), hq=0) == E
    assert _extend(_pool(), _seqs(), scale=0.0) == E
    assert _extend(_pool(), _seqs(), scale=-1.0) == E
    assert _extend(_pool(), _seqs(), scale=float("nan")) == E
    assert _extend(_pool(), _seqs(), scale=float("inf")) == E
    assert _extend(_pool(), _seqs(), out=FAKE_Q + 64) == E           # out overlaps q
    assert _extend(_pool(), _seqs(), out=FAKE_K + 128) == E          # out inside the K pool
    # 2^24 new tokens x 128 query heads = 2^31 packed rows: past the kernels' 32-bit row indices
    big = _seqs(P=(0,), S=(1 << 24,), max_blocks=1 << 20)
    assert _extend(_pool(nb=1 << 20), big, hq=128) == E
    assert _extend(_pool(nb=1 << 20), big, hq=128, ws=0x60000000000, ws_bytes=1 << 40) == E
    pool = _pool(nb=1 << 20)
    assert kvt.lib().kvt_extend_workspace_bytes(ctypes.byref(pool), ctypes.byref(big.struct), 128) == 0
    # device buffers must be 16-byte aligned (lse 4-byte)
    assert _extend(_pool(), _seqs(), q=FAKE_Q + 8) == E
    assert _extend(_pool(), _seqs(), out=FAKE_OUT + 8) == E
    assert _extend(_pool(k=FAKE_K + 8), _seqs()) == E
    assert kvt.lib().kvt_extend_attention(ctypes.byref(_pool()), ctypes.byref(_seqs().struct), FAKE_Q, 4, 0.125,
                                          FAKE_OUT, FAKE_OUT + (1 << 30) + 2, None, 0, None) == E
    s8k = _seqs(P=(8192,), S=(512,), max_blocks=544)
    assert _extend(_pool(nb=65536, hkv=8, d=128), s8k, hq=32, ws=0x60000000008, ws_bytes=1 << 30) == E
    assert _append(_pool(), _seqs(), kn=FAKE_Q + 4) == E


@no_gpu_only
def test_decode_specific_checks():
    E, U = kvt.KVT_ERR_INVALID_ARG, kvt.KVT_ERR_UNSUPPORTED
    one = _seqs(S=(1,))
    assert _decode(None, one) == E
    assert _decode(_pool(), _seqs()) == E                            # suffix 16: not a decode step
    assert _decode(_pool(), _seqs(P=(240, 240), S=(1, 2), max_blocks=16)) == E
    assert _decode(_pool(), one, q=0) == E
    assert _decode(_pool(), one, out=0) == E
    assert _decode(_pool(hkv=2), one, hq=3) == E
    assert _decode(_pool(), one, scale=0.0) == E
    assert _decode(_pool(), one, out=FAKE_Q + 64) == E
    assert _decode(_pool(), one, hq=33) == U                         # more than 32 query heads per kv-head
    assert _decode(_pool(d=96), one) == U
    host = np.arange(16, dtype=np.int32).reshape(1, 16); host[0, 3] = 64
    assert _decode(_pool(), _seqs(S=(1,), host=host)) == kvt.KVT_ERR_OUT_OF_RANGE


def _cascade(pool, seqs, shared, hq=4, scale=0.125, q=FAKE_Q, out=FAKE_OUT, ws=None, ws_bytes=0):
    return kvt.lib().kvt_cascade_extend_attention(ctypes.byref(pool), ctypes.byref(seqs.struct), shared, q, hq,
                                                  scale, out, None, ws, ws_bytes, None)


@no_gpu_only
def test_cascade_specific_checks():
    E = kvt.KVT_ERR_INVALID_ARG
    two = _seqs(P=(240, 100), S=(16, 16), max_blocks=16)
    for bad in (0, 8, 17, 112, -16):          # not a positive multiple of 16, or longer than a prefix (100)
        assert _cascade(_pool(), two, bad, ws=0x60000000000, ws_bytes=1 << 30) == E
    host = np.stack([np.arange(16), np.arange(16, 32)]).astype(np.int32)   # first pages differ
    assert _cascade(_pool(), _seqs(P=(240, 100), S=(16, 16), max_blocks=16, host=host), 64,
                    ws=0x60000000000, ws_bytes=1 << 30) == E
    # a call that takes the shared pass (short messages over a long shared prefix) needs its partials
    pool = _pool(nb=1 << 20, hkv=8, d=128)
    short = _seqs(P=[32768 + 37 * i for i in range(16)], S=[16] * 16, max_blocks=2100)
    assert kvt.lib().kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(short.struct), 32768, 96) == 1
    assert _cascade(pool, short, 32768, hq=96, ws=0x60000000000, ws_bytes=16) == kvt.KVT_ERR_WORKSPACE


def test_cascade_workspace_bytes():
    pool = _pool(nb=1 << 20, hkv=8, d=128)
    s = _seqs(P=(8192, 20000), S=(2048, 1000), max_blocks=2048)
    L = kvt.lib()
    # the shared pass: one fp32 partial set per key split of the shared part
    # and of the private parts, merged by the combine kernel
    ws = L.kvt_cascade_workspace_bytes_ex(ctypes.byref(pool), ctypes.byref(s.struct), 4096,
                                          kvt.CASCADE_SHARED_PASS, 96)
    rows = 3048 * 96
    parts = ws // (rows * (128 + 2) * 4)
    assert parts >= 2 and ws == -(-parts * rows * 128 * 4 // 256) * 256 + parts * rows * 2 * 4
    # this shape runs the plain extend plan by default, with its workspace
    assert L.kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(s.struct), 4096, 96) == 0
    assert (L.kvt_cascade_workspace_bytes(ctypes.byref(pool), ctypes.byref(s.struct), 4096, 96)
            == L.kvt_extend_workspace_bytes(ctypes.byref(pool), ctypes.byref(s.struct), 96))
    assert L.kvt_cascade_workspace_bytes(ctypes.byref(pool), ctypes.byref(s.struct), 4100, 96) == 0


def test_cascade_runs_the_plain_plan_when_its_estimate_loses():
    """Short messages over a long shared prefix take the shared pass; long
    suffixes (the forked-agents shape: every sequence's row tiles nearly full)
    take the plain extend plan, whose workspace the call then asks for."""
    L = kvt.lib()
    pool = _pool(nb=1 << 20, hkv=8, d=128)
    P = [32768 + 37 * i for i in range(16)]
    short = _seqs(P=P, S=[16] * 16, max_blocks=2100)
    assert L.kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(short.struct), 32768, 96) == 1
    P = [4096 + 3000 * i for i in range(16)]
    S = [256 + 250 * i for i in range(16)]
    long_ = _seqs(P=P, S=S, max_blocks=5000)
    assert L.kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(long_.struct), 4096, 96) == 0
    assert (L.kvt_cascade_workspace_bytes(ctypes.byref(pool), ctypes.byref(long_.struct), 4096, 96)
            == L.kvt_extend_workspace_bytes(ctypes.byref(pool), ctypes.byref(long_.struct), 96))
    assert L.kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(long_.struct), 4100, 96) == -1


def test_cascade_splits_short_private_parts_to_fill_the_launch():
    """16 short messages over a 32K shared prefix: the shared part takes 8
    key splits (768 workgroups, three full rounds of 256 CUs) and the 128
    private (row tile, kv-head) units, each under 1024 private keys, take 2
    splits so that they fill a whole fourth round instead of half of it: 10
    partial sets in the workspace.  The plain extend's rule (at least 1024
    keys of the shortest sequence per split) would not split them."""
    L = kvt.lib()
    pool = _pool(nb=1 << 20, hkv=8, d=128)
    s = _seqs(P=[32768 + 37 * i for i in range(16)], S=[16] * 16, max_blocks=2100)
    ws = L.kvt_cascade_workspace_bytes_ex(ctypes.byref(pool), ctypes.byref(s.struct), 32768,
                                          kvt.CASCADE_SHARED_PASS, 96)
    rows = 16 * 16 * 96
    assert ws == -(-10 * rows * 128 * 4 // 256) * 256 + 10 * rows * 2 * 4
    assert L.kvt_cascade_uses_shared_pass(ctypes.byref(pool), ctypes.byref(s.struct), 32768, 96) == 1


def _copy(pool, ids=FAKE_BT, ids_host=None, n=4, host=FAKE_OUT, direction=0):
    h = None if ids_host is None else np.ascontiguousarray(ids_host, dtype=np.int32).ctypes.data_as(
        ctypes.POINTER(ctypes.c_int32))
    return kvt.lib().kvt_copy_blocks(ctypes.byref(pool) if pool is not None else None, ids, h, n, host, direction,
                                     None)


@no_gpu_only
def test_copy_blocks_checks():
    E, O = kvt.KVT_ERR_INVALID_ARG, kvt.KVT_ERR_OUT_OF_RANGE
    assert _copy(_pool(), n=0, ids=None, host=None) == kvt.KVT_OK          # nothing to move
    assert _copy(None) == E
    assert _copy(_pool(d=96)) == kvt.KVT_ERR_UNSUPPORTED
    assert _copy(_pool(), n=-1) == E
    assert _copy(_pool(), ids=None) == E
    assert _copy(_pool(), host=None) == E
    assert _copy(_pool(), direction=2) == E
    assert _copy(_pool(), ids_host=[0, 1, 64, 2]) == O                      # pool has 64 pages
    assert _copy(_pool(), ids_host=[0, -1, 3, 2]) == O
    assert _copy(_pool(), ids_host=[5, 1, 5, 2], direction=1) == O          # one page written twice
    # host memory that HIP did not pin is refused before anything is enqueued
    pageable = np.zeros(4 * 2 * 16 * 64, dtype=np.uint16)
    assert _copy(_pool(), ids_host=[0, 1, 2, 3], host=pageable.ctypes.data) == E


def test_decode_workspace_bytes_follow_the_split_plan():
    def ws(pool, seqs, hq):
        return kvt.lib().kvt_decode_workspace_bytes(ctypes.byref(pool), ctypes.byref(seqs.struct), hq)
    pool = _pool(nb=1 << 20, hkv=8, d=128)
    # 4 sequences x 8 kv-heads = 32 units: splits until 512 workgroups, capped at 16
    s = _seqs(P=(65535, 40000, 30000, 20000), S=(1, 1, 1, 1), max_blocks=4096)
    rows = 4 * 96
    assert ws(pool, s, 96) == 16 * rows * 128 * 4 + 16 * rows * 2 * 4
    # the shortest sequence keeps >= 1024 keys per split: 3000 keys -> 2 splits
    s2 = _seqs(P=(65535, 2999), S=(1, 1), max_blocks=4096)
    assert ws(pool, s2, 96) == 2 * 2 * 96 * 128 * 4 + 2 * 2 * 96 * 2 * 4
    # 64 sequences x 8 kv-heads = 512 units: no split
    s3 = _seqs(P=(4095,) * 64, S=(1,) * 64, max_blocks=256)
    assert ws(pool, s3, 96) == 0
    assert ws(pool, _seqs(), 96) == 0                                # not a decode step


@no_gpu_only
def test_append_specific_checks():
    E = kvt.KVT_ERR_INVALID_ARG
    assert _append(_pool(), _seqs(), kn=0) == E
    assert _append(_pool(), _seqs(), vn=0) == E
    assert _append(_pool(), _seqs(), kn=FAKE_K + 4096) == E          # source inside the pool


@no_gpu_only
def test_checked_mode_rejects_out_of_range_ids():
    O = kvt.KVT_ERR_OUT_OF_RANGE
    table = np.arange(16, dtype=np.int32).reshape(1, 16)
    bad = table.copy(); bad[0, 7] = 64                               # pool has 64 blocks: id 64 is outside
    assert _extend(_pool(), _seqs(host=bad)) == O
    assert _append(_pool(), _seqs(host=bad)) == O
    neg = table.copy(); neg[0, 0] = -1
    assert _extend(_pool(), _seqs(host=neg)) == O


@no_gpu_only
def test_checked_append_rejects_two_tokens_on_one_slot():
    # two sequences whose new positions land on the same page slot
    host = np.array([[0, 1, 2], [5, 1, 6]], dtype=np.int32)
    s = _seqs(P=(16, 16), S=(4, 4), max_blocks=3, host=host)
    assert _append(_pool(), s) == kvt.KVT_ERR_OUT_OF_RANGE


def _ws_bytes(pool, seqs, hq):
    return kvt.lib().kvt_extend_workspace_bytes(ctypes.byref(pool), ctypes.byref(seqs.struct), hq)


def test_workspace_bytes_follow_the_split_plan():
    pool = _pool(nb=65536, hkv=8, d=128)
    # short suffix (512 tokens x 32 heads): 64 row tiles -> 4 key splits
    s = _seqs(P=(8192,), S=(512,), max_blocks=544)
    rows = 512 * 32
    assert _ws_bytes(pool, s, 32) == 4 * rows * 128 * 4 + 4 * rows * 2 * 4
    # long suffix (2048 x 96 heads): 768 row tiles fill the chip, no split
    s3 = _seqs(P=(131072,), S=(2048,), max_blocks=8320)
    assert _ws_bytes(_pool(nb=1 << 20, hkv=8, d=128), s3, 96) == 0
    # one GPU's share under 4-way head parallelism: 192 row tiles -> 4 splits
    assert _ws_bytes(_pool(nb=1 << 20, hkv=2, d=128), s3, 24) == 4 * 2048 * 24 * (128 + 2) * 4
    # a ragged batch (contexts 1K..32K, 16 new tokens each): the shortest
    # context alone would allow no split, yet the 32K sequence's row tile
    # would run alone at the end; list scheduling splits 16 ways
    s4 = _seqs(P=[1024 * 2 ** i for i in range(6)], S=[16] * 6, max_blocks=2100)
    rows4 = 6 * 16 * 96
    assert _ws_bytes(_pool(nb=1 << 20, hkv=8, d=128), s4, 96) == 16 * rows4 * 128 * 4 + 16 * rows4 * 2 * 4
    # invalid arguments -> 0
    assert _ws_bytes(pool, s, 33) == 0


@no_gpu_only
def test_small_workspace_is_rejected():
    pool = _pool(nb=65536, hkv=8, d=128)
    s = _seqs(P=(8192,), S=(512,), max_blocks=544)
    assert _extend(pool, s, hq=32, scale=0.088, ws=0x60000000000, ws_bytes=16) == kvt.KVT_ERR_WORKSPACE


@no_gpu_only
def test_noalloc_rejects_plans_beyond_its_static_scratch():
    """kvt_extend_attention_noalloc runs the same split plan as
    kvt_extend_attention; a plan whose partials exceed the static scratch is
    refused on the host (one GPU's share of the 128K turn under 4-way head
    parallelism: 4 key splits x 2048 x 24 rows x 130 floats = 102 MB)."""
    pool = _pool(nb=1 << 20, hkv=2, d=128)
    s = _seqs(P=(131072,), S=(2048,), max_blocks=8320)
    need = _ws_bytes(pool, s, 24)
    assert need > kvt.NOALLOC_SCRATCH_BYTES
    L = kvt.lib()
    st = L.kvt_extend_attention_noalloc(ctypes.byref(pool), ctypes.byref(s.struct), FAKE_Q, 24, 0.088, FAKE_OUT,
                                        None, None)
    assert st == kvt.KVT_ERR_SCRATCH_LIMIT
    assert "scratch" in kvt.status_str(st)
    # the same checks as the workspace entry point run first
    assert L.kvt_extend_attention_noalloc(ctypes.byref(pool), ctypes.byref(s.struct), 0, 24, 0.088, FAKE_OUT,
                                          None, None) == kvt.KVT_ERR_INVALID_ARG
    assert L.kvt_extend_attention_noalloc(ctypes.byref(pool), ctypes.byref(s.struct), FAKE_Q, 25, 0.088, FAKE_OUT,
                                          None, None) == kvt.KVT_ERR_INVALID_ARG


def test_binding_fails_loudly_without_the_library(monkeypatch):
    monkeypatch.setattr(kvt, "_lib", None)
    monkeypatch.setattr(kvt, "LIB_PATH", "/nonexistent/libkvt.so")
    with pytest.raises(RuntimeError, match="missing"):
        kvt.lib()


def test_length_arrays_reject_values_outside_int32():
    """The binding's host arrays: short lists of ints take a fast path, the
    rest goes through numpy; neither wraps a value outside int32."""
    assert list(kvt._i32_array([0, 5, 2 ** 31 - 1])) == [0, 5, 2 ** 31 - 1]
    assert list(kvt._i32_array(np.array([[1, 2], [3, 4]]))) == [1, 2, 3, 4]
    assert list(kvt._i32_array(list(range(100)))) == list(range(100))      # long list: numpy path
    assert list(kvt._i32_array((np.int64(7), 8))) == [7, 8]                 # numpy scalars: numpy path
    assert list(kvt._i32_array(np.array([3, 2 ** 31 - 1], dtype=np.int64))) == [3, 2 ** 31 - 1]
    assert list(kvt._i32_array(np.array([7], dtype=np.uint64))) == [7]
    for bad in ([2 ** 31], [-2 ** 31 - 1], [1, 2 ** 40], list(range(99)) + [2 ** 33],
                np.array([2 ** 33 + 5], dtype=np.int64), np.array([-2 ** 31 - 1], dtype=np.int64),
                np.array([2 ** 32], dtype=np.uint64), [2 ** 70]):
        with pytest.raises((OverflowError, ValueError)):
            kvt._i32_array(bad)
