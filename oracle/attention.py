"""Plain fp64 definitions of paged append and extend attention (test oracle).

TEST INFRASTRUCTURE -- see the package docstring.  Numpy only; fp64 for all
floating point; no blocking, fusion or online rescaling beyond what the
definition states (row chunks only bound memory: each row is computed by the
same formula independently).

Array conventions (the caller's stored values, unmodified):
* bf16 tensors arrive as ``uint16`` bit patterns, fp32 tensors as ``float32``;
* pools are ``[num_blocks][num_kv_heads][16][head_dim]``;
* ``q``/``out`` rows are packed by sequence: row ``off_b + i`` is suffix token i
  of sequence b, ``off_b = S_0 + ... + S_{b-1}``;
* query head h reads kv-head ``h // (Hq // Hkv)`` (consecutive head groups).
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

PAGE = 16


def storage_to_f64(a: np.ndarray) -> np.ndarray:
    """Exact widening of stored values to float64 (bf16 bits or float32)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if a.dtype == np.float32 or a.dtype == np.float64:
        return a.astype(np.float64)
    raise TypeError(f"unsupported storage dtype {a.dtype}")


def _offsets(suffix_len) -> np.ndarray:
    s = np.asarray(suffix_len, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(s)])


def oracle_append(k_pool, v_pool, block_table, prefix_len, suffix_len, k_new, v_new):
    """Write each new token's K/V row into its page slot; return new pools.

    Token t of sequence b is logical position p = P_b + t; it is stored in
    physical page ``block_table[b][p // 16]`` at slot ``p % 16``, for every
    kv-head.  A bitwise copy: no arithmetic on the values.  Every other byte
    of the pools is returned unchanged.
    """
    kp = np.array(k_pool, copy=True)
    vp = np.array(v_pool, copy=True)
    off = _offsets(suffix_len)
    for b in range(len(prefix_len)):
        P = int(prefix_len[b])
        for t in range(int(suffix_len[b])):
            p = P + t
            page = int(block_table[b][p // PAGE])
            kp[page, :, p % PAGE, :] = k_new[off[b] + t]
            vp[page, :, p % PAGE, :] = v_new[off[b] + t]
    return kp, vp


def gather_logical(pool, block_table_row, length: int, kv_head: int) -> np.ndarray:
    """Logical positions 0..length-1 of one kv-head, read through the block table, in fp64."""
    n_pages = (length + PAGE - 1) // PAGE
    pages = np.asarray(block_table_row[:n_pages], dtype=np.int64)
    rows = storage_to_f64(pool[pages, kv_head])          # [n_pages, 16, D]
    return rows.reshape(n_pages * PAGE, -1)[:length]


def oracle_extend(q, k_pool, v_pool, block_table, prefix_len, suffix_len, num_kv_heads: int,
                  scale: float, rows: Optional[Sequence[Optional[np.ndarray]]] = None,
                  chunk_rows: int = 256):
    """Extend attention of every (or the selected) suffix token, in fp64.

    For sequence b, suffix token i and query head h (kv-head g = h // G):
      s_j   = scale * <q[b,i,h], K_b[j]>      for j = 0 .. P_b + i (inclusive)
      out   = sum_j softmax(s)_j * V_b[j]
      lse   = ln sum_j exp(s_j)
    with K_b, V_b the logical sequence read through the block table.

    ``rows``: optional per-sequence arrays of suffix-token indices; when given,
    only those tokens are computed and the outputs hold them in order
    (sequence by sequence).  Returns ``(out [n, Hq, D], lse [n, Hq])`` as float64.
    """
    q = np.asarray(q)
    T, Hq, D = q.shape
    Hkv = int(num_kv_heads)
    G = Hq // Hkv
    off = _offsets(suffix_len)
    B = len(prefix_len)
    sel = []
    for b in range(B):
        r = np.arange(int(suffix_len[b])) if rows is None or rows[b] is None else np.asarray(rows[b], dtype=np.int64)
        sel.append(r)
    n_out = sum(len(r) for r in sel)
    out = np.empty((n_out, Hq, D), dtype=np.float64)
    lse = np.empty((n_out, Hq), dtype=np.float64)
    base = 0
    for b in range(B):
        P = int(prefix_len[b])
        L = P + int(suffix_len[b])
        toks = sel[b]
        for g in range(Hkv):
            Kb = gather_logical(k_pool, block_table[b], L, g)   # [L, D]
            Vb = gather_logical(v_pool, block_table[b], L, g)
            key_pos = np.arange(L)
            step = max(1, chunk_rows // G)
            for c0 in range(0, len(toks), step):
                tk = toks[c0:c0 + step]
                Qc = storage_to_f64(q[off[b] + tk, g * G:(g + 1) * G, :])   # [nt, G, D]
                nt = Qc.shape[0]
                Qc = Qc.reshape(nt * G, D)
                limit = np.repeat(P + tk, G)                               # last visible position per row
                scores = scale * (Qc @ Kb.T)                               # [nt*G, L]
                scores[key_pos[None, :] > limit[:, None]] = -np.inf
                mx = scores.max(axis=1)
                w = np.exp(scores - mx[:, None])
                z = w.sum(axis=1)
                o = (w @ Vb) / z[:, None]
                out[base + c0: base + c0 + nt, g * G:(g + 1) * G, :] = o.reshape(nt, G, D)
                lse[base + c0: base + c0 + nt, g * G:(g + 1) * G] = (mx + np.log(z)).reshape(nt, G)
        base += len(toks)
    return out, lse


def brute_force_extend(q, logical_k: Sequence[np.ndarray], logical_v: Sequence[np.ndarray],
                       prefix_len, suffix_len, num_kv_heads: int, scale: float):
    """Pure-Python loops over the un-paged logical sequences (tiny inputs only).

    ``logical_k[b]`` / ``logical_v[b]`` are ``[P_b + S_b, Hkv, D]`` stored values
    in logical order, built before any paging.  Uses ``math.fsum`` and
    ``math.exp`` so the result is accurate to a few ulps of fp64.
    """
    q = storage_to_f64(q)
    T, Hq, D = q.shape
    G = Hq // int(num_kv_heads)
    off = _offsets(suffix_len)
    out = np.zeros((T, Hq, D), dtype=np.float64)
    lse = np.zeros((T, Hq), dtype=np.float64)
    for b in range(len(prefix_len)):
        K = storage_to_f64(logical_k[b]).tolist()
        V = storage_to_f64(logical_v[b]).tolist()
        P = int(prefix_len[b])
        for i in range(int(suffix_len[b])):
            row = off[b] + i
            for h in range(Hq):
                g = h // G
                qv = q[row, h].tolist()
                s = [scale * math.fsum(qv[d] * K[j][g][d] for d in range(D)) for j in range(P + i + 1)]
                m = max(s)
                e = [math.exp(x - m) for x in s]
                z = math.fsum(e)
                for d in range(D):
                    out[row, h, d] = math.fsum(e[j] * V[j][g][d] for j in range(len(e))) / z
                lse[row, h] = m + math.log(z)
    return out, lse
