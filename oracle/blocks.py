"""Plain definitions of the page moves between the HBM tier and host memory
(test oracle).

TEST INFRASTRUCTURE -- see the package docstring.  Numpy only; a bitwise copy,
no arithmetic on the values.

The multi-tier cache keeps whole pages in GPU HBM, host memory or remote
memory and moves them between tiers as pages are admitted and evicted
(paper §6, with the local GPU <-> CPU engine of §7).  A move of the page list
``ids`` copies, for every listed page and both pools, the page's
``[num_kv_heads][16][head_dim]`` block; the host side packs the list in order
as ``[n][K | V][num_kv_heads][16][head_dim]``.
"""
from __future__ import annotations

import numpy as np


def oracle_to_host(k_pool, v_pool, ids) -> np.ndarray:
    """host[i][0] = K page ids[i], host[i][1] = V page ids[i]."""
    ids = np.asarray(ids, dtype=np.int64)
    host = np.empty((len(ids), 2) + tuple(np.shape(k_pool)[1:]), dtype=np.asarray(k_pool).dtype)
    for i, p in enumerate(ids):
        host[i, 0] = k_pool[p]
        host[i, 1] = v_pool[p]
    return host


def oracle_to_device(k_pool, v_pool, ids, host):
    """Return new pools where page ids[i] of K and V holds host[i][0] and
    host[i][1]; every other page is unchanged.  ids must be distinct."""
    ids = np.asarray(ids, dtype=np.int64)
    if len(set(ids.tolist())) != len(ids):
        raise ValueError("a page may be written once per move")
    kp = np.array(k_pool, copy=True)
    vp = np.array(v_pool, copy=True)
    for i, p in enumerate(ids):
        kp[p] = host[i, 0]
        vp[p] = host[i, 1]
    return kp, vp
