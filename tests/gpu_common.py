"""Shared helpers of the GPU parity tests (harness only: staging, comparisons)."""
from __future__ import annotations

import functools
import sys
import time

import numpy as np

from oracle import oracle_append, oracle_extend, storage_to_f64
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import make_config, stage_on_device, torch_to_np

# parity tolerance for bf16 inputs
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
# relative L2 bound beside the absolute ones: at 128K+ keys the outputs' own
# scale (std ~ sqrt(e / n)) is close to MEAN_ABS, so an all-zero or
# quarter-wrong output can sit inside the absolute bounds but not this one
# (the kernels measure 2e-3 .. 4e-3: bf16 rounding of P and of the output)
REL_L2 = 1e-2


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=8)
def cached_config(name: str, variant: str = "normal"):
    t0 = time.time()
    w = make_config(name, variant=variant)
    say(f"generated {name}/{variant} in {time.time() - t0:.1f}s")
    return w


@functools.lru_cache(maxsize=8)
def oracle_pools(name: str, variant: str = "normal"):
    w = cached_config(name, variant)
    return oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)


def stage(w, device="cuda"):
    import torch
    say(f"staging {w.name}/{w.variant}: B={w.num_seqs} Hq={w.num_q_heads} Hkv={w.num_kv_heads} D={w.head_dim} "
        f"NB={w.num_blocks} T={w.total_tokens}")
    d = stage_on_device(w, device)
    torch.cuda.synchronize()
    return d


def run_append(w, d, checked=False):
    import torch
    say(f"kvt_append_kv {w.name}/{w.variant}")
    kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"],
                  checked=checked)
    torch.cuda.synchronize()


def run_extend(w, d, **kw):
    import torch
    say(f"kvt_extend_attention {w.name}/{w.variant} {kw if kw else ''}")
    r = kvt.extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                             w.scale, **kw)
    torch.cuda.synchronize()
    return r


def to_f64(t, dtype):
    return storage_to_f64(torch_to_np(t, dtype))


def sample_rows(w, per_seq: int, seed: int = 0):
    """First/last tokens plus seeded random ones, per sequence (None = all)."""
    rng = np.random.default_rng(seed)
    rows = []
    for b in range(w.num_seqs):
        S = int(w.suffix_len[b])
        if per_seq is None or S <= per_seq:
            rows.append(np.arange(S))
            continue
        edge = min(4, per_seq // 4)
        pick = set(range(edge)) | set(range(S - edge, S))
        pick |= set(rng.choice(S, per_seq - len(pick), replace=False).tolist())
        rows.append(np.array(sorted(pick)[:per_seq]))
    return rows


def gather_rows(arr, w, rows):
    off = w.seq_offsets
    idx = np.concatenate([off[b] + np.asarray(rows[b]) for b in range(w.num_seqs)])
    return arr[idx]


def compare(got, want, label, max_abs=MAX_ABS, mean_abs=MEAN_ABS, rel_l2=REL_L2):
    diff = np.abs(got - want)
    ma, me = float(diff.max()), float(diff.mean())
    rel = float(np.linalg.norm(got - want) / max(1e-30, np.linalg.norm(want)))
    say(f"{label}: max_abs={ma:.3e} mean_abs={me:.3e} rel_l2={rel:.3e} (n={got.size})")
    assert np.all(np.isfinite(got)), f"{label}: non-finite output"
    assert ma <= max_abs, f"{label}: max_abs {ma} > {max_abs}"
    assert me <= mean_abs, f"{label}: mean_abs {me} > {mean_abs}"
    assert rel <= rel_l2, f"{label}: rel_l2 {rel} > {rel_l2}"
    return ma, me, rel
