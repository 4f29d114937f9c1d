"""The C ABI from a native program: ``tests/kvt_run`` (built with the library
from ``tests/kvt_run.cpp``) allocates with hipMalloc, calls kvt_append_kv and
kvt_extend_attention in checked mode and writes out and lse; its results are
compared with the fp64 oracle.  No Python or torch is in that process, so
the library's contract (plain pointers, caller-owned memory, the caller's
stream) is exercised as a C or C++ caller would."""
import os
import subprocess

import numpy as np
import pytest

from oracle import oracle_append, oracle_extend, storage_to_f64
from paper_2609_39819_amd.workloads import build_workload

from gpu_common import compare, say

pytestmark = pytest.mark.gpu

RUNNER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "kvt_run")


def _write_input(path, w):
    with open(path, "wb") as f:
        np.array([w.num_seqs, w.num_q_heads, w.num_kv_heads, w.head_dim, w.num_blocks, w.block_table.shape[1]],
                 dtype=np.int32).tofile(f)
        np.array([w.scale], dtype=np.float32).tofile(f)
        np.asarray(w.prefix_len, dtype=np.int32).tofile(f)
        np.asarray(w.suffix_len, dtype=np.int32).tofile(f)
        np.ascontiguousarray(w.block_table, dtype=np.int32).tofile(f)
        for compact in (w.k_pool_c, w.v_pool_c):           # full pools: NaN except the used pages
            pool = np.full((w.num_blocks,) + compact.shape[1:], 0x7FC0, dtype=np.uint16)
            pool[w.phys_ids] = compact
            pool.tofile(f)
        for a in (w.k_new, w.v_new, w.q):
            np.ascontiguousarray(a, dtype=np.uint16).tofile(f)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", [
    ([2000, 0, 333], [100, 17, 1], 12, 2, 128),      # ragged, with a sequence of one new token
    ([5000], [2], 8, 8, 64),                           # D = 64, G = 1; short suffix: split key range
])
def test_native_caller_matches_oracle(tmp_path, case):
    if not os.path.exists(RUNNER):
        pytest.fail(f"{RUNNER} is missing: build with `python -m paper_2609_39819_amd.build`")
    P, S, Hq, Hkv, D = case
    w = build_workload(name="native", seed=930 + D, prefix_len=P, suffix_len=S, num_q_heads=Hq, num_kv_heads=Hkv,
                       head_dim=D, dtype="bf16", num_blocks=1024)
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_input(inp, w)
    say(f"kvt_run: P={P} S={S} Hq={Hq} Hkv={Hkv} D={D}")
    r = subprocess.run([RUNNER, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    say(r.stdout.strip(), r.stderr.strip())
    assert r.returncode == 0, r.stderr
    T = int(np.sum(S))
    raw = np.fromfile(outp, dtype=np.uint8)
    out = raw[:T * Hq * D * 2].view(np.uint16).reshape(T, Hq, D)
    lse = raw[T * Hq * D * 2:].view(np.float32).reshape(T, Hq)
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, Hkv, w.scale)
    compare(storage_to_f64(out), ref_o, "native out")
    compare(lse.astype(np.float64), ref_l, "native lse")
