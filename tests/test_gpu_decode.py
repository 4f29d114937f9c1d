"""Decode step (``kvt_decode_attention``) against the fp64 oracle.

One new token per sequence is the suffix-of-one case of extend attention, so
the reference is ``oracle_extend`` with S_b = 1 on the pools ``oracle_append``
produced.  Covered: the 32-sequence decode batch (all rows, lse, split and
unsplit, run-to-run bit identity, agreement with the extend kernel), the
256-sequence batch (one launch: sampled sequences against the oracle, every
row of a needle batch against its target value), needle queries, and edge
shapes (a single key, page and tile boundaries, the largest and smallest
query groups, D = 64, fp32 storage, more sequences than one launch holds,
one long sequence split 16 ways).
"""
import numpy as np
import pytest

from oracle import oracle_append, oracle_extend
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload

from gpu_common import cached_config, compare, oracle_pools, run_append, run_extend, say, stage, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def run_decode(w, d, **kw):
    say(f"kvt_decode_attention {w.name}/{w.variant} {kw if kw else ''}")
    r = kvt.decode_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.scale, **kw)
    torch.cuda.synchronize()
    return r


@pytest.mark.timeout(900)
def test_decode_batch_matches_oracle():
    w = cached_config("decode_batch")
    d = stage(w)
    run_append(w, d)
    out, lse = run_decode(w, d, return_lse=True)
    kp, vp = oracle_pools("decode_batch")
    say(f"oracle over {w.num_seqs} sequences x {w.num_q_heads} heads")
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale)
    compare(to_f64(out, w.dtype), ref_o, "decode_batch out")
    compare(lse.cpu().numpy().astype(np.float64), ref_l, "decode_batch lse")
    again = run_decode(w, d)
    assert torch.equal(again.view(torch.int16), out.view(torch.int16)), "decode is not run-to-run deterministic"
    unsplit = run_decode(w, d, use_workspace=False)
    compare(to_f64(unsplit, w.dtype), ref_o, "decode_batch unsplit")
    ext = run_extend(w, d)
    compare(to_f64(ext, w.dtype), ref_o, "decode_batch through extend")
    del d
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_decode_batch256_in_one_launch():
    """256 sequences fit one launch's descriptors.  On the needle variant of
    the 256-sequence batch: 32 sampled sequences (every query head, out and
    lse) against the oracle, and every row against the value at its target
    position (a closed form that needs no oracle)."""
    from oracle import gather_logical
    w = cached_config("decode_batch256", "needle")
    d = stage(w)
    run_append(w, d)
    out, lse = run_decode(w, d, return_lse=True)
    got = to_f64(out, w.dtype)                                   # [256, Hq, D]
    kp, vp = oracle_pools("decode_batch256", "needle")
    pick = np.sort(np.random.default_rng(256).choice(w.num_seqs, 32, replace=False))
    chosen = set(pick.tolist())
    rows = [np.arange(1) if b in chosen else np.arange(0) for b in range(w.num_seqs)]
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale,
                                 rows=rows)
    compare(got[pick], ref_o, "decode_batch256 out (32 sequences)")
    compare(lse.cpu().numpy().astype(np.float64)[pick], ref_l, "decode_batch256 lse (32 sequences)")
    tgt, G = w.extra["needle_target"], w.group
    want = np.empty_like(got)
    for b in range(w.num_seqs):
        L = int(w.prefix_len[b]) + 1
        for g in range(w.num_kv_heads):
            v = gather_logical(vp, w.compact_table[b], L, g)
            want[b, g * G:(g + 1) * G] = v[tgt[b, g * G:(g + 1) * G]]
    compare(got, want, "decode_batch256 needle vs V[target] (every row)")
    del d
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_decode_needle_finds_every_page():
    """q = 2 K[t] for a random earlier position t: out ~ V[t], so a wrong page,
    slot or head mapping is an O(1) error."""
    w = build_workload(name="decode_needle", seed=731, prefix_len=[5000, 12000, 300, 77], suffix_len=[1, 1, 1, 1],
                       num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16", num_blocks=8192,
                       variant="needle")
    d = stage(w)
    run_append(w, d, checked=True)
    out = run_decode(w, d, checked=True)
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref, _ = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale)
    compare(to_f64(out, w.dtype), ref, "decode needle")
    assert np.mean(np.abs(ref)) > 0.5
    del d
    torch.cuda.empty_cache()


_rng = np.random.default_rng(770)
DEC_EDGE = [
    # (prefix lengths, Hq, Hkv, D, dtype)
    ([0], 4, 1, 64, "bf16"),                                   # a single key
    ([15, 16, 17, 31, 32, 33], 12, 1, 128, "bf16"),            # page and tile boundaries
    ([1000, 5, 2047], 32, 1, 128, "bf16"),                     # G = 32, the largest group
    ([300, 4097], 8, 8, 128, "bf16"),                          # G = 1
    ([4000, 100], 8, 2, 64, "f32"),                            # fp32 storage, D = 64
    (_rng.integers(0, 3000, size=70).tolist(), 12, 1, 128, "bf16"),   # 70 sequences, one launch
    ([20000], 12, 1, 128, "bf16"),                             # one sequence split 16 ways
    ([3, 9000, 64], 24, 2, 64, "bf16"),                        # D = 64, ragged
    (_rng.integers(0, 400, size=300).tolist(), 8, 2, 64, "bf16"),   # 300 sequences: two launches
]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", range(len(DEC_EDGE)))
def test_decode_edge_shapes(case):
    P, Hq, Hkv, D, dt = DEC_EDGE[case]
    pages = sum((p + 1 + 15) // 16 for p in P)
    w = build_workload(name=f"dec_edge{case}", seed=700 + case, prefix_len=P, suffix_len=[1] * len(P),
                       num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype=dt, num_blocks=max(4096, 2 * pages))
    d = stage(w)
    run_append(w, d, checked=True)
    out, lse = run_decode(w, d, return_lse=True, checked=True)
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, Hkv, w.scale)
    compare(to_f64(out, dt), ref_o, f"dec_edge{case} out")
    compare(lse.cpu().numpy().astype(np.float64), ref_l, f"dec_edge{case} lse")
    del d
    torch.cuda.empty_cache()
