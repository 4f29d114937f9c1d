"""Cascade extend (``kvt_cascade_extend_attention[_ex]``) against the fp64 oracle.

The cascade computes the same attention as extend (shared keys for the whole
batch at once, private keys per sequence, log-sum-exp merge), so the
reference is ``oracle_extend``.  In its default mode the call runs the plain
extend plan whenever the library's estimate says the shared pass loses; the
tests check that choice where it is clear-cut (the forked-agents workload:
plain, bit-identical to ``kvt_extend_attention``; short messages over a long
shared prefix: the shared pass) and force the shared pass on the
forked-agents workload and on edge shapes (a shared length that is not a
multiple of the 64-key tile, a sequence whose whole prefix is shared, a
single sequence, D = 64, fp32 storage, key splits in the private parts),
which are too small for it to win on its own), and check that on the edge
shapes the default mode gives the bits of the plan it reports.
"""
import numpy as np
import pytest

from oracle import oracle_append, oracle_extend
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload, config_shapes

from gpu_common import (cached_config, compare, gather_rows, oracle_pools, run_append, run_extend, sample_rows, say,
                        stage, to_f64)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def run_cascade(w, d, shared, **kw):
    say(f"kvt_cascade_extend_attention {w.name}/{w.variant} shared={shared} {kw if kw else ''}")
    r = kvt.cascade_extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len,
                                     w.suffix_len, shared, w.scale, **kw)
    torch.cuda.synchronize()
    return r


def uses_shared(w, d, shared):
    return kvt.cascade_uses_shared_pass(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                                        shared, w.num_q_heads)


@pytest.mark.timeout(900)
def test_forked_agents_default_runs_the_plain_plan():
    """Long suffixes: the estimate picks the plain extend plan, so the cascade
    call gives exactly the bits of kvt_extend_attention."""
    w = cached_config("forked_agents")
    shared = config_shapes("forked_agents")["shared_prefix"]
    d = stage(w)
    run_append(w, d)
    assert not uses_shared(w, d, shared)
    out, lse = run_cascade(w, d, shared, return_lse=True)
    plain, plain_lse = run_extend(w, d, return_lse=True)
    assert torch.equal(out.view(torch.int16), plain.view(torch.int16))
    assert torch.equal(lse, plain_lse)
    del d
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_forked_agents_shared_pass_matches_oracle():
    w = cached_config("forked_agents")
    shared = config_shapes("forked_agents")["shared_prefix"]
    d = stage(w)
    run_append(w, d)
    out, lse = run_cascade(w, d, shared, return_lse=True, mode=kvt.CASCADE_SHARED_PASS)
    rows = sample_rows(w, 6)
    kp, vp = oracle_pools("forked_agents")
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale,
                                 rows=rows)
    compare(gather_rows(to_f64(out, w.dtype), w, rows), ref_o, "forked cascade out")
    compare(gather_rows(lse.cpu().numpy().astype(np.float64), w, rows), ref_l, "forked cascade lse")
    assert bool(torch.isfinite(out.float()).all())
    plain = run_extend(w, d)
    compare(to_f64(out, w.dtype), to_f64(plain, w.dtype), "cascade vs extend", max_abs=1e-2, mean_abs=5e-4)
    del d
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_short_messages_over_a_long_shared_prefix():
    """16 sub-agents adding 16 tokens each over 32768 shared positions: the
    shared pass runs with its own key splits."""
    w = cached_config("forked_short")
    shared = config_shapes("forked_short")["shared_prefix"]
    d = stage(w)
    run_append(w, d)
    assert uses_shared(w, d, shared), "short messages over a long shared prefix take the shared pass by default"
    out, lse = run_cascade(w, d, shared, return_lse=True)
    rows = sample_rows(w, 8)
    kp, vp = oracle_pools("forked_short")
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale,
                                 rows=rows)
    compare(gather_rows(to_f64(out, w.dtype), w, rows), ref_o, "forked_short cascade out")
    compare(gather_rows(lse.cpu().numpy().astype(np.float64), w, rows), ref_l, "forked_short cascade lse")
    plain = run_extend(w, d)
    compare(to_f64(out, w.dtype), to_f64(plain, w.dtype), "cascade vs extend", max_abs=1e-2, mean_abs=5e-4)
    del d
    torch.cuda.empty_cache()


_casc_rng = np.random.default_rng(77)
CASC_EDGE = [
    # (prefix lengths, suffix lengths, shared, Hq, Hkv, D, dtype)
    ([200, 500, 96], [40, 300, 7], 48, 12, 1, 128, "bf16"),          # shared not a multiple of 64
    ([4096, 6000], [100, 2048], 4096, 12, 2, 128, "bf16"),            # one prefix entirely shared
    ([9000], [513], 1024, 8, 2, 128, "bf16"),                         # a single sequence
    ([3000, 2000, 2500], [64, 65, 63], 1600, 16, 8, 64, "bf16"),      # D = 64
    ([700, 900], [33, 40], 320, 4, 1, 64, "f32"),                     # fp32 storage
    ([40000, 33000], [16, 20], 16384, 8, 8, 128, "bf16"),             # short suffixes: private parts split
    # 300 sequences: the shared part and 255 private parts in the first
    # launch, the other 45 private parts in a second
    ((64 + _casc_rng.integers(0, 400, size=300)).tolist(), _casc_rng.integers(1, 9, size=300).tolist(), 64, 4, 2, 64,
     "bf16"),
]
# the default mode's choice for each shape (the host estimate's)
CASC_EDGE_AUTO_SHARED = [True, False, True, True, True, True, True]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", range(len(CASC_EDGE)))
def test_cascade_edge_shapes(case):
    P, S, shared, Hq, Hkv, D, dt = CASC_EDGE[case]
    w = build_workload(name=f"casc_edge{case}", seed=800 + case, prefix_len=P, suffix_len=S, num_q_heads=Hq,
                       num_kv_heads=Hkv, head_dim=D, dtype=dt, num_blocks=16384, shared_prefix_blocks=shared // 16)
    d = stage(w)
    run_append(w, d, checked=True)
    out, lse = run_cascade(w, d, shared, return_lse=True, checked=True, mode=kvt.CASCADE_SHARED_PASS)
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, Hkv, w.scale)
    compare(to_f64(out, dt), ref_o, f"casc_edge{case} out")
    compare(lse.cpu().numpy().astype(np.float64), ref_l, f"casc_edge{case} lse")
    # the default mode runs the plan it reports, bit for bit: the shared
    # pass where short suffixes meet a prefix mostly shared (or where the
    # plain extend cannot split), the plain extend for the one shape with a
    # long suffix
    assert uses_shared(w, d, shared) == CASC_EDGE_AUTO_SHARED[case]
    auto = run_cascade(w, d, shared, checked=True)
    same_plan = out if CASC_EDGE_AUTO_SHARED[case] else run_extend(w, d, checked=True)
    assert torch.equal(auto.view(torch.int16 if dt == "bf16" else torch.int32),
                       same_plan.view(torch.int16 if dt == "bf16" else torch.int32))
    del d
    torch.cuda.empty_cache()
