"""kvt_extend_attention_noalloc against kvt_extend_attention (GPU).

Two calls in a row through the C ABI, the second with a smaller input, each
split over key ranges so that its partial results live in the library's
static scratch: out and lse must be bit-identical to kvt_extend_attention
with a caller workspace (same plan, same kernels), and within the parity
bounds of the fp64 oracle.  The second call finds the first call's partials
in the scratch and must not be affected by them.
"""
import numpy as np
import pytest

from oracle import oracle_append, oracle_extend
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload

from gpu_common import compare, say, stage, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = [
    # (P, S, Hq, Hkv): 8K GQA shape (4 key splits, 34 MB of partials), then a
    # smaller ragged two-sequence batch (fewer rows, other split count)
    ([8192], [512], 32, 8),
    ([6000, 4100], [100, 37], 16, 4),
]


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


@pytest.mark.timeout(300)
def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    for i, (P, S, Hq, Hkv) in enumerate(CASES):
        w = build_workload(name=f"noalloc{i}", seed=990 + i, prefix_len=P, suffix_len=S, num_q_heads=Hq,
                           num_kv_heads=Hkv, head_dim=128, dtype="bf16", num_blocks=8192)
        d = stage(w)
        kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
        need = kvt.extend_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                                          Hq)
        say(f"noalloc call {i}: P={P} S={S} Hq={Hq} Hkv={Hkv}, partials {need} bytes")
        assert 0 < need <= kvt.NOALLOC_SCRATCH_BYTES, "the call is split and its partials fit the scratch"
        ref, ref_lse = kvt.extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len,
                                            w.suffix_len, w.scale, return_lse=True)
        out = torch.full_like(d["q"], float("nan"))
        lse = torch.full((w.total_tokens, Hq), float("nan"), dtype=torch.float32, device="cuda")
        kvt.extend_attention_noalloc(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len,
                                     w.suffix_len, w.scale, out=out, lse=lse)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"call {i}: out differs"
        assert torch.equal(lse, ref_lse), f"call {i}: lse differs"
        kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new,
                               w.v_new)
        ro, rl = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, Hkv, w.scale)
        compare(to_f64(out, w.dtype), ro, f"noalloc call {i} out")
        compare(lse.cpu().numpy().astype(np.float64), rl, f"noalloc call {i} lse")
        del d
        torch.cuda.empty_cache()
