"""Invariants of extend attention, checked on the GPU through the C-ABI.

* paging relabel: moving every page to another physical id and rewriting the
  block table to match leaves out and lse bit-identical, split and unsplit
  (the kernels' arithmetic depends on the logical sequence only);
* reuse = recompute: extend(P, S) gives the last S rows of extend(0, P + S)
  over the same K/V (the premise of prefix reuse, paper §1, §2.2), each
  within the parity tolerance of the oracle and of each other;
* chunked turns: append + extend(P, S1), then append + extend(P + S1, S2),
  leave the same pool bytes as one append of S1 + S2 tokens and give the rows
  of extend(P, S1 + S2) within tolerance;
* fork sharing: sequences that share their first pages (a forked context,
  §5.2, §6.1) give bit-identical results to the same batch with private
  copies of those pages;
* the decoding step obeys the first and last of these as well.
"""
import numpy as np
import pytest

from oracle import oracle_append, oracle_extend
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload

from gpu_common import compare, say, stage, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def pages_needed(P, S, shared_blocks=0):
    L = np.asarray(P) + np.asarray(S)
    return int(shared_blocks + ((L + 15) // 16 - shared_blocks).sum())


def bits(t):
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)


def extend(d, w, q=None, prefix=None, suffix=None, pools=None, table=None, **kw):
    kp, vp = pools if pools is not None else (d["k_pool"], d["v_pool"])
    r = kvt.extend_attention(d["q"] if q is None else q, kp, vp, d["block_table"] if table is None else table,
                             w.prefix_len if prefix is None else prefix, w.suffix_len if suffix is None else suffix,
                             w.scale, return_lse=True, checked=True, **kw)
    torch.cuda.synchronize()
    return r


def append(d, w, prefix, suffix, k_new, v_new):
    kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], prefix, suffix, k_new, v_new, checked=True)
    torch.cuda.synchronize()


@pytest.mark.timeout(300)
def test_paging_relabel_is_bit_identical():
    P, S = [3000, 517, 64], [300, 45, 1]
    w = build_workload(name="relabel", seed=9301, prefix_len=P, suffix_len=S, num_q_heads=16, num_kv_heads=4,
                       head_dim=128, dtype="bf16", num_blocks=pages_needed(P, S) + 500)
    d = stage(w)
    append(d, w, w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
    perm = torch.randperm(w.num_blocks, generator=torch.Generator().manual_seed(9301)).to("cuda")
    k2 = torch.empty_like(d["k_pool"]).index_copy_(0, perm, d["k_pool"])    # page i moves to perm[i]
    v2 = torch.empty_like(d["v_pool"]).index_copy_(0, perm, d["v_pool"])
    bt = d["block_table"]
    bt2 = torch.where(bt >= 0, perm[bt.clamp(min=0).long()].to(torch.int32), bt).contiguous()
    for use_ws in (True, False):
        o1, l1 = extend(d, w, use_workspace=use_ws)
        o2, l2 = extend(d, w, pools=(k2, v2), table=bt2, use_workspace=use_ws)
        say(f"relabel, {'split plan' if use_ws else 'unsplit'}: comparing bits")
        assert torch.equal(bits(o1), bits(o2)), "output changed under a page relabelling"
        assert torch.equal(bits(l1), bits(l2)), "lse changed under a page relabelling"


@pytest.mark.timeout(300)
def test_prefix_reuse_equals_full_recompute():
    P, S = 1500, 200
    w = build_workload(name="recompute", seed=9302, prefix_len=[0], suffix_len=[P + S], num_q_heads=24,
                       num_kv_heads=2, head_dim=128, dtype="bf16", num_blocks=pages_needed([0], [P + S]) + 40)
    d = stage(w)
    append(d, w, w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
    o_full, l_full = extend(d, w)
    o_ext, l_ext = extend(d, w, q=d["q"][P:], prefix=[P], suffix=[S])
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, [0], [P + S], w.k_new, w.v_new)
    ref, ref_l = oracle_extend(w.q[P:], kp, vp, w.compact_table, [P], [S], w.num_kv_heads, w.scale)
    compare(to_f64(o_ext, w.dtype), ref, "extend(P, S) vs oracle")
    compare(to_f64(o_full[P:], w.dtype), ref, "last S rows of extend(0, P+S) vs oracle")
    compare(to_f64(o_ext, w.dtype), to_f64(o_full[P:], w.dtype), "reuse vs recompute", max_abs=1e-2,
            mean_abs=5e-4)
    compare(l_ext.cpu().numpy().astype(np.float64), ref_l, "extend(P, S) lse vs oracle")
    compare(l_full[P:].cpu().numpy().astype(np.float64), ref_l, "recompute lse vs oracle")


@pytest.mark.timeout(300)
def test_chunked_turns_equal_one_turn():
    P, S1, S2 = 777, 130, 95              # every boundary falls inside a page
    w = build_workload(name="chunked", seed=9303, prefix_len=[P], suffix_len=[S1 + S2], num_q_heads=8,
                       num_kv_heads=1, head_dim=128, dtype="bf16", num_blocks=pages_needed([P], [S1 + S2]) + 30)
    one = stage(w)
    append(one, w, w.prefix_len, w.suffix_len, one["k_new"], one["v_new"])
    o_one, _ = extend(one, w)
    two = stage(w)
    append(two, w, [P], [S1], two["k_new"][:S1], two["v_new"][:S1])
    o_a, _ = extend(two, w, q=two["q"][:S1], prefix=[P], suffix=[S1])
    append(two, w, [P + S1], [S2], two["k_new"][S1:], two["v_new"][S1:])
    o_b, _ = extend(two, w, q=two["q"][S1:], prefix=[P + S1], suffix=[S2])
    say("chunked turns: comparing pool bytes")
    assert torch.equal(bits(one["k_pool"]), bits(two["k_pool"])), "K pages differ between one and two appends"
    assert torch.equal(bits(one["v_pool"]), bits(two["v_pool"])), "V pages differ between one and two appends"
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref, _ = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale)
    two_turns = to_f64(torch.cat([o_a, o_b]), w.dtype)
    compare(two_turns, ref, "two turns vs oracle")
    compare(to_f64(o_one, w.dtype), ref, "one turn vs oracle")
    compare(two_turns, to_f64(o_one, w.dtype), "two turns vs one turn", max_abs=1e-2, mean_abs=5e-4)


@pytest.mark.timeout(300)
def test_fork_sharing_is_bit_identical_to_private_copies():
    sh = 64                                # shared pages = 1024 positions
    P, S = [2000, 2300, 1800, 1024], [120, 64, 200, 7]
    w = build_workload(name="forks", seed=9304, prefix_len=P, suffix_len=S, num_q_heads=12, num_kv_heads=2,
                       head_dim=128, dtype="bf16", shared_prefix_blocks=sh,
                       num_blocks=pages_needed(P, S, sh) + 3 * sh + 20)
    d = stage(w)
    append(d, w, w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
    bt = w.block_table.copy()
    assert all(np.array_equal(bt[b, :sh], bt[0, :sh]) for b in range(len(P))), "workload lost its shared pages"
    used = set(bt[bt >= 0].tolist())
    free = [i for i in range(w.num_blocks) if i not in used]
    k2, v2 = d["k_pool"].clone(), d["v_pool"].clone()
    for b in range(1, len(P)):             # sequences 1.. get private copies of the shared pages
        fresh = np.asarray(free[(b - 1) * sh:b * sh], dtype=np.int64)
        src = torch.from_numpy(bt[b, :sh].astype(np.int64)).to("cuda")
        dst = torch.from_numpy(fresh).to("cuda")
        k2.index_copy_(0, dst, d["k_pool"].index_select(0, src))
        v2.index_copy_(0, dst, d["v_pool"].index_select(0, src))
        bt[b, :sh] = fresh
    bt2 = torch.from_numpy(bt).to("cuda")
    for use_ws in (True, False):
        o1, l1 = extend(d, w, use_workspace=use_ws)
        o2, l2 = extend(d, w, pools=(k2, v2), table=bt2, use_workspace=use_ws)
        say(f"fork sharing, {'split plan' if use_ws else 'unsplit'}: comparing bits")
        assert torch.equal(bits(o1), bits(o2)), "shared pages and private copies give different outputs"
        assert torch.equal(bits(l1), bits(l2)), "shared pages and private copies give different lse"
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref, _ = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale)
    compare(to_f64(o1, w.dtype), ref, "forked batch vs oracle")


@pytest.mark.timeout(300)
def test_decode_is_invisible_to_paging_and_fork_sharing():
    """One decoding step (one new token per sequence, key splits over the
    long contexts): relabelling every page, and private copies of a shared
    prefix, leave out and lse bit-identical."""
    sh = 32
    P, S = [6000, 2700, 3333, 2048], [1, 1, 1, 1]     # >= 2048 keys each: two key splits
    w = build_workload(name="decode-inv", seed=9305, prefix_len=P, suffix_len=S, num_q_heads=32, num_kv_heads=4,
                       head_dim=128, dtype="bf16", shared_prefix_blocks=sh,
                       num_blocks=pages_needed(P, S, sh) + 3 * sh + 50)
    d = stage(w)
    append(d, w, w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])

    def decode(pools=None, table=None):
        kp, vp = pools if pools is not None else (d["k_pool"], d["v_pool"])
        r = kvt.decode_attention(d["q"], kp, vp, d["block_table"] if table is None else table, w.prefix_len,
                                 w.scale, return_lse=True, checked=True)
        torch.cuda.synchronize()
        return r

    o1, l1 = decode()
    perm = torch.randperm(w.num_blocks, generator=torch.Generator().manual_seed(9305)).to("cuda")
    k2 = torch.empty_like(d["k_pool"]).index_copy_(0, perm, d["k_pool"])
    v2 = torch.empty_like(d["v_pool"]).index_copy_(0, perm, d["v_pool"])
    bt = d["block_table"]
    bt2 = torch.where(bt >= 0, perm[bt.clamp(min=0).long()].to(torch.int32), bt).contiguous()
    o2, l2 = decode(pools=(k2, v2), table=bt2)
    say("decode relabel: comparing bits")
    assert torch.equal(bits(o1), bits(o2)) and torch.equal(bits(l1), bits(l2)), "decode changed under a relabelling"

    host = w.block_table.copy()
    used = set(host[host >= 0].tolist())
    free = [i for i in range(w.num_blocks) if i not in used]
    k3, v3 = d["k_pool"].clone(), d["v_pool"].clone()
    for b in range(1, len(P)):
        fresh = np.asarray(free[(b - 1) * sh:b * sh], dtype=np.int64)
        src = torch.from_numpy(host[b, :sh].astype(np.int64)).to("cuda")
        dst = torch.from_numpy(fresh).to("cuda")
        k3.index_copy_(0, dst, d["k_pool"].index_select(0, src))
        v3.index_copy_(0, dst, d["v_pool"].index_select(0, src))
        host[b, :sh] = fresh
    o3, l3 = decode(pools=(k3, v3), table=torch.from_numpy(host).to("cuda"))
    say("decode fork sharing: comparing bits")
    assert torch.equal(bits(o1), bits(o3)) and torch.equal(bits(l1), bits(l3)), "decode differs on private copies"
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ref, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale)
    compare(to_f64(o1, w.dtype), ref, "decode vs oracle")
    compare(l1.cpu().numpy().astype(np.float64), ref_l, "decode lse vs oracle")
