"""The library under HIP graph capture and on concurrent streams.

The entry points enqueue kernels on the caller's stream and allocate
nothing, so a serving loop can capture append + attention once and replay
it.  Each replay here is checked bit for bit against the eager result (the
kernels are deterministic), with the program's own eager work and
synchronisations between replays.  Two calls on two streams at once must
give the same bits as one after the other (the library keeps no state
between calls).
"""
import pytest

from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload

from gpu_common import say, stage

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _decode_inputs():
    w = build_workload(name="graph_decode", seed=881, prefix_len=[3000, 2100, 5000, 4095, 2048, 2600, 9000, 2500],
                       suffix_len=[1] * 8, num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                       num_blocks=4096)
    return w, stage(w)


@pytest.mark.timeout(300)
def test_append_and_decode_replay_from_a_graph():
    w, d = _decode_inputs()
    need = kvt.decode_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.num_q_heads)
    assert need > 0, "the key range is split, so the combine kernel is captured too"
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(d["q"])
    lse = torch.empty((w.total_tokens, w.num_q_heads), dtype=torch.float32, device="cuda")

    def step():
        kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
        kvt.decode_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.scale, out=out,
                             lse=lse, workspace=ws if need else None, use_workspace=need > 0)

    step()
    torch.cuda.synchronize()
    ref_out, ref_lse = out.clone(), lse.clone()
    say(f"decode graph: {w.num_seqs} sequences, workspace {need} bytes")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                                       # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        out.zero_()
        lse.zero_()
        torch.randn(1 << 20, device="cuda").sum()           # the program's own eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16)), f"replay {r}: out differs"
        assert torch.equal(lse, ref_lse), f"replay {r}: lse differs"
    del g


@pytest.mark.timeout(300)
def test_extend_replays_from_a_graph_and_runs_on_two_streams():
    w = build_workload(name="graph_extend", seed=882, prefix_len=[8000, 6000], suffix_len=[64, 32], num_q_heads=16,
                       num_kv_heads=4, head_dim=128, dtype="bf16", num_blocks=4096)
    d = stage(w)
    kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
    need = kvt.extend_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                                      w.num_q_heads)
    assert need > 0, "the key range is split, so the combine kernel is captured too"
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(d["q"])

    def run(o, wsb):
        kvt.extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, w.scale,
                             out=o, workspace=wsb if need else None, use_workspace=need > 0)

    run(out, ws)
    torch.cuda.synchronize()
    ref = out.clone()
    say(f"extend graph: workspace {need} bytes")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        run(out, ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(out, ws)
    for r in range(3):
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"replay {r} differs"
    del g
    # two streams at once, each with its own output and workspace
    out2 = torch.empty_like(out)
    ws2 = torch.empty_like(ws)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    out.zero_()
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            run(out, ws)
        with torch.cuda.stream(s2):
            run(out2, ws2)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert torch.equal(out2.view(torch.int16), ref.view(torch.int16))


@pytest.mark.timeout(300)
def test_explicit_stream_owns_the_buffers_the_binding_allocates():
    """``stream=`` for a stream other than the current one: the output, lse
    and split workspace the binding allocates belong to that stream, so
    allocations and writes on the current stream right after the call (before
    any synchronisation) cannot land on the workspace the kernels still use."""
    w = build_workload(name="stream_arg", seed=883, prefix_len=[8000, 6000], suffix_len=[64, 32], num_q_heads=16,
                       num_kv_heads=4, head_dim=128, dtype="bf16", num_blocks=4096)
    d = stage(w)
    kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
    need = kvt.extend_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                                      w.num_q_heads)
    assert need > 0, "the call is split, so the binding allocates a workspace"
    ref, ref_lse = kvt.extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len,
                                        w.suffix_len, w.scale, return_lse=True)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    for r in range(3):
        s.wait_stream(torch.cuda.current_stream())
        out, lse = kvt.extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len,
                                        w.suffix_len, w.scale, return_lse=True, stream=s)
        # the current stream allocates workspace-sized buffers and writes them at once
        junk = [torch.empty(need, dtype=torch.uint8, device="cuda") for _ in range(4)]
        for j in junk:
            j.fill_(0x7F)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"call {r}: out differs"
        assert torch.equal(lse, ref_lse), f"call {r}: lse differs"
        del junk, out, lse
