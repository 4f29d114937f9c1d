"""Page moves between the HBM pools and pinned host memory
(``kvt_copy_blocks``) against the oracle: bit-exact, both directions."""
import numpy as np
import pytest

from oracle import oracle_to_device, oracle_to_host
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload, stage_on_device, torch_to_np

from gpu_common import say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _pinned_like(shape, dtype):
    return torch.empty(shape, dtype=dtype, pin_memory=True)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("hkv,d,dt,n", [(8, 128, "bf16", 1000), (1, 64, "f32", 37), (2, 128, "bf16", 1)])
def test_offload_and_reload_are_bit_exact(hkv, d, dt, n):
    w = build_workload(name="copy", seed=900 + n, prefix_len=[n * 16 + 5], suffix_len=[1], num_q_heads=hkv,
                       num_kv_heads=hkv, head_dim=d, dtype=dt, num_blocks=4 * n + 64)
    dev = stage_on_device(w, "cuda")
    kp, vp = dev["k_pool"], dev["v_pool"]
    rng = np.random.default_rng(n)
    ids = rng.permutation(w.num_blocks)[:n].astype(np.int32)          # used and unused pages, any order
    ids_d = torch.from_numpy(ids).cuda()
    host = _pinned_like((n, 2) + tuple(kp.shape[1:]), kp.dtype)
    say(f"offload {n} pages of {hkv}x16x{d} {dt}")
    kvt.copy_blocks(kp, vp, ids_d, host, to_host=True, checked=True)
    torch.cuda.synchronize()
    k_np, v_np = torch_to_np(kp, dt), torch_to_np(vp, dt)
    want = oracle_to_host(k_np, v_np, ids)
    got = torch_to_np(host, dt)
    assert np.array_equal(got.view(np.uint8), want.view(np.uint8))
    # reload the pages, shifted, into other pages of the pool
    dst = np.roll(ids, 1).astype(np.int32)
    say(f"reload {n} pages")
    kvt.copy_blocks(kp, vp, torch.from_numpy(dst).cuda(), host, to_host=False, checked=True)
    torch.cuda.synchronize()
    k_want, v_want = oracle_to_device(k_np, v_np, dst, want)
    assert np.array_equal(torch_to_np(kp, dt).view(np.uint8), k_want.view(np.uint8))
    assert np.array_equal(torch_to_np(vp, dt).view(np.uint8), v_want.view(np.uint8))


@pytest.mark.timeout(120)
def test_out_of_pool_ids_are_skipped_unchecked():
    w = build_workload(name="copy_oob", seed=950, prefix_len=[100], suffix_len=[1], num_q_heads=2, num_kv_heads=2,
                       head_dim=64, dtype="bf16", num_blocks=32)
    dev = stage_on_device(w, "cuda")
    kp, vp = dev["k_pool"], dev["v_pool"]
    ids = torch.tensor([3, 32, 7, 1 << 30], dtype=torch.int32, device="cuda")
    host = _pinned_like((4, 2) + tuple(kp.shape[1:]), kp.dtype)
    host.zero_()
    kvt.copy_blocks(kp, vp, ids, host, to_host=True)
    torch.cuda.synchronize()
    k_np = torch_to_np(kp, "bf16")
    got = torch_to_np(host, "bf16")
    assert np.array_equal(got[0, 0], k_np[3]) and np.array_equal(got[2, 0], k_np[7])
    assert not got[1].any() and not got[3].any()                       # skipped: host untouched
