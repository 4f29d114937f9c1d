"""Seeded random shapes through the C-ABI against the fp64 oracle.

Each case draws a batch (1-6 sequences, reused prefixes 0-2500 positions,
1-200 new tokens each), a head layout (1-8 kv-heads, 1-16 query heads per
kv-head), the head size (64 or 128), the storage type (bf16, sometimes fp32)
and a pool with spare pages, then checks:

* append: bit-exact K and V pages (checked mode);
* extend: output and lse against the oracle, with the planned key splits
  (workspace) and without them (no workspace);
* cascade extend, for cases drawn with a shared prefix;
* decode, for cases drawn with one new token per sequence.

A second, wider set draws up to 12 sequences, prefixes up to 4000 positions,
shared prefixes up to 119 pages and 1-24 query heads per kv-head (new tokens
scaled so the oracle's work per case stays bounded).
"""
import numpy as np
import pytest

from oracle import oracle_append, oracle_extend
from paper_2609_39819_amd import kvt
from paper_2609_39819_amd.workloads import build_workload, torch_to_np

from gpu_common import compare, say, stage, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

N_CASES = 48


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def draw(case: int) -> dict:
    rng = np.random.default_rng(9000 + case)
    B = int(rng.integers(1, 7))
    kind = ("decode" if case % 6 == 5 else "shared" if case % 6 == 2 else "plain")
    hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16]))
    D = int(rng.choice([64, 128]))
    dtype = "f32" if rng.random() < 0.2 else "bf16"
    sh = 0
    if kind == "decode":
        P = rng.integers(0, 2500, B)
        S = np.ones(B, dtype=np.int64)
    elif kind == "shared":
        sh = int(rng.integers(1, 40))                     # shared pages (16 positions each)
        P = sh * 16 + rng.integers(0, 1500, B)
        S = rng.integers(1, 200, B)
    else:
        P = rng.integers(0, 2500, B)
        S = rng.integers(1, 200, B)
    return dict(kind=kind, B=B, P=[int(x) for x in P], S=[int(x) for x in S], hkv=hkv, G=G, D=D, dtype=dtype,
                shared_blocks=sh, extra_pages=int(rng.integers(0, 300)))


def draw_wide(case: int) -> dict:
    rng = np.random.default_rng(20000 + case)
    B = int(rng.integers(1, 13))
    kind = ("decode" if case % 5 == 4 else "shared" if case % 5 == 2 else "plain")
    hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 3, 5, 7, 8, 12, 16, 24]))
    D = int(rng.choice([64, 128]))
    dtype = "f32" if rng.random() < 0.2 else "bf16"
    sh = 0
    smax = max(2, 2400 // (B * G * hkv))
    if kind == "decode":
        P = rng.integers(0, 4000, B)
        S = np.ones(B, dtype=np.int64)
    elif kind == "shared":
        sh = int(rng.integers(1, 120))
        P = sh * 16 + rng.integers(0, 2500, B)
        S = rng.integers(1, smax + 1, B)
    else:
        P = rng.integers(0, 4000, B)
        S = rng.integers(1, smax + 1, B)
    return dict(kind=kind, B=B, P=[int(x) for x in P], S=[int(x) for x in S], hkv=hkv, G=G, D=D, dtype=dtype,
                shared_blocks=sh, extra_pages=int(rng.integers(0, 300)))


CASES = [draw(c) for c in range(N_CASES)]
N_WIDE = 100
WIDE = [draw_wide(c) for c in range(N_WIDE)]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", range(N_CASES))
def test_random_shape(case):
    check(CASES[case], f"rand{case}", 9100 + case)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", range(N_WIDE))
def test_random_wide_shape(case):
    check(WIDE[case], f"wide{case}", 21000 + case)


def check(c, case, seed):
    say(f"random case {case}: {c}")
    L = np.asarray(c["P"]) + np.asarray(c["S"])
    pages = int(c["shared_blocks"] + ((L + 15) // 16 - c["shared_blocks"]).sum())
    w = build_workload(name=case, seed=seed, prefix_len=c["P"], suffix_len=c["S"],
                       num_q_heads=c["G"] * c["hkv"], num_kv_heads=c["hkv"], head_dim=c["D"], dtype=c["dtype"],
                       num_blocks=pages + c["extra_pages"], shared_prefix_blocks=c["shared_blocks"])
    d = stage(w)
    kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"],
                  checked=True)
    torch.cuda.synchronize()
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)
    ids = torch.from_numpy(w.phys_ids).cuda()
    for name, dev, ref in (("k", d["k_pool"], kp), ("v", d["v_pool"], vp)):
        got = torch_to_np(dev.index_select(0, ids), w.dtype)
        assert np.array_equal(got.view(np.uint8), np.ascontiguousarray(ref).view(np.uint8)), f"{name} pages differ"
    ref_o, ref_l = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale)
    args = (d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len)

    if c["kind"] == "decode" and c["G"] <= 32:
        out, lse = kvt.decode_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.scale,
                                        return_lse=True, checked=True)
        torch.cuda.synchronize()
        compare(to_f64(out, w.dtype), ref_o, f"{case} decode out")
        compare(lse.cpu().numpy().astype(np.float64), ref_l, f"{case} decode lse")

    for use_ws in (True, False):
        out, lse = kvt.extend_attention(*args, w.scale, return_lse=True, use_workspace=use_ws, checked=True)
        torch.cuda.synchronize()
        tag = "split plan" if use_ws else "unsplit"
        compare(to_f64(out, w.dtype), ref_o, f"{case} extend ({tag}) out")
        compare(lse.cpu().numpy().astype(np.float64), ref_l, f"{case} extend ({tag}) lse")

    if c["kind"] == "shared":
        out, lse = kvt.cascade_extend_attention(*args, c["shared_blocks"] * 16, w.scale, return_lse=True,
                                                mode=kvt.CASCADE_SHARED_PASS,
                                                checked=True)
        torch.cuda.synchronize()
        compare(to_f64(out, w.dtype), ref_o, f"{case} cascade out")
        compare(lse.cpu().numpy().astype(np.float64), ref_l, f"{case} cascade lse")
    del d
    torch.cuda.empty_cache()
