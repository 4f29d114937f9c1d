"""Pins for the fp64 oracle (CPU only).

Each test ties ``oracle/`` to something other than itself: hand-derived closed
forms, pure-Python brute force over the un-paged sequence, a library routine
(torch's causal SDPA in fp64, scipy's logsumexp), closed forms of degenerate
inputs, and invariants the definition implies (prefix reuse equals recompute,
paging independence, head-group sharing).  A few tests plant a mistake in the
oracle's inputs to show the pins have teeth.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import brute_force_extend, oracle_append, oracle_extend, storage_to_f64, gather_logical
from paper_2609_39819_amd.workloads import build_workload, bf16_bits_to_f32

HERE = os.path.dirname(os.path.abspath(__file__))


def _pool_f64_view(w):
    return w.k_pool_c, w.v_pool_c


def _appended(w):
    """Compact pools after the oracle writes the suffix K/V."""
    return oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)


def _oracle(w, **kw):
    kp, vp = _appended(w)
    return oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale, **kw)


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(1e-300, np.max(np.abs(b)))


# ---------------------------------------------------------------------------
# hand-derived closed forms
# ---------------------------------------------------------------------------

def _eval(expr):
    return eval(expr, {"__builtins__": {}}, {"e": math.e, "log": math.log, "exp": math.exp})


def test_hand_cases():
    with open(os.path.join(HERE, "golden", "hand_cases.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        P, S, Hq, Hkv = c["prefix_len"], c["suffix_len"], c["num_q_heads"], c["num_kv_heads"]
        k = np.array(c["k"], dtype=np.float32)
        D = k.shape[-1]
        k = k.reshape(P + S, Hkv, D)
        v = np.array(c["v"], dtype=np.float32).reshape(P + S, Hkv, D)
        q = np.array(c["q"], dtype=np.float32).reshape(S, Hq, D)
        want_out = np.vectorize(_eval, otypes=[float])(np.array(c["out"], dtype=object)).reshape(S, Hq, D)
        want_lse = np.vectorize(_eval, otypes=[float])(np.array(c["lse"], dtype=object)).reshape(S, Hq)
        # page it by hand: one block, physical id 3 of a 5-block NaN pool
        kp = np.full((5, Hkv, 16, D), np.nan, np.float32)
        vp = np.full((5, Hkv, 16, D), np.nan, np.float32)
        kp[3, :, :P, :] = k[:P].transpose(1, 0, 2)
        vp[3, :, :P, :] = v[:P].transpose(1, 0, 2)
        bt = np.array([[3]], dtype=np.int32)
        kp, vp = oracle_append(kp, vp, bt, [P], [S], k[P:], v[P:])
        out, lse = oracle_extend(q, kp, vp, bt, [P], [S], Hkv, c["scale"])
        assert np.allclose(out, want_out, rtol=1e-14, atol=1e-14), c["name"]
        assert np.allclose(lse, want_lse, rtol=1e-14, atol=1e-14), c["name"]
        bo, bl = brute_force_extend(q, [k], [v], [P], [S], Hkv, c["scale"])
        assert np.allclose(bo, want_out, rtol=1e-14, atol=1e-14), c["name"]
        assert np.allclose(bl, want_lse, rtol=1e-14, atol=1e-14), c["name"]


# ---------------------------------------------------------------------------
# brute force over the un-paged logical sequence
# ---------------------------------------------------------------------------

SWEEP = [
    # (P list, S list, Hq, Hkv, D, dtype)
    ([p], [s], 4, 1, 8, "bf16") for p in (0, 1, 15, 16, 17, 33) for s in (1, 5, 16, 40)
] + [
    ([17, 0, 33], [5, 16, 1], 12, 1, 8, "bf16"),
    ([16, 15], [40, 3], 4, 4, 8, "f32"),
    ([33], [16], 12, 1, 64, "bf16"),
    ([240], [16], 4, 1, 64, "f32"),
    ([1, 47, 16], [17, 2, 31], 24, 2, 8, "bf16"),
]


@pytest.mark.parametrize("case", range(len(SWEEP)))
def test_oracle_matches_brute_force(case):
    P, S, Hq, Hkv, D, dt = SWEEP[case]
    w = build_workload(name="sweep", seed=100 + case, prefix_len=P, suffix_len=S, num_q_heads=Hq,
                       num_kv_heads=Hkv, head_dim=D, dtype=dt, num_blocks=64, keep_logical=True)
    out, lse = _oracle(w)
    bo, bl = brute_force_extend(w.q, w.logical_k, w.logical_v, w.prefix_len, w.suffix_len, Hkv, w.scale)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    assert _rel(out, bo) <= 1e-12
    assert np.max(np.abs(lse - bl)) <= 1e-12 * max(1.0, np.max(np.abs(bl)))


def test_brute_force_catches_planted_mistakes():
    """Inputs that stand for plausible oracle bugs (mask shifted by one, two
    pages swapped, wrong head grouping) must fail the brute-force comparison."""
    w = build_workload(name="mut", seed=7, prefix_len=[33], suffix_len=[20], num_q_heads=8, num_kv_heads=2,
                       head_dim=8, dtype="bf16", num_blocks=64, keep_logical=True)
    bo, _ = brute_force_extend(w.q, w.logical_k, w.logical_v, w.prefix_len, w.suffix_len, 2, w.scale)
    kp, vp = _appended(w)
    # off-by-one causal window (the diagonal position left out)
    o1, _ = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len - 1, w.suffix_len, 2, w.scale)
    assert _rel(o1, bo) > 1e-3
    # two pages swapped in the table (one of them straddles the causal edge;
    # swapping two pages every query sees fully would be invisible, since
    # attention is a set function of the visible positions)
    bt = w.compact_table.copy()
    bt[0, [0, 2]] = bt[0, [2, 0]]
    o2, _ = oracle_extend(w.q, kp, vp, bt, w.prefix_len, w.suffix_len, 2, w.scale)
    assert _rel(o2, bo) > 1e-3
    # interleaved head grouping (h % Hkv instead of h // G)
    perm = np.array([h // 2 + (h % 2) * 4 for h in range(8)])
    o3, _ = oracle_extend(w.q[:, perm], kp, vp, w.compact_table, w.prefix_len, w.suffix_len, 2, w.scale)
    assert _rel(o3[:, np.argsort(perm)], bo) > 1e-3


# ---------------------------------------------------------------------------
# the oracle's own input decoding and row sampling
# ---------------------------------------------------------------------------

# bf16 bit pattern -> value, derived from the format (sign, 8 exponent bits with
# bias 127, 7 fraction bits): 0x3F80 = +2^0; 0xC020 = -(1 + 1/4) * 2^1;
# 0x0001 = the smallest subnormal 2^-126 * 2^-7; 0x0080 = the smallest normal
# 2^-126; 0x7F7F = the largest finite (2 - 2^-7) * 2^127; 0x4049 =
# (1 + 73/128) * 2^1; 0x3E80 = 2^-2; 0x7F80 / 0xFF80 = +-inf; 0x8000 = -0.
BF16_PATTERNS = [
    (0x3F80, 1.0), (0xC020, -2.5), (0x0001, 2.0 ** -133), (0x0080, 2.0 ** -126),
    (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127), (0x4049, 3.140625), (0x3E80, 0.25),
    (0x7F80, math.inf), (0xFF80, -math.inf), (0x8000, -0.0), (0x0000, 0.0),
]


def test_bf16_storage_decodes_fixed_bit_patterns():
    """Every CPU comparison on bf16 data widens both sides through
    ``storage_to_f64``; pin its bf16 branch on hand-decoded bit patterns (a
    shifted, sign-dropped or byte-swapped decoding fails here) and against
    torch's own bfloat16 -> float64 conversion."""
    torch = pytest.importorskip("torch")
    bits = np.array([p for p, _ in BF16_PATTERNS], dtype=np.uint16)
    got = storage_to_f64(bits)
    assert got.dtype == np.float64
    for (p, want), g in zip(BF16_PATTERNS, got):
        assert g == want and math.copysign(1.0, g) == math.copysign(1.0, want), hex(p)
    assert np.isnan(storage_to_f64(np.array([0x7FC0, 0xFFC1], dtype=np.uint16))).all()
    # all 65536 patterns agree with torch's conversion (NaNs as NaNs)
    every = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):          # widening NaN payloads
        ours = storage_to_f64(every)
    theirs = torch.from_numpy(every.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(theirs)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint64), theirs[~nan].view(np.uint64))
    # float32 storage is widened unchanged
    f = np.array([1.5, -0.0, 3.4e38, 1e-45], dtype=np.float32)
    assert np.array_equal(storage_to_f64(f).view(np.uint64), f.astype(np.float64).view(np.uint64))


def test_row_sampling_equals_brute_force_rows():
    """``oracle_extend(rows=...)`` computes only the chosen suffix tokens; on a
    ragged three-sequence batch (G = 12, chunks of two tokens so a selection
    crosses several chunk boundaries, one sequence with no rows selected, one
    with all) its rows equal brute force at those rows and the full call's."""
    P, S = [37, 0, 120], [23, 9, 31]
    w = build_workload(name="rows", seed=23, prefix_len=P, suffix_len=S, num_q_heads=24, num_kv_heads=2,
                       head_dim=16, dtype="bf16", num_blocks=64, keep_logical=True)
    kp, vp = _appended(w)
    rows = [np.array([0, 3, 4, 5, 11, 21, 22]), np.array([], dtype=np.int64), None]
    out, lse = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, 2, w.scale, rows=rows,
                             chunk_rows=24)
    assert out.shape == (7 + 0 + 31, 24, 16) and lse.shape == (38, 24)
    bo, bl = brute_force_extend(w.q, w.logical_k, w.logical_v, w.prefix_len, w.suffix_len, 2, w.scale)
    fo, fl = oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, 2, w.scale)
    off = w.seq_offsets
    idx = np.concatenate([off[0] + rows[0], off[2] + np.arange(S[2])])
    assert _rel(out, bo[idx]) <= 1e-12
    assert np.max(np.abs(lse - bl[idx])) <= 1e-12 * np.max(np.abs(bl))
    assert np.array_equal(out, fo[idx]) and np.array_equal(lse, fl[idx])


# ---------------------------------------------------------------------------
# library routines
# ---------------------------------------------------------------------------

def test_no_prefix_is_textbook_causal_attention():
    """P = 0 reduces to causal self-attention over the S new tokens: compare
    with torch's scaled_dot_product_attention(is_causal=True) in fp64."""
    torch = pytest.importorskip("torch")
    S, H, D = 37, 3, 16
    w = build_workload(name="p0", seed=11, prefix_len=[0], suffix_len=[S], num_q_heads=H, num_kv_heads=H,
                       head_dim=D, dtype="bf16", num_blocks=16, keep_logical=True)
    out, _ = _oracle(w)
    q = torch.from_numpy(storage_to_f64(w.q)).permute(1, 0, 2)
    k = torch.from_numpy(storage_to_f64(w.logical_k[0])).permute(1, 0, 2)
    v = torch.from_numpy(storage_to_f64(w.logical_v[0])).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True, scale=w.scale)
    assert _rel(out, ref.permute(1, 0, 2).numpy()) <= 1e-12


def test_lse_matches_scipy_logsumexp():
    sp = pytest.importorskip("scipy.special")
    w = build_workload(name="lse", seed=12, prefix_len=[50], suffix_len=[9], num_q_heads=4, num_kv_heads=2,
                       head_dim=32, dtype="bf16", num_blocks=16, keep_logical=True)
    _, lse = _oracle(w)
    for i in range(9):
        for h in range(4):
            k = storage_to_f64(w.logical_k[0][:50 + i + 1, h // 2])
            s = w.scale * (k @ storage_to_f64(w.q[i, h]))
            assert abs(lse[i, h] - sp.logsumexp(s)) <= 1e-12 * max(1, abs(lse[i, h]))


# ---------------------------------------------------------------------------
# closed forms of degenerate inputs
# ---------------------------------------------------------------------------

def test_zero_keys_average_the_visible_values():
    """K = 0 makes every logit 0, so each output is the plain mean of V over
    positions 0..P+i: the divisor P+i+1 pins the causal window length."""
    P, S = [70, 3], [21, 40]
    w = build_workload(name="kz", seed=13, prefix_len=P, suffix_len=S, num_q_heads=6, num_kv_heads=2,
                       head_dim=16, dtype="bf16", num_blocks=64, variant="kzero", keep_logical=True)
    out, lse = _oracle(w)
    off = w.seq_offsets
    for b in range(2):
        v = storage_to_f64(w.logical_v[b])                      # [L, Hkv, D]
        csum = np.cumsum(v, axis=0)
        for i in range(S[b]):
            n = P[b] + i + 1
            mean = csum[n - 1] / n                               # [Hkv, D]
            want = np.repeat(mean, 3, axis=0)
            assert np.allclose(out[off[b] + i], want, rtol=1e-12, atol=1e-12)
            assert np.allclose(lse[off[b] + i], math.log(n), rtol=0, atol=1e-12)


def test_constant_values_reproduce_the_constant():
    w = build_workload(name="vc", seed=14, prefix_len=[100], suffix_len=[30], num_q_heads=8, num_kv_heads=4,
                       head_dim=32, dtype="bf16", num_blocks=64, variant="vconst")
    out, _ = _oracle(w)
    c = storage_to_f64(w.extra["vconst"])                         # [Hkv, D]
    want = np.repeat(c, 2, axis=0)[None]
    assert np.allclose(out, want, rtol=1e-13, atol=1e-13)


def test_needle_selects_its_target_value():
    """A needle query puts logit ~40 on its target position t; every other
    logit is N(0, 1600/|K_t|^2), so the output is V[t] up to a residual mass
    of about e^-30 here, and lse sits at 40 up to the bf16 rounding of q."""
    w = build_workload(name="nd", seed=15, prefix_len=[2000], suffix_len=[8], num_q_heads=4, num_kv_heads=1,
                       head_dim=128, dtype="bf16", num_blocks=256, variant="needle", keep_logical=True)
    out, lse = _oracle(w)
    tgt = w.extra["needle_target"]
    v = storage_to_f64(w.logical_v[0])
    want = v[tgt, 0, :]                                          # [T, Hq, D]
    assert np.max(np.abs(out - want)) < 1e-9
    assert np.max(np.abs(lse - 40.0)) < 0.5


def test_needle_targets_cover_every_page():
    """Per kv-head the latest (token, head) pairs point at distinct pages, so
    when a sequence has at least as many pairs per kv-head as pages, every
    page (the partly filled last one too) is a target of every kv-head, and
    every target is a position its query may see."""
    P, S = [130, 61], [40, 7]
    w = build_workload(name="cov", seed=24, prefix_len=P, suffix_len=S, num_q_heads=6, num_kv_heads=2,
                       head_dim=16, dtype="bf16", num_blocks=64, variant="needle")
    tgt = w.extra["needle_target"]
    off = w.seq_offsets
    for b in range(2):
        t = tgt[off[b]:off[b + 1]]
        assert np.all(t >= 0) and np.all(t <= P[b] + np.arange(S[b])[:, None])
        nblk = (P[b] + S[b] + 15) // 16
        for g in range(2):
            pages = set((t[:, 3 * g:3 * g + 3] // 16).reshape(-1).tolist())
            if S[b] * 3 >= nblk:
                assert pages == set(range(nblk))


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def test_gqa_equals_mha_with_repeated_kv_heads():
    w = build_workload(name="gqa", seed=16, prefix_len=[45, 9], suffix_len=[12, 30], num_q_heads=12,
                       num_kv_heads=3, head_dim=16, dtype="bf16", num_blocks=32)
    out, lse = _oracle(w)
    kp, vp = _appended(w)
    kr = np.repeat(kp, 4, axis=1)        # kv-head g copied to heads 4g..4g+3
    vr = np.repeat(vp, 4, axis=1)
    o2, l2 = oracle_extend(w.q, kr, vr, w.compact_table, w.prefix_len, w.suffix_len, 12, w.scale)
    assert _rel(o2, out) <= 1e-13 and np.max(np.abs(l2 - lse)) <= 1e-13


def test_paging_is_invisible():
    """Relabelling physical pages (moving blocks and rewriting the table
    consistently) leaves the result bit-identical."""
    w = build_workload(name="perm", seed=17, prefix_len=[77, 160], suffix_len=[19, 4], num_q_heads=4,
                       num_kv_heads=2, head_dim=16, dtype="bf16", num_blocks=64)
    out, lse = _oracle(w)
    kp, vp = _appended(w)
    rng = np.random.default_rng(0)
    n = kp.shape[0]
    perm = rng.permutation(n)              # new position of old block i is perm[i]
    kq = np.empty_like(kp); vq = np.empty_like(vp)
    kq[perm] = kp; vq[perm] = vp
    bt = np.where(w.compact_table >= 0, perm[np.maximum(w.compact_table, 0)], -1).astype(np.int32)
    o2, l2 = oracle_extend(w.q, kq, vq, bt, w.prefix_len, w.suffix_len, 2, w.scale)
    assert np.array_equal(o2, out) and np.array_equal(l2, lse)


def test_prefix_reuse_equals_full_recompute():
    """Reusing P cached positions and extending by S gives the same rows as
    prefilling all P+S positions from scratch (the premise of KV reuse, §1)."""
    P, S = 53, 27
    full = build_workload(name="full", seed=18, prefix_len=[0], suffix_len=[P + S], num_q_heads=6,
                          num_kv_heads=2, head_dim=16, dtype="bf16", num_blocks=16, keep_logical=True)
    o_full, l_full = _oracle(full)
    # same logical data, now with the first P positions treated as a reused prefix
    kp = np.full_like(full.k_pool_c, 0); vp = np.full_like(full.v_pool_c, 0)
    kp[...] = full.k_pool_c; vp[...] = full.v_pool_c
    kp, vp = oracle_append(kp, vp, full.compact_table, [0], [P], full.k_new[:P], full.v_new[:P])
    kp, vp = oracle_append(kp, vp, full.compact_table, [P], [S], full.k_new[P:], full.v_new[P:])
    o_ext, l_ext = oracle_extend(full.q[P:], kp, vp, full.compact_table, [P], [S], 2, full.scale)
    assert _rel(o_ext, o_full[P:]) <= 1e-13
    assert np.max(np.abs(l_ext - l_full[P:])) <= 1e-13


def test_chunked_turns_equal_one_turn():
    """append+extend(P, S1) then append+extend(P+S1, S2) equals append+extend(P, S1+S2)."""
    P, S1, S2 = 40, 13, 22
    w = build_workload(name="chunk", seed=19, prefix_len=[P], suffix_len=[S1 + S2], num_q_heads=4,
                       num_kv_heads=1, head_dim=16, dtype="bf16", num_blocks=16)
    o_one, _ = _oracle(w)
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, [P], [S1], w.k_new[:S1], w.v_new[:S1])
    o_a, _ = oracle_extend(w.q[:S1], kp, vp, w.compact_table, [P], [S1], 1, w.scale)
    kp, vp = oracle_append(kp, vp, w.compact_table, [P + S1], [S2], w.k_new[S1:], w.v_new[S1:])
    o_b, _ = oracle_extend(w.q[S1:], kp, vp, w.compact_table, [P + S1], [S2], 1, w.scale)
    assert _rel(np.concatenate([o_a, o_b]), o_one) <= 1e-13


def test_shift_of_all_keys_moves_only_lse():
    """Adding one vector u to every key adds scale*<q,u> to every logit of a
    row: the output is unchanged and lse moves by exactly that amount."""
    w = build_workload(name="shift", seed=20, prefix_len=[31], suffix_len=[6], num_q_heads=2, num_kv_heads=1,
                       head_dim=8, dtype="f32", num_blocks=8)
    out, lse = _oracle(w)
    kp, vp = _appended(w)
    u = np.linspace(-1, 1, 8)
    ks = storage_to_f64(kp) + u
    o2, l2 = oracle_extend(w.q, ks, vp, w.compact_table, w.prefix_len, w.suffix_len, 1, w.scale)
    assert _rel(o2, out) <= 1e-12
    want = lse + w.scale * (storage_to_f64(w.q) @ u)
    assert np.allclose(l2, want, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# append
# ---------------------------------------------------------------------------

def test_append_places_every_token_and_touches_nothing_else():
    P, S = [0, 17, 40, 64], [5, 31, 24, 1]
    w = build_workload(name="app", seed=21, prefix_len=P, suffix_len=S, num_q_heads=2, num_kv_heads=2,
                       head_dim=8, dtype="bf16", num_blocks=40, keep_logical=True)
    kp, vp = _appended(w)
    touched = np.zeros(kp.shape[:3], dtype=bool)          # [block, head, slot]
    for b in range(4):
        L = P[b] + S[b]
        for g in range(2):
            # read back through the table: logical order must be the generator's logical sequence
            assert np.array_equal(gather_logical(kp, w.compact_table[b], L, g),
                                  storage_to_f64(w.logical_k[b][:, g]))
            assert np.array_equal(gather_logical(vp, w.compact_table[b], L, g),
                                  storage_to_f64(w.logical_v[b][:, g]))
        for j in range(P[b], L):
            touched[w.compact_table[b, j // 16], :, j % 16] = True
    # every other byte unchanged (including the NaN canaries and prefix slots)
    assert np.array_equal(kp[~touched], w.k_pool_c[~touched])
    assert np.array_equal(vp[~touched], w.v_pool_c[~touched])
    # the slots that were written held NaN before (fresh slots only)
    assert np.all(w.k_pool_c[touched] == 0x7FC0)


def test_append_leaves_shared_fork_blocks_alone():
    """Forked sequences share their first pages (§5.2); appending into every
    child must not change a byte of the shared pages."""
    w = build_workload(name="fork", seed=22, prefix_len=[48, 60, 33], suffix_len=[9, 20, 40], num_q_heads=2,
                       num_kv_heads=1, head_dim=8, dtype="bf16", num_blocks=64, shared_prefix_blocks=2)
    kp, vp = _appended(w)
    shared = w.compact_table[0, :2]
    assert np.all(w.compact_table[:, :2] == shared)
    assert np.array_equal(kp[shared], w.k_pool_c[shared]) and np.array_equal(vp[shared], w.v_pool_c[shared])


# ---------------------------------------------------------------------------
# page moves between HBM and host (oracle_to_host / oracle_to_device)
# ---------------------------------------------------------------------------

def _tiny_pools():
    # page p, head g, slot s, dim d holds the integer 1000*p + 100*g + 10*s + d
    nb, hkv, d = 5, 2, 3
    p, g, s, e = np.meshgrid(np.arange(nb), np.arange(hkv), np.arange(16), np.arange(d), indexing="ij")
    k = (1000 * p + 100 * g + 10 * s + e).astype(np.float32)
    return k, -k


def test_to_host_packs_pages_in_list_order():
    from oracle import oracle_to_host
    k, v = _tiny_pools()
    host = oracle_to_host(k, v, [3, 0, 3])
    assert host.shape == (3, 2, 2, 16, 3)
    assert host[0, 0, 1, 2, 1] == 3000 + 100 + 20 + 1          # K of page 3, head 1, slot 2, dim 1
    assert host[1, 1, 0, 15, 2] == -(0 + 0 + 150 + 2)          # V of page 0, head 0, slot 15, dim 2
    assert np.array_equal(host[0], host[2])                    # a page may be read twice


def test_to_device_round_trip_and_untouched_pages():
    from oracle import oracle_to_device, oracle_to_host
    k, v = _tiny_pools()
    host = oracle_to_host(k, v, [4, 1])
    k2, v2 = oracle_to_device(np.zeros_like(k), np.zeros_like(v), [2, 0], host)
    assert np.array_equal(k2[2], k[4]) and np.array_equal(v2[0], v[1])
    assert not k2[1].any() and not k2[3].any() and not v2[4].any()    # only listed pages change
    # offload then reload of the same list is the identity on those pages
    k3, v3 = oracle_to_device(np.zeros_like(k), np.zeros_like(v), [4, 1], host)
    assert np.array_equal(k3[[4, 1]], k[[4, 1]]) and np.array_equal(v3[[4, 1]], v[[4, 1]])
    with pytest.raises(ValueError):
        oracle_to_device(k, v, [1, 1], host)
    # bitwise: NaN payloads survive
    nan_bits = np.array([0x7FC1], dtype=np.uint16)
    kb = np.zeros((2, 1, 16, 1), dtype=np.uint16); kb[1, 0, 5, 0] = nan_bits[0]
    assert oracle_to_host(kb, kb, [1])[0, 0, 0, 5, 0] == 0x7FC1
