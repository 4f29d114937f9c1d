"""Closed forms checked over every row at full size (no oracle sampling).

The oracle compares sampled rows at the 128K turn, the forked batch, the
258K mutation and the ragged agent batch (a split plan over contexts of very
different lengths); these inputs have answers that need no oracle, so every
(token, head) row of the output is checked against them:

* needle: each query's target logit is 40 and every other visible logit is
  N(0, 1600/|K_t|^2), so out = V_b[target] up to a residual mass far below the
  bf16 rounding of the output; at the 128K turn and the 258K mutation the
  targets of every kv-head cover every page of the sequence, so a wrong page,
  slot or head anywhere shows as an O(1) error;
* zero keys: every logit is 0, so out = mean of V over positions 0..P_b+i
  (fp64 prefix sums): pins the causal window of every row;
* constant values: V = c_g for kv-head g, so out = c_g: pins the normaliser.

Bounds: the parity bounds (max-abs 2e-2, mean-abs 2e-3, rel-L2 1e-2) over all
rows; the window means use the tighter 2e-3 / 5e-4 of the smaller tests.
"""
import numpy as np
import pytest

from oracle import gather_logical, storage_to_f64
from paper_2609_39819_amd.workloads import torch_to_np

from gpu_common import MAX_ABS, MEAN_ABS, REL_L2, cached_config, oracle_pools, run_append, run_extend, say, stage

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


class Stats:
    """max-abs, mean-abs and rel-L2 accumulated over row blocks."""

    def __init__(self, label):
        self.label, self.max, self.abs_sum, self.n, self.d2, self.r2 = label, 0.0, 0.0, 0, 0.0, 0.0
        self.finite = True

    def add(self, got, want):
        diff = np.abs(got - want)
        self.finite &= bool(np.isfinite(got).all())
        self.max = max(self.max, float(diff.max()))
        self.abs_sum += float(diff.sum())
        self.n += diff.size
        self.d2 += float((diff * diff).sum())
        self.r2 += float((want * want).sum())

    def check(self, max_abs=MAX_ABS, mean_abs=MEAN_ABS, rel_l2=REL_L2):
        mean, rel = self.abs_sum / self.n, (self.d2 / max(self.r2, 1e-300)) ** 0.5
        say(f"{self.label}: max_abs={self.max:.3e} mean_abs={mean:.3e} rel_l2={rel:.3e} (n={self.n}, every row)")
        assert self.finite, f"{self.label}: non-finite output"
        assert self.max <= max_abs, f"{self.label}: max_abs {self.max} > {max_abs}"
        assert mean <= mean_abs, f"{self.label}: mean_abs {mean} > {mean_abs}"
        assert rel <= rel_l2, f"{self.label}: rel_l2 {rel} > {rel_l2}"


def _run(name, variant):
    w = cached_config(name, variant)
    d = stage(w)
    run_append(w, d)
    out = run_extend(w, d)
    got = torch_to_np(out, w.dtype)                 # stored bits, converted per head below
    del d, out
    torch.cuda.empty_cache()
    return w, got


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name", ["react_128k", "forked_agents", "mutation_258k", "ragged_agents"])
def test_needle_every_row_returns_its_target_value(name):
    w, got = _run(name, "needle")
    _, vp = oracle_pools(name, "needle")
    tgt = w.extra["needle_target"]
    off, G = w.seq_offsets, w.group
    st = Stats(f"{name} needle vs V[target]")
    for b in range(w.num_seqs):
        L = int(w.prefix_len[b] + w.suffix_len[b])
        nblk = (L + 15) // 16
        rows = slice(int(off[b]), int(off[b + 1]))
        for g in range(w.num_kv_heads):
            v = gather_logical(vp, w.compact_table[b], L, g)            # [L, D] fp64
            for h in range(g * G, (g + 1) * G):
                st.add(storage_to_f64(got[rows, h, :]), v[tgt[rows, h]])
            pages = np.unique(tgt[rows, g * G:(g + 1) * G] // 16)
            if int(w.suffix_len[b]) * G >= nblk:
                # every page of the sequence is some query's target for this kv-head
                assert pages.size == nblk and pages[0] == 0 and pages[-1] == nblk - 1, (b, g, pages.size, nblk)
    st.check()


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name", ["forked_agents", "mutation_258k", "ragged_agents"])
def test_zero_keys_every_row_is_its_window_mean(name):
    w, got = _run(name, "kzero")
    _, vp = oracle_pools(name, "kzero")
    off, G = w.seq_offsets, w.group
    st = Stats(f"{name} kzero vs window means")
    for b in range(w.num_seqs):
        P, S = int(w.prefix_len[b]), int(w.suffix_len[b])
        rows = slice(int(off[b]), int(off[b + 1]))
        n = (P + np.arange(S) + 1)[:, None]
        for g in range(w.num_kv_heads):
            cs = np.cumsum(gather_logical(vp, w.compact_table[b], P + S, g), axis=0)
            want = cs[P + np.arange(S)] / n                              # [S, D]
            for h in range(g * G, (g + 1) * G):
                st.add(storage_to_f64(got[rows, h, :]), want)
    st.check(max_abs=2e-3, mean_abs=5e-4)


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name", ["forked_agents", "mutation_258k"])
def test_constant_values_every_row(name):
    w, got = _run(name, "vconst")
    c = storage_to_f64(w.extra["vconst"])                                # [Hkv, D]
    G = w.group
    st = Stats(f"{name} vconst vs c")
    worst = 0.0
    for h in range(w.num_q_heads):
        o = storage_to_f64(got[:, h, :])
        st.add(o, np.broadcast_to(c[h // G], o.shape))
        worst = max(worst, float(np.max(np.abs(o - c[h // G]) / np.maximum(np.abs(c[h // G]), 1e-3))))
    st.check()
    assert worst < 2 ** -7, worst     # sum_j p_j c / sum_j p_j = c up to bf16 rounding of p and of the output
