"""Seeded synthetic workloads for paged-KV extend attention.

This module holds input recipes only: sequence lengths, physical block
placement and random tensor values.  It contains none of the attention
arithmetic; the fp64 oracle and the HIP library both consume what it
produces, and neither imports the other.

Shapes follow the long-context agent workloads the paper characterises
(contexts of a few thousand to a quarter million tokens, a tool output appended
as the new suffix, forked sub-agents sharing a parent prefix, a mid-context
edit that forces a suffix recompute; paper §2.2, §5.1, §5.2).  The paper's
own replay drives its serving stack with random prompts of recorded lengths
(§8.1), so random N(0,1) tensors at these lengths stand in for its traces.

Storage conventions
-------------------
* bf16 tensors are numpy ``uint16`` arrays holding raw bf16 bit patterns
  (numpy has no bf16 type); fp32 tensors are ``float32``.
* Values are drawn as float32 N(0,1) from ``numpy.random.default_rng(seed)``
  and rounded to bf16 with round-to-nearest-even, so both sides see the exact
  stored values.
* A paged pool is ``[num_blocks][num_kv_heads][16][head_dim]``; K and V live
  in separate pools of the same shape.
* Every pool slot that holds no token is NaN, so a stray read shows up.

Draw order for a seed: random lengths (only the forked-batch workload has
them) -> physical block ids (one permutation of the pool, consumed in order)
-> logical K and V of each sequence -> Q -> variant-specific draws.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import math
from typing import List, Optional

import numpy as np

BLOCK_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)

# --------------------------------------------------------------------------
# bf16 bit helpers (input rounding only)
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray, chunk: int = 1 << 24) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    flat = x.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)
    for s in range(0, flat.size, chunk):
        u = flat[s:s + chunk].view(np.uint32)
        # u + 0x7FFF + lsb only wraps for NaN bit patterns, which are replaced below
        r = u + np.uint32(0x7FFF)
        r += (u >> 16) & np.uint32(1)
        r >>= 16
        r = r.astype(np.uint16)
        nan = np.isnan(flat[s:s + chunk])
        if nan.any():
            r[nan] = BF16_NAN
        out[s:s + chunk] = r
    return out.reshape(x.shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float32 exactly."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# workload container
# --------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str                      # "bf16" | "f32"
    prefix_len: np.ndarray          # int32 [B]
    suffix_len: np.ndarray          # int32 [B]
    num_blocks: int                 # physical pool size NB
    block_table: np.ndarray         # int32 [B, max_blocks] physical ids, -1 past the last used block
    phys_ids: np.ndarray            # int64 [NBc] physical id of each compact block
    compact_table: np.ndarray       # int32 [B, max_blocks] indices into phys_ids, -1 padding
    k_pool_c: np.ndarray            # [NBc, Hkv, 16, D] compact pool: prefix slots filled, rest NaN
    v_pool_c: np.ndarray
    k_new: np.ndarray               # [T, Hkv, D] suffix K handed to append
    v_new: np.ndarray
    q: np.ndarray                   # [T, Hq, D]
    scale: float
    variant: str = "normal"
    logical_k: Optional[List[np.ndarray]] = None   # per sequence [P+S, Hkv, D] (small workloads)
    logical_v: Optional[List[np.ndarray]] = None
    extra: dict = field(default_factory=dict)

    @property
    def num_seqs(self) -> int:
        return int(self.prefix_len.shape[0])

    @property
    def total_tokens(self) -> int:
        return int(self.suffix_len.sum())

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def max_blocks(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def seq_offsets(self) -> np.ndarray:
        """Row offset of each sequence's first suffix token in the packed tensors."""
        return np.concatenate([[0], np.cumsum(self.suffix_len)]).astype(np.int64)


def _nan_like_storage(shape, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return np.full(shape, BF16_NAN, dtype=np.uint16)
    return np.full(shape, np.nan, dtype=np.float32)


def _normal(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    return x


# logit of a needle query's target position (natural-log units)
NEEDLE_LOGIT = 40.0


def _needle_query(keys: np.ndarray, dtype: str, scale: float) -> np.ndarray:
    """Stored queries whose logit against their own target key is about
    NEEDLE_LOGIT: q = NEEDLE_LOGIT / (scale * |k|^2) * k, rounded to storage."""
    k = bf16_bits_to_f32(keys) if dtype == "bf16" else keys
    k64 = k.astype(np.float64)
    n2 = np.maximum((k64 * k64).sum(axis=-1, keepdims=True), 1e-30)
    qv = (NEEDLE_LOGIT / (scale * n2) * k64).astype(np.float32)
    return f32_to_bf16_bits(qv) if dtype == "bf16" else qv


def build_workload(
    *,
    name: str,
    seed: int,
    prefix_len,
    suffix_len,
    num_q_heads: int,
    num_kv_heads: int,
    head_dim: int,
    dtype: str = "bf16",
    num_blocks: Optional[int] = None,
    shared_prefix_blocks: int = 0,
    variant: str = "normal",
    keep_logical: Optional[bool] = None,
    rng: Optional[np.random.Generator] = None,
    extra_table_cols: int = 0,
) -> Workload:
    """General seeded builder.

    ``shared_prefix_blocks`` > 0 gives every sequence the same first
    ``shared_prefix_blocks`` physical blocks (a forked context inheriting its
    parent's prefix, §5.2 / §6.1); their contents are drawn once.

    ``variant``:
      * ``normal``  Q, K, V ~ N(0,1)
      * ``kzero``   every key is zero (logits all zero)
      * ``vconst``  every value row of kv-head g equals one vector c_g
      * ``needle``  q[t,h] = NEEDLE_LOGIT / (scale * |K_b[target]|^2) * K_b[target]
                    (stored rounded), so the target's logit is NEEDLE_LOGIT
                    whatever its key's norm and it outweighs every other
                    visible position by a factor of about e^14 even at 262144
                    positions; the target is uniform over the positions that
                    query may see, except that for each kv-head the latest
                    (token, head) pairs point at distinct pages, last page
                    first, so every page of a sequence is some query's target
                    when the sequence has at least as many pairs per kv-head
                    as pages; stores ``extra["needle_target"]``
    """
    if rng is None:
        rng = np.random.default_rng(seed)
    P = np.asarray(prefix_len, dtype=np.int64).reshape(-1)
    S = np.asarray(suffix_len, dtype=np.int64).reshape(-1)
    B = P.shape[0]
    assert S.shape[0] == B and B >= 1
    assert (P >= 0).all() and (S >= 1).all()
    assert num_q_heads % num_kv_heads == 0
    Hq, Hkv, D = num_q_heads, num_kv_heads, head_dim
    G = Hq // Hkv
    L = P + S
    nblk = (L + BLOCK_SIZE - 1) // BLOCK_SIZE
    sh = int(shared_prefix_blocks)
    if sh:
        assert (P >= sh * BLOCK_SIZE).all(), "shared blocks must hold prefix tokens only"
    n_ids = int(sh + (nblk - sh).sum())
    if num_blocks is None:
        num_blocks = n_ids
    assert n_ids <= num_blocks
    if keep_logical is None:
        keep_logical = int(L.sum()) * Hkv * D <= (1 << 22)

    # ---- physical placement: one permutation of the pool, consumed in order
    perm = rng.permutation(num_blocks)[:n_ids].astype(np.int64)
    max_blocks = int(nblk.max()) + int(extra_table_cols)
    block_table = np.full((B, max_blocks), -1, dtype=np.int32)
    compact_table = np.full((B, max_blocks), -1, dtype=np.int32)
    cur = sh
    for b in range(B):
        cidx = np.empty(nblk[b], dtype=np.int64)
        cidx[:sh] = np.arange(sh)
        k = nblk[b] - sh
        cidx[sh:] = np.arange(cur, cur + k)
        cur += k
        compact_table[b, :nblk[b]] = cidx
        block_table[b, :nblk[b]] = perm[cidx]
    phys_ids = perm

    # ---- logical K / V per sequence
    shared_tok = sh * BLOCK_SIZE
    if shared_tok:
        k_sh = _normal(rng, (shared_tok, Hkv, D), dtype)
        v_sh = _normal(rng, (shared_tok, Hkv, D), dtype)
    logical_k, logical_v = [], []
    for b in range(B):
        n = int(L[b]) - shared_tok
        kb = _normal(rng, (n, Hkv, D), dtype)
        vb = _normal(rng, (n, Hkv, D), dtype)
        if shared_tok:
            kb = np.concatenate([k_sh, kb], axis=0)
            vb = np.concatenate([v_sh, vb], axis=0)
        logical_k.append(kb)
        logical_v.append(vb)

    # ---- Q
    T = int(S.sum())
    q = _normal(rng, (T, Hq, D), dtype)
    off = np.concatenate([[0], np.cumsum(S)])

    extra = {}
    if variant == "kzero":
        zero = np.uint16(0) if dtype == "bf16" else np.float32(0.0)
        for kb in logical_k:
            kb[...] = zero
    elif variant == "vconst":
        c = _normal(rng, (Hkv, D), dtype)
        for vb in logical_v:
            vb[...] = c[None, :, :]
        extra["vconst"] = c
    elif variant == "needle":
        # each (token, head) points at one visible key of its own sequence
        targets = np.empty((T, Hq), dtype=np.int64)
        scale = 1.0 / math.sqrt(D)
        for b in range(B):
            t = np.arange(S[b])
            hi = P[b] + t  # inclusive upper bound of visible positions
            u = rng.random((S[b], Hq))
            tgt = np.minimum((u * (hi[:, None] + 1)).astype(np.int64), hi[:, None])
            # page coverage: pair k of kv-head g in (latest token first, head)
            # order targets page nblk-1-k; page 16*(nblk-1-k) <= P + token
            # holds because the page index falls by one per pair and the
            # token by one per G pairs
            n_cov = int(min(nblk[b], S[b] * G))
            k = np.arange(n_cov)
            tok = S[b] - 1 - k // G
            page = nblk[b] - 1 - k
            slot_hi = np.minimum(BLOCK_SIZE - 1, P[b] + tok - BLOCK_SIZE * page)
            for g in range(Hkv):
                us = rng.random(n_cov)
                slot = np.minimum((us * (slot_hi + 1)).astype(np.int64), slot_hi)
                tgt[tok, g * G + k % G] = BLOCK_SIZE * page + slot
            targets[off[b]:off[b + 1]] = tgt
            kb = logical_k[b]
            for h in range(Hq):
                g = h // G
                q[off[b]:off[b + 1], h, :] = _needle_query(kb[tgt[:, h], g, :], dtype, scale)
        extra["needle_target"] = targets
    elif variant != "normal":
        raise ValueError(f"unknown variant {variant!r}")

    # ---- page the prefix into the compact pool; suffix goes to k_new / v_new
    n_c = phys_ids.shape[0]
    k_pool_c = _nan_like_storage((n_c, Hkv, BLOCK_SIZE, D), dtype)
    v_pool_c = _nan_like_storage((n_c, Hkv, BLOCK_SIZE, D), dtype)
    for b in range(B):
        p = int(P[b])
        full = p // BLOCK_SIZE
        if full:
            cb = compact_table[b, :full]
            k_pool_c[cb] = logical_k[b][:full * BLOCK_SIZE].reshape(full, BLOCK_SIZE, Hkv, D).transpose(0, 2, 1, 3)
            v_pool_c[cb] = logical_v[b][:full * BLOCK_SIZE].reshape(full, BLOCK_SIZE, Hkv, D).transpose(0, 2, 1, 3)
        for j in range(full * BLOCK_SIZE, p):
            cb = compact_table[b, j // BLOCK_SIZE]
            k_pool_c[cb, :, j % BLOCK_SIZE, :] = logical_k[b][j]
            v_pool_c[cb, :, j % BLOCK_SIZE, :] = logical_v[b][j]
    k_new = np.concatenate([logical_k[b][P[b]:] for b in range(B)], axis=0)
    v_new = np.concatenate([logical_v[b][P[b]:] for b in range(B)], axis=0)

    return Workload(
        name=name, seed=seed, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, dtype=dtype,
        prefix_len=P.astype(np.int32), suffix_len=S.astype(np.int32), num_blocks=int(num_blocks),
        block_table=block_table, phys_ids=phys_ids, compact_table=compact_table,
        k_pool_c=k_pool_c, v_pool_c=v_pool_c, k_new=np.ascontiguousarray(k_new),
        v_new=np.ascontiguousarray(v_new), q=q, scale=1.0 / math.sqrt(D), variant=variant,
        logical_k=logical_k if keep_logical else None,
        logical_v=logical_v if keep_logical else None, extra=extra,
    )


# --------------------------------------------------------------------------
# the five named workloads
# --------------------------------------------------------------------------

CONFIG_NAMES = ("tiny", "gqa_8k", "react_128k", "forked_agents", "mutation_258k")
# one GPU's share of the 128K turn under 4-way tensor parallelism (heads split
# with no communication: 24 query heads over 2 kv-heads per GPU)
# one decoding step of a batch of 32 agent contexts (one new token each), and
# of 256 contexts (a serving batch: one launch of 256 sequence descriptors)
# 16 forked sub-agents each adding a short message over a long shared context
# 8 agents at different depths of their ReAct loops in one extend call (a
# ragged batch: contexts log-uniform over 2K..128K, 32..128 new tokens each)
EXTRA_CONFIG_NAMES = ("react_128k_tp4", "decode_batch", "decode_batch256", "forked_short", "ragged_agents")


def config_shapes(name: str) -> dict:
    """Static description of a named workload (no random draws)."""
    if name == "tiny":
        return dict(seed=1, num_q_heads=4, num_kv_heads=1, head_dim=64, dtype="f32",
                    num_blocks=64, prefix=240, suffix=16)
    if name == "gqa_8k":
        return dict(seed=2, num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=65536, prefix=8192, suffix=512)
    if name == "react_128k":
        return dict(seed=3, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 20, prefix=131072, suffix=2048)
    if name == "react_128k_tp4":
        return dict(seed=6, num_q_heads=24, num_kv_heads=2, head_dim=128, dtype="bf16",
                    num_blocks=1 << 20, prefix=131072, suffix=2048)
    if name == "decode_batch":
        return dict(seed=7, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 20, num_seqs=32, prefix=(2048, 32768), suffix=1)
    if name == "decode_batch256":
        return dict(seed=10, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 18, num_seqs=256, prefix=(1024, 8192), suffix=1)
    if name == "forked_agents":
        return dict(seed=4, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 20, num_seqs=16, shared_prefix=4096,
                    private_prefix=(4096, 65536), suffix=(256, 4096))
    if name == "forked_short":
        return dict(seed=8, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 18, num_seqs=16, shared_prefix=32768,
                    private_prefix=(0, 1023), suffix=(16, 16))
    if name == "ragged_agents":
        return dict(seed=11, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 20, num_seqs=8, prefix=(2048, 131072), suffix=(32, 128))
    if name == "mutation_258k":
        return dict(seed=5, num_q_heads=96, num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=1 << 20, prefix=204800, suffix=57344)
    raise KeyError(name)


def forked_lengths(rng: np.random.Generator, num_seqs: int, shared: int, private, suffix):
    """Per-sequence lengths of the forked-agents workload.

    Reading: the private part of each prefix is uniform over the inclusive
    integer range ``private``; the total prefix adds the shared part.
    """
    lp = rng.integers(private[0], private[1], size=num_seqs, endpoint=True)
    sl = rng.integers(suffix[0], suffix[1], size=num_seqs, endpoint=True)
    return shared + lp, sl


def make_config(name: str, variant: str = "normal", keep_logical: Optional[bool] = None) -> Workload:
    c = config_shapes(name)
    rng = np.random.default_rng(c["seed"])
    if name in ("forked_agents", "forked_short"):
        P, S = forked_lengths(rng, c["num_seqs"], c["shared_prefix"], c["private_prefix"], c["suffix"])
        sh_blocks = c["shared_prefix"] // BLOCK_SIZE
    elif name == "ragged_agents":
        # context lengths log-uniform over the range, new tokens uniform
        lo, hi = np.log(c["prefix"][0]), np.log(c["prefix"][1])
        P = np.round(np.exp(rng.uniform(lo, hi, size=c["num_seqs"]))).astype(np.int64)
        S = rng.integers(c["suffix"][0], c["suffix"][1], size=c["num_seqs"], endpoint=True)
        sh_blocks = 0
    elif name in ("decode_batch", "decode_batch256"):
        # reused context lengths uniform over the inclusive range, one new token each
        P = rng.integers(c["prefix"][0], c["prefix"][1], size=c["num_seqs"], endpoint=True)
        S = np.ones(c["num_seqs"], dtype=np.int64)
        sh_blocks = 0
    else:
        P, S = np.array([c["prefix"]]), np.array([c["suffix"]])
        sh_blocks = 0
    return build_workload(
        name=name, seed=c["seed"], prefix_len=P, suffix_len=S,
        num_q_heads=c["num_q_heads"], num_kv_heads=c["num_kv_heads"], head_dim=c["head_dim"],
        dtype=c["dtype"], num_blocks=c["num_blocks"], shared_prefix_blocks=sh_blocks,
        variant=variant, keep_logical=keep_logical, rng=rng)


def algorithmic_flops(prefix_len, suffix_len, num_q_heads: int, head_dim: int) -> int:
    """Work counted for throughput: QK^T plus PV over causal (query, key) pairs only.

    Query i of sequence b sees keys 0..P_b+i, i.e. P_b+i+1 keys; each pair costs
    2*D flops for the score and 2*D for the value accumulation.
    """
    P = np.asarray(prefix_len, dtype=np.int64)
    S = np.asarray(suffix_len, dtype=np.int64)
    pairs = int((S * P + S * (S + 1) // 2).sum())
    return 4 * head_dim * num_q_heads * pairs


def kv_bytes(prefix_len, suffix_len, num_kv_heads: int, head_dim: int, elem_bytes: int) -> int:
    """K+V bytes of every sequence's logical cache, each read once."""
    L = np.asarray(prefix_len, dtype=np.int64) + np.asarray(suffix_len, dtype=np.int64)
    return int(L.sum()) * num_kv_heads * head_dim * 2 * elem_bytes


# --------------------------------------------------------------------------
# device staging (test / bench harness only; torch indexing sets up inputs)
# --------------------------------------------------------------------------

def torch_storage_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def np_to_torch(a: np.ndarray, dtype: str, device):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == "bf16":
        t = t.view(torch.bfloat16)
    return t.to(device)


def torch_to_np(t, dtype: str) -> np.ndarray:
    import torch
    t = t.detach().to("cpu").contiguous()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def stage_on_device(w: Workload, device="cuda", num_blocks: Optional[int] = None):
    """Allocate the full physical pools (NaN everywhere), copy the compact
    blocks to their physical ids, and upload Q, the suffix K/V and the block table."""
    import torch
    nb = w.num_blocks if num_blocks is None else num_blocks
    tdt = torch_storage_dtype(w.dtype)
    shape = (nb, w.num_kv_heads, BLOCK_SIZE, w.head_dim)
    k_pool = torch.full(shape, float("nan"), dtype=tdt, device=device)
    v_pool = torch.full(shape, float("nan"), dtype=tdt, device=device)
    ids = torch.from_numpy(w.phys_ids).to(device)
    k_pool.index_copy_(0, ids, np_to_torch(w.k_pool_c, w.dtype, device))
    v_pool.index_copy_(0, ids, np_to_torch(w.v_pool_c, w.dtype, device))
    return dict(
        k_pool=k_pool, v_pool=v_pool,
        q=np_to_torch(w.q, w.dtype, device),
        k_new=np_to_torch(w.k_new, w.dtype, device),
        v_new=np_to_torch(w.v_new, w.dtype, device),
        block_table=torch.from_numpy(w.block_table).to(device),
    )


# --------------------------------------------------------------------------
# event trace for the host block manager
# --------------------------------------------------------------------------

def agent_events(seed: int = 9, agents: int = 256, concurrency: int = 32, calls=(8, 40),
                 system_tokens=(512, 4096), tool_tokens=(64, 4096), tool_wait=(16, 128), fork_prob: float = 0.1,
                 one_off_prob: float = 0.08, edit_prob: float = 0.03, pin_prob: float = 0.25):
    """A seeded stream of block-manager calls from interleaved ReAct agents.

    Each agent spawns, appends a system prompt (pinned for a share of agents)
    and a task, then runs U[calls] LLM calls -- issue, start of prefill, end
    of prefill, end of request -- each followed by a tool output of
    U[tool_tokens] tokens appended as a new message (paper §2.2, §5.2).  At
    a call boundary an agent may fork a sub-agent that runs a few calls over
    the shared prefix and terminates, or edit an earlier message (replace);
    a share of agents are one-off.  At most ``concurrency`` agents (plus
    their sub-agents) run at once, their next events interleaved at random;
    while its tool runs, an agent sits out U[tool_wait] events of the others
    (so few requests are in flight at once, as in a ReAct workload where
    tools and LLM calls alternate); an agent unpins its system prompt and
    terminates when done.

    Yields ``(op, args)`` with the method names of the manager; every call
    is valid for the state the earlier calls produce.  Token counts only --
    no attention arithmetic.
    """
    rng = np.random.default_rng(seed)
    next_id = [0]

    def new_id():
        next_id[0] += 1
        return next_id[0] - 1

    def call(c):
        yield "begin_request", (c,)
        yield "start_prefill", (c,)
        yield "prefill_done", (c,)
        yield "end_request", (c,)
        yield "wait", int(rng.integers(tool_wait[0], tool_wait[1], endpoint=True))

    def sub_agent(c, n_calls, n_msgs):
        for _ in range(n_calls):
            yield from call(c)
            yield "append", (c, int(rng.integers(tool_tokens[0], tool_tokens[1], endpoint=True)))
            n_msgs += 1
        yield "terminate", (c,)

    def agent(c):
        yield "spawn", (c,)
        yield "append", (c, int(rng.integers(system_tokens[0], system_tokens[1], endpoint=True)))
        pinned = rng.random() < pin_prob
        if pinned:
            yield "pin", (c, 0)
        yield "append", (c, int(rng.integers(32, 512, endpoint=True)))
        n_msgs = 2
        if rng.random() < one_off_prob:
            yield "one_off", (c,)
            yield from call(c)
            yield "terminate", (c,)
            if pinned:
                yield "unpin", (c, 0)
            return
        for _ in range(int(rng.integers(calls[0], calls[1], endpoint=True))):
            yield from call(c)
            yield "append", (c, int(rng.integers(tool_tokens[0], tool_tokens[1], endpoint=True)))
            n_msgs += 1
            u = rng.random()
            if u < fork_prob:
                k = new_id()
                yield "fork", (c, k)
                yield ("start", sub_agent(k, int(rng.integers(2, 6, endpoint=True)), n_msgs))
            elif u < fork_prob + edit_prob and n_msgs > 3:
                yield "replace", (c, int(rng.integers(2, n_msgs)), int(rng.integers(tool_tokens[0], tool_tokens[1])))
        yield "terminate", (c,)
        if pinned:
            yield "unpin", (c, 0)

    running, wake, started, t = [], [], 0, 0      # programs, the event count each may resume at
    while running or started < agents:
        while started < agents and len(running) < concurrency:
            running.append(agent(new_id()))
            wake.append(t)
            started += 1
        ready = [i for i in range(len(running)) if wake[i] <= t]
        if not ready:
            t = min(wake)
            continue
        i = ready[int(rng.integers(0, len(ready)))]
        try:
            ev = next(running[i])
        except StopIteration:
            running.pop(i)
            wake.pop(i)
            continue
        if ev[0] == "start":
            running.append(ev[1])
            wake.append(t)
        elif ev[0] == "wait":
            wake[i] = t + ev[1]
        else:
            t += 1
            yield ev
