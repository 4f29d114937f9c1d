"""The block manager driving the kernels' block tables over several turns.

The manager (``kvt_mgr_*``) models the reusable cache tier: KV is written
back into its pages after prefill (paper §6.2), while a running request
computes into working pages of its own.  Here one pool holds both: pages
[0, C) are the manager's, pages [C, N) are working pages.  Every turn of a
context:

1. ``begin_request`` / ``start_prefill`` give the hit prefix (whole messages);
2. the block table is the hit messages' cache pages (``message_pages``)
   followed by working pages for the rest;
3. ``kvt_append_kv`` writes the recomputed tokens' K/V, then
   ``kvt_extend_attention`` runs, checked against the fp64 oracle over the
   context's true K/V (so a wrong or stale cache page is an O(1) error);
4. ``prefill_done`` admits the new messages; each admitted one is copied
   from its working pages into the cache pages the manager chose (test
   plumbing), and ``end_request`` closes the turn.

Messages are multiples of 16 tokens, so cached messages start on page
boundaries and their page runs concatenate into a block table.  The turns
cover reuse, a fork that shares the parent's pages, eviction under pressure
(a later miss recomputes) and a replaced message.
"""
import math

import numpy as np
import pytest

from oracle import oracle_extend
from paper_2609_39819_amd import kvt

from gpu_common import compare, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HKV, HQ, D = 2, 8, 128
CACHE_PAGES, WORK_PAGES = 40, 48


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


class World:
    """The manager, the device pools and the true K/V of every message."""

    def __init__(self, seed):
        self.rng = np.random.default_rng(seed)
        self.mgr = kvt.Manager(CACHE_PAGES)
        nb = CACHE_PAGES + WORK_PAGES
        nan = torch.full((nb, HKV, 16, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        self.k_pool, self.v_pool = nan.clone(), nan.clone()
        self.ctx = {}          # context -> list of content ids (one per message)
        self.kv = {}           # content id -> (k, v) bf16 [tokens][HKV][D] on the host
        self.next_content = 0
        self.scale = 1.0 / math.sqrt(D)

    def _content(self, tokens):
        cid = self.next_content
        self.next_content += 1
        k = torch.from_numpy(self.rng.standard_normal((tokens, HKV, D), dtype=np.float32)).to(torch.bfloat16)
        v = torch.from_numpy(self.rng.standard_normal((tokens, HKV, D), dtype=np.float32)).to(torch.bfloat16)
        self.kv[cid] = (k, v)
        return cid

    def spawn(self, c):
        self.mgr.spawn(c)
        self.ctx[c] = []

    def fork(self, p, c):
        self.mgr.fork(p, c)
        self.ctx[c] = list(self.ctx[p])

    def append(self, c, tokens):
        assert tokens % 16 == 0
        self.mgr.append(c, tokens)
        self.ctx[c].append(self._content(tokens))

    def replace(self, c, i, tokens):
        """Message i gets new content; the later ones keep their text but
        their KV changes with the prefix, so they get new content too."""
        self.mgr.replace(c, i, tokens)
        self.ctx[c][i] = self._content(tokens)
        for j in range(i + 1, len(self.ctx[c])):
            self.ctx[c][j] = self._content(self.kv[self.ctx[c][j]][0].shape[0])

    def turn(self, c, label):
        """One request of context c; returns (hit tokens, admit report)."""
        msgs = self.ctx[c]
        sizes = [self.kv[m][0].shape[0] for m in msgs]
        L = sum(sizes)
        self.mgr.begin_request(c)
        hit = self.mgr.start_prefill(c)["hit_tokens"]
        bounds = np.concatenate([[0], np.cumsum(sizes)])
        nhit = int(np.searchsorted(bounds, hit))
        assert bounds[nhit] == hit, "hits are whole messages"
        table = []
        for i in range(nhit):
            pages = self.mgr.message_pages(c, i)
            assert pages is not None and len(pages) == sizes[i] // 16
            assert all(0 <= p < CACHE_PAGES for p in pages)
            table += pages
        new = L - hit
        work = list(range(CACHE_PAGES, CACHE_PAGES + new // 16))
        assert len(work) <= WORK_PAGES
        table += work
        bt = torch.tensor([table], dtype=torch.int32, device="cuda")
        k_all = torch.cat([self.kv[m][0] for m in msgs])
        v_all = torch.cat([self.kv[m][1] for m in msgs])
        q = torch.from_numpy(self.rng.standard_normal((new, HQ, D), dtype=np.float32)).to(torch.bfloat16)
        say(f"{label}: context {c}, {len(msgs)} messages, {L} tokens, hit {hit}, table {len(table)} pages")
        kvt.append_kv(self.k_pool, self.v_pool, bt, [hit], [new], k_all[hit:].cuda(), v_all[hit:].cuda())
        out = kvt.extend_attention(q.cuda(), self.k_pool, self.v_pool, bt, [hit], [new], self.scale)
        torch.cuda.synchronize()
        ident = np.arange(len(table), dtype=np.int32)[None, :]
        kp = k_all.float().numpy().reshape(len(table), 16, HKV, D).transpose(0, 2, 1, 3)
        vp = v_all.float().numpy().reshape(len(table), 16, HKV, D).transpose(0, 2, 1, 3)
        ref, _ = oracle_extend(q.float().numpy(), kp, vp, ident, [hit], [new], HKV, self.scale)
        compare(out.float().cpu().numpy().astype(np.float64), ref, label)
        rep = self.mgr.prefill_done(c)
        # write-back: each admitted message moves from its working pages to its cache pages
        for i in range(nhit, len(msgs)):
            pages = self.mgr.message_pages(c, i)
            if pages is None:
                continue
            first = CACHE_PAGES + (int(bounds[i]) - hit) // 16
            src = torch.arange(first, first + len(pages), device="cuda")
            dst = torch.tensor(pages, device="cuda")
            self.k_pool[dst] = self.k_pool[src]
            self.v_pool[dst] = self.v_pool[src]
        self.mgr.end_request(c)
        torch.cuda.synchronize()
        return hit, rep


@pytest.mark.timeout(300)
def test_manager_pages_serve_as_block_tables():
    w = World(990)
    w.spawn(1)
    w.append(1, 64)
    w.append(1, 48)
    hit, rep = w.turn(1, "first turn")
    assert hit == 0 and rep["admitted_pages"] == 7
    w.append(1, 32)
    hit, rep = w.turn(1, "second turn reuses both messages")
    assert hit == 112 and rep["admitted_pages"] == 2
    w.fork(1, 2)
    w.append(2, 16)
    hit, _ = w.turn(2, "forked child over the parent's pages")
    assert hit == 144
    # pressure: 40 cache pages, 9 held for context 1 and 1 for context 2; a
    # 32-page context pushes out the most recently suspended KV
    w.spawn(3)
    w.append(3, 320)
    w.append(3, 192)
    _, rep = w.turn(3, "large context under pressure")
    assert rep["released_entries"] > 0
    hit, _ = w.turn(1, "context 1 after evictions")
    assert hit < 144
    w.replace(1, 1, 64)
    hit, _ = w.turn(1, "after replacing message 1")
    assert hit <= 64
    hit, _ = w.turn(2, "forked child after its parent's edit")
    # every page handed out is inside the cache range and no two live messages share one
    seen = {}
    for c, msgs in w.ctx.items():
        for i in range(len(msgs)):
            pages = w.mgr.message_pages(c, i)
            for p in pages or []:
                assert 0 <= p < CACHE_PAGES
                seen.setdefault(p, set()).add(w.ctx[c][i])
    assert all(len(v) == 1 for v in seen.values()), "a page holds two different contents"
