"""Host block manager (CPU only): hand-worked pins, then library vs oracle.

The pins are traces worked by hand from the paper's rules -- lifecycle
transitions (§5.2), the aggregate state of shared KV and Algorithm 1's
admission order (§6.1), MRU inside the Suspended tier (§6.2) -- plus the
readings the library documents (lowest free page ids first, earliest first
inside the other tiers, ties inside one call by creation order, KV held from
the start of the prefill that reads it to the end of its request).  Each pin
runs on both the oracle model and the library.

Then seeded random event streams drive both side by side: every call must
succeed or fail on both, return the same report, and leave the same
observable state (free pages; every message's state, entry tier and page
ids).  Along the way the oracle's own state is checked against properties
Algorithm 1 fixes whatever the bookkeeping: pages are a partition, Temporary
KV is never admitted, held KV is never released, Pinned KV is released only
for a Pinned newcomer, and the KV released by one write-back is a prefix of
the order Discarded (earliest first), Suspended (latest first), Active
(earliest first), then Pinned, with no release once the newcomers fit.
"""
import numpy as np
import pytest

from oracle import OracleManager
from paper_2609_39819_amd import kvt

PINNED, ACTIVE, SUSPENDED, EXPIRED, TEMPORARY = 0, 1, 2, 3, 4
T_PINNED, T_ACTIVE, T_SUSPENDED, T_DISCARDED = 0, 1, 2, 3
REPORT_KEYS = ("admitted_entries", "admitted_pages", "bypassed_entries", "rejected_entries", "released_entries",
               "released_pages", "hit_tokens", "miss_tokens")


def test_state_codes_match_the_header():
    assert (kvt.KVT_PINNED, kvt.KVT_ACTIVE, kvt.KVT_SUSPENDED, kvt.KVT_EXPIRED, kvt.KVT_TEMPORARY) == (0, 1, 2, 3, 4)
    assert (kvt.KVT_TIER_PINNED, kvt.KVT_TIER_ACTIVE, kvt.KVT_TIER_SUSPENDED, kvt.KVT_TIER_DISCARDED) == (0, 1, 2, 3)


@pytest.fixture(params=["oracle", "library"])
def make(request):
    if request.param == "oracle":
        return OracleManager
    return kvt.Manager


def _err(m):
    return (ValueError,) if isinstance(m, OracleManager) else (kvt.KvtError,)


def serve(m, c):
    """One whole request; returns (start_prefill report, prefill_done report)."""
    m.begin_request(c)
    hit = m.start_prefill(c)
    adm = m.prefill_done(c)
    m.end_request(c)
    return hit, adm


def new_ctx(m, c, *tokens, pin=()):
    m.spawn(c)
    for t in tokens:
        m.append(c, t)
    for i in pin:
        m.pin(c, i)


# ---------------------------------------------------------------------------
# hand-worked pins
# ---------------------------------------------------------------------------

def test_pin_tier_order_and_mru(make):
    """Discarded goes first; inside Suspended the most recently suspended goes
    first even when an older, smaller entry would have been enough."""
    m = make(8)
    for c, t in ((1, 32), (2, 48), (3, 16)):              # 2, 3 and 1 pages
        new_ctx(m, c, t)
        hit, adm = serve(m, c)
        assert hit["miss_tokens"] == t and hit["hit_tokens"] == 0
        assert adm["admitted_entries"] == 1 and adm["released_entries"] == 0
    assert (m.message_pages(1, 0), m.message_pages(2, 0), m.message_pages(3, 0)) == ([0, 1], [2, 3, 4], [5])
    assert m.message_state(2, 0) == SUSPENDED and m.entry_tier(2, 0) == T_SUSPENDED
    m.terminate(1)
    assert m.message_state(1, 0) == EXPIRED and m.entry_tier(1, 0) == T_DISCARDED
    assert m.message_pages(1, 0) == [0, 1]                # Expired KV stays until capacity is needed
    assert m.free_pages() == 2

    new_ctx(m, 4, 64)                                     # 4 pages: 2 missing, Discarded covers them
    _, adm = serve(m, 4)
    assert (adm["released_entries"], adm["released_pages"], adm["admitted_pages"]) == (1, 2, 4)
    assert m.message_pages(1, 0) is None and m.message_pages(4, 0) == [0, 1, 6, 7]
    assert m.free_pages() == 0

    new_ctx(m, 5, 16)                                     # 1 page: MRU takes context 4's (4 pages)
    _, adm = serve(m, 5)
    assert (adm["released_entries"], adm["released_pages"]) == (1, 4)
    assert m.message_pages(4, 0) is None and m.message_pages(3, 0) == [5] and m.message_pages(2, 0) == [2, 3, 4]
    assert m.message_pages(5, 0) == [0] and m.free_pages() == 3

    # context 2 runs again with a new message: its old entry re-enters
    # Suspended now, its new one in the same call (created later: newer)
    m.append(2, 16)
    hit, adm = serve(m, 2)
    assert (hit["hit_tokens"], hit["miss_tokens"]) == (48, 16)
    assert adm["admitted_entries"] == 1 and adm["released_entries"] == 0
    assert m.message_pages(2, 1) == [1] and m.free_pages() == 2

    new_ctx(m, 6, 64)                                     # 2 missing: context 2's new entry, then its old one
    _, adm = serve(m, 6)
    assert (adm["released_entries"], adm["released_pages"]) == (2, 4)
    assert m.message_pages(2, 0) is None and m.message_pages(2, 1) is None
    assert m.message_pages(3, 0) == [5] and m.message_pages(5, 0) == [0] and m.message_pages(6, 0) == [1, 2, 3, 4]

    # context 2's first message lost its KV, so both messages are misses; the
    # write-back needs 3 + 1 pages with 2 free: MRU takes context 6's entry
    hit, adm = serve(m, 2)
    assert (hit["hit_tokens"], hit["miss_tokens"]) == (0, 64)
    assert (adm["admitted_entries"], adm["admitted_pages"], adm["released_entries"], adm["released_pages"]) == \
        (2, 4, 1, 4)
    assert m.message_pages(2, 0) == [1, 2, 3] and m.message_pages(2, 1) == [4] and m.message_pages(6, 0) is None
    assert m.free_pages() == 2


def test_pin_active_fallback_and_pinned_competition(make):
    m = make(6)
    new_ctx(m, 1, 32, pin=[0])
    serve(m, 1)
    assert m.message_state(1, 0) == PINNED and m.entry_tier(1, 0) == T_PINNED and m.message_pages(1, 0) == [0, 1]
    new_ctx(m, 2, 32)
    serve(m, 2)
    new_ctx(m, 3, 32)
    serve(m, 3)
    m.begin_request(2)                                   # issued, prefill not started: Active, not held
    assert m.message_state(2, 0) == ACTIVE and m.entry_tier(2, 0) == T_ACTIVE

    new_ctx(m, 4, 48)                                    # 3 pages, 0 free: Suspended (2) then Active (2)
    _, adm = serve(m, 4)
    assert (adm["released_entries"], adm["released_pages"], adm["admitted_pages"]) == (2, 4, 3)
    assert m.message_pages(2, 0) is None and m.message_pages(3, 0) is None
    assert m.message_pages(4, 0) == [2, 3, 4] and m.message_pages(1, 0) == [0, 1] and m.free_pages() == 1
    hit = m.start_prefill(2)
    assert (hit["hit_tokens"], hit["miss_tokens"]) == (0, 32)
    m.end_request(2)                                     # aborted before prefill finished

    new_ctx(m, 5, 80)                                    # 5 pages, 1 free: Suspended frees 3, still short
    _, adm = serve(m, 5)
    assert (adm["released_entries"], adm["released_pages"], adm["rejected_entries"], adm["admitted_entries"]) == \
        (1, 3, 1, 0)
    assert m.message_pages(5, 0) is None and m.message_pages(1, 0) == [0, 1]   # Pinned untouched
    assert m.free_pages() == 4                           # freed pages stay freed

    new_ctx(m, 6, 80, pin=[0])                           # a Pinned newcomer competes with Pinned KV
    _, adm = serve(m, 6)
    assert (adm["released_entries"], adm["released_pages"], adm["admitted_pages"]) == (1, 2, 5)
    assert m.message_pages(1, 0) is None and m.message_pages(6, 0) == [0, 1, 2, 3, 4]


def test_pin_temporary_bypasses_the_cache(make):
    m = make(4)
    m.spawn(1)
    m.append(1, 16)
    m.one_off(1)
    m.append(1, 20)
    assert m.message_state(1, 0) == TEMPORARY and m.message_state(1, 1) == TEMPORARY
    with pytest.raises(_err(m)):
        m.pin(1, 0)
    hit, adm = serve(m, 1)
    assert hit["miss_tokens"] == 36
    assert (adm["bypassed_entries"], adm["admitted_entries"], adm["released_entries"]) == (2, 0, 0)
    assert m.message_pages(1, 0) is None and m.free_pages() == 4
    assert m.entry_tier(1, 0) == T_DISCARDED
    hit, _ = serve(m, 1)
    assert hit["miss_tokens"] == 36                      # never reused


def test_pin_shared_kv_takes_the_strongest_state(make):
    m = make(8)
    new_ctx(m, 1, 32)
    serve(m, 1)
    m.fork(1, 2)
    assert m.message_pages(2, 0) == [0, 1] and m.message_state(2, 0) == SUSPENDED
    m.pin(2, 0)                                          # the child's protection covers the shared KV
    assert m.message_state(1, 0) == SUSPENDED and m.message_state(2, 0) == PINNED
    assert m.entry_tier(1, 0) == T_PINNED
    m.unpin(2, 0)
    assert m.message_state(2, 0) == SUSPENDED and m.entry_tier(1, 0) == T_SUSPENDED
    m.terminate(1)                                       # parent gone, child still Suspended
    assert m.message_state(1, 0) == EXPIRED and m.entry_tier(2, 0) == T_SUSPENDED
    hit, _ = serve(m, 2)
    assert (hit["hit_tokens"], hit["miss_tokens"]) == (32, 0)
    m.terminate(2)
    assert m.entry_tier(2, 0) == T_DISCARDED
    new_ctx(m, 3, 128)                                   # 8 pages, 6 free: the shared KV is reclaimed
    _, adm = serve(m, 3)
    assert (adm["released_entries"], adm["released_pages"], adm["admitted_pages"]) == (1, 2, 8)
    assert m.message_pages(3, 0) == list(range(8))


def test_pin_in_flight_kv_is_not_released(make):
    m = make(4)
    new_ctx(m, 1, 32)
    serve(m, 1)
    new_ctx(m, 2, 32)
    serve(m, 2)
    m.begin_request(1)
    hit = m.start_prefill(1)                             # context 1's prefill reads its entry
    assert hit["hit_tokens"] == 32 and m.entry_tier(1, 0) == T_ACTIVE
    new_ctx(m, 3, 48)
    _, adm = serve(m, 3)                                 # Suspended frees 2; the held Active entry is skipped
    assert (adm["released_entries"], adm["released_pages"], adm["rejected_entries"]) == (1, 2, 1)
    assert m.message_pages(1, 0) == [0, 1]
    m.prefill_done(1)
    m.end_request(1)
    assert m.message_state(1, 0) == SUSPENDED
    _, adm = serve(m, 3)                                 # now it may go
    assert (adm["released_entries"], adm["admitted_pages"]) == (1, 3)
    assert m.message_pages(1, 0) is None and m.message_pages(3, 0) == [0, 1, 2]


def test_pin_replace_and_remove_expire_the_suffix(make):
    m = make(8)
    new_ctx(m, 1, 16, 16, 16)
    serve(m, 1)
    assert [m.message_pages(1, i) for i in range(3)] == [[0], [1], [2]]
    m.replace(1, 1, 32)                                  # message 1 and the later one change
    assert m.message_state(1, 0) == SUSPENDED
    assert m.message_state(1, 1) == ACTIVE and m.message_state(1, 2) == ACTIVE
    assert m.entry_tier(1, 1) is None and m.message_pages(1, 2) is None
    hit, adm = serve(m, 1)
    assert (hit["hit_tokens"], hit["miss_tokens"]) == (16, 48)
    assert (adm["admitted_entries"], adm["admitted_pages"]) == (2, 3)
    assert m.message_pages(1, 1) == [3, 4] and m.message_pages(1, 2) == [5]
    new_ctx(m, 2, 48)                                    # 1 missing: the old version of message 1 goes first
    _, adm = serve(m, 2)
    assert (adm["released_entries"], adm["released_pages"]) == (1, 1)
    assert m.message_pages(2, 0) == [1, 6, 7]
    m.remove(1, 0)                                       # everything after it changes too
    assert [m.message_state(1, i) for i in range(2)] == [ACTIVE, ACTIVE]
    assert m.message_pages(1, 0) is None and m.message_pages(1, 1) is None
    # 5 pages, none free: the Discarded tier alone covers it, earliest first:
    # old message 2 ([2], from the replace), then message 0 and the replayed
    # 1 and 2 (one call: creation order); context 2's Suspended KV stays
    new_ctx(m, 3, 80)
    _, adm = serve(m, 3)
    assert (adm["released_entries"], adm["released_pages"]) == (4, 5)
    assert m.message_pages(3, 0) == [0, 2, 3, 4, 5] and m.message_pages(2, 0) == [1, 6, 7]


def test_pin_event_rules(make):
    m = make(4)
    m.spawn(1)
    with pytest.raises(_err(m)):
        m.spawn(1)
    with pytest.raises(_err(m)):
        m.append(1, 0)
    m.append(1, 5)
    with pytest.raises(_err(m)):
        m.unpin(1, 0)                                    # not pinned
    with pytest.raises(_err(m)):
        m.pin(1, 1)                                      # no such message
    with pytest.raises(_err(m)):
        m.start_prefill(1)                               # not issued
    m.begin_request(1)
    for bad in (lambda: m.begin_request(1), lambda: m.fork(1, 2), lambda: m.terminate(1), lambda: m.one_off(1),
                lambda: m.replace(1, 0, 3), lambda: m.remove(1, 0), lambda: m.prefill_done(1)):
        with pytest.raises(_err(m)):
            bad()
    m.pin(1, 0)
    m.unpin(1, 0)
    assert m.message_state(1, 0) == ACTIVE               # unpinned during a request
    m.start_prefill(1)
    m.prefill_done(1)
    m.end_request(1)
    m.pin(1, 0)
    m.terminate(1)
    assert m.message_state(1, 0) == PINNED               # Pinned keeps its protection
    assert m.message_pages(1, 0) == [0]
    with pytest.raises(_err(m)):
        m.append(1, 3)
    m.unpin(1, 0)
    assert m.message_state(1, 0) == EXPIRED and m.entry_tier(1, 0) == T_DISCARDED


@pytest.mark.parametrize("pages", [0, 1, 63, 64, 65, 4095, 4096, 4097, 70000])
def test_pool_sizes_across_bitmap_words(pages):
    """Fill the pool, free a scattered part of it and refill: the library's
    two-level bitmap hands out the same lowest ids as the oracle's set."""
    o, lib = OracleManager(pages), kvt.Manager(pages)
    assert lib.free_pages() == pages
    rng = np.random.default_rng(pages)
    sizes = []
    left = pages
    while left > 0:
        t = int(rng.integers(1, 40 * 16))
        sizes.append(t)
        left -= (t + 15) // 16
    for m in (o, lib):
        for c, t in enumerate(sizes):
            new_ctx(m, c, t)
            serve(m, c)
        for c in range(0, len(sizes), 3):
            m.terminate(c)
        new_ctx(m, 10**6, max(1, pages // 2) * 16)
        serve(m, 10**6)
    for c in list(range(len(sizes))) + [10**6]:
        assert o.message_pages(c, 0) == lib.message_pages(c, 0), c
    assert o.free_pages() == lib.free_pages()


def test_replay_equals_the_calls_one_by_one():
    """kvt_mgr_replay runs an encoded trace exactly as the calls would: the
    same successes, summed reports, free pages and final page ids."""
    from paper_2609_39819_amd.workloads import agent_events
    events = list(agent_events(seed=3, agents=40, concurrency=10))
    events += [("pin", (10**6, 0)), ("append", (0, 0)), ("fork", (0, 0))]       # three that fail
    one, rep = kvt.Manager(2048), kvt.Manager(2048)
    ok1, tot = 0, {k: 0 for k in REPORT_KEYS}
    for op, args in events:
        try:
            r = getattr(one, op)(*args)
        except kvt.KvtError:
            continue
        ok1 += 1
        for k in tot:
            tot[k] += (r or {}).get(k, 0)
    ok2, tot2 = rep.replay(kvt.Manager.encode(events))
    assert (ok2, tot2) == (ok1, tot) and ok1 == len(events) - 3
    assert one.free_pages() == rep.free_pages()
    for c in range(200):
        for i in range(60):
            assert one.message_pages(c, i) == rep.message_pages(c, i)
    bad = np.array([[99, 0, 0, 0]], dtype=np.int64)                             # unknown op: skipped
    assert rep.replay(bad) == (0, {k: 0 for k in REPORT_KEYS})
    assert kvt.lib().kvt_mgr_replay(None, None, 0, None) == -1
    assert kvt.lib().kvt_mgr_replay(rep._h, None, 1, None) == -1
    assert kvt.lib().kvt_mgr_replay(rep._h, None, 0, None) == 0


def test_manager_bounds():
    lib = kvt.Manager(4)
    lib.spawn(1)
    for bad in (0, -5, (1 << 40) + 1):
        with pytest.raises(kvt.KvtError):
            lib.append(1, bad)
    lib.append(1, 1 << 40)                               # the largest message is accepted ...
    lib.begin_request(1)
    lib.start_prefill(1)
    assert lib.prefill_done(1)["rejected_entries"] == 1  # ... and does not fit
    lib.append(1, 20)
    lib.end_request(1)
    serve(lib, 1)
    assert kvt.lib().kvt_mgr_message_pages(lib._h, 1, 1, None, 5) == 2   # NULL buffer: count only
    assert lib.message_pages(1, 1) == [0, 1]
    assert kvt.Manager(0).free_pages() == 0
    with pytest.raises(ValueError):
        kvt.Manager(-1)
    with pytest.raises(ValueError):
        kvt.Manager(1 << 31)


# ---------------------------------------------------------------------------
# library vs oracle on seeded random event streams
# ---------------------------------------------------------------------------

OPS = ("spawn", "fork", "append", "one_off", "pin", "unpin", "replace", "remove", "terminate", "begin_request",
       "start_prefill", "prefill_done", "end_request")


class RandomDriver:
    """Seeded calls, mostly ones the state allows (read off the oracle's
    contexts), a tenth of them arbitrary -- unknown contexts, bad indexes,
    events out of order -- which both sides must reject alike."""

    def __init__(self, seed, live_target):
        self.rng = np.random.default_rng(seed)
        self.live_target = live_target
        self.next_id = 0

    def _new_id(self):
        self.next_id += 1
        return self.next_id - 1

    def next(self, o):
        rng = self.rng
        if rng.random() < 0.1:
            op = OPS[int(rng.integers(0, len(OPS)))]
            c = int(rng.integers(-1, self.next_id + 1))
            i = int(rng.integers(-1, 6))
            return op, {"spawn": (c,), "fork": (c, int(rng.integers(0, self.next_id + 1))), "append": (c, i * 9),
                        "pin": (c, i), "unpin": (c, i), "remove": (c, i), "replace": (c, i, i * 7)}.get(op, (c,))
        live = [c for c, x in o.ctxs.items() if not x.terminated]
        if len(live) < self.live_target and rng.random() < 0.3:
            if live and rng.random() < 0.4:
                idle = [c for c in live if o.ctxs[c].phase == 0]
                if idle:
                    return "fork", (int(rng.choice(idle)), self._new_id())
            return "spawn", (self._new_id(),)
        if not live:
            return "spawn", (self._new_id(),)
        c = int(rng.choice(live))
        x = o.ctxs[c]
        n = len(x.msgs)
        i = int(rng.integers(0, n)) if n else 0
        tokens = int(rng.integers(1, 90))
        if x.phase == 0:
            choices = ["append"] * 3 + ["begin_request"] * 4 + ["pin", "unpin", "replace", "remove"] + \
                      ["terminate"] * (1 if len(live) > self.live_target or rng.random() < 0.1 else 0) + ["one_off"] * (1 if rng.random() < 0.05 else 0) + \
                      ["fork"] * (1 if len(live) < 2 * self.live_target else 0)
        else:
            nxt = {1: "start_prefill", 2: "prefill_done", 3: "end_request"}[x.phase]
            choices = [nxt] * 6 + ["end_request", "append", "pin", "unpin"]
        op = choices[int(rng.integers(0, len(choices)))]
        if op in ("pin", "unpin") and n:
            cand = [j for j, v in enumerate(x.msgs) if (v.state == PINNED) == (op == "unpin")]
            if cand:
                i = int(rng.choice(cand))
        return op, {"append": (c, tokens), "pin": (c, i), "unpin": (c, i), "remove": (c, i),
                    "replace": (c, i, tokens), "fork": (c, self._new_id())}.get(op, (c,))


def _observe(m, ctx_lens):
    out = [m.free_pages()]
    for c in sorted(ctx_lens):
        for i in range(ctx_lens[c]):
            out.append((c, i, m.message_state(c, i), m.entry_tier(c, i), m.message_pages(c, i)))
    return out


def _release_order(entries, pinned_too):
    d = sorted((e for e in entries if e.tier == T_DISCARDED), key=lambda e: e.since)
    s = sorted((e for e in entries if e.tier == T_SUSPENDED), key=lambda e: e.since, reverse=True)
    a = sorted((e for e in entries if e.tier == T_ACTIVE), key=lambda e: e.since)
    p = sorted((e for e in entries if e.tier == T_PINNED), key=lambda e: e.since) if pinned_too else []
    return d + s + a + p


class Checker:
    """Properties of the oracle's state that Algorithm 1 and the hold rule fix,
    with the holds tracked here from the call sequence (not from the
    oracle's own counters): a context's resident KV is held from its
    start_prefill, its new KV from its prefill_done, until its end_request."""

    def __init__(self, o, num_pages):
        self.o, self.num_pages, self.held = o, num_pages, {}

    def _held(self):
        return {id(e): e for es in self.held.values() for e in es}

    def before(self, op):
        if op != "prefill_done":
            return None
        held = self._held()
        res = [e for e in self.o.entries if e.resident]
        return [e for e in res if id(e) not in held], len(self.o.free), len(self.o.entries)

    def after(self, op, args, rep, snap):
        o = self.o
        if op in ("start_prefill", "prefill_done"):
            c = args[0]
            self.held.setdefault(c, []).extend(v.entry for v in o.ctxs[c].msgs
                                               if v.entry is not None and v.entry.resident)
        elif op == "end_request":
            self.held.pop(args[0], None)
        if op == "prefill_done":
            self._write_back(snap, rep)
        owned = [p for e in o.entries if e.resident for p in e.page_ids]
        assert len(owned) == len(set(owned)) and not set(owned) & o.free
        assert set(owned) | o.free == set(range(self.num_pages))
        for e in o.entries:
            assert len(e.page_ids) == (e.pages if e.resident else 0)
        assert all(e.resident for e in self._held().values()), "held KV was released"

    def _write_back(self, snap, rep):
        """One prefill_done: the released KV is a prefix of the tier order."""
        releasable, free_before, known = snap
        fresh = self.o.entries[known:]
        released = [e for e in releasable if not e.resident]
        temporary = [e for e in fresh if all(v.state == TEMPORARY for v in e.versions)]
        assert not any(e.resident for e in temporary) and rep["bypassed_entries"] == len(temporary)
        pinned_newcomer = any(e.tier == T_PINNED for e in fresh if e not in temporary)
        order = _release_order(releasable, pinned_newcomer)
        assert set(map(id, released)) == set(map(id, order[:len(released)])), \
            "released KV is not a prefix of the order"
        assert len(released) == rep["released_entries"] and sum(e.pages for e in released) == rep["released_pages"]
        if released:
            need = sum(e.pages for e in fresh if e not in temporary)
            assert free_before + rep["released_pages"] - order[len(released) - 1].pages < need, "released too much"


@pytest.mark.parametrize("seed,num_pages,live", [(1, 24, 6), (2, 24, 10), (3, 48, 8), (4, 12, 5), (5, 96, 14),
                                                 (6, 30, 8), (7, 16, 4), (8, 64, 12)])
def test_library_matches_the_oracle_on_random_streams(seed, num_pages, live):
    o, lib = OracleManager(num_pages), kvt.Manager(num_pages)
    chk = Checker(o, num_pages)
    ok = {"prefill_done": 0, "start_prefill": 0, "released": 0, "rejected": 0}
    drv = RandomDriver(seed, live)
    for step in range(1500):
        op, args = drv.next(o)
        snap = chk.before(op)
        try:
            r_o, e_o = getattr(o, op)(*args), None
        except ValueError as ex:
            r_o, e_o = None, ex
        try:
            r_l, e_l = getattr(lib, op)(*args), None
        except kvt.KvtError as ex:
            r_l, e_l = None, ex
        assert (e_o is None) == (e_l is None), f"step {step} {op}{args}: oracle {e_o!r} library {e_l!r}"
        assert r_o == r_l, f"step {step} {op}{args}: {r_o} != {r_l}"
        if e_o is None:
            ok[op] = ok.get(op, 0) + 1
            chk.after(op, args, r_o, snap)
            if op == "prefill_done":
                ok["released"] += r_o["released_entries"]
                ok["rejected"] += r_o["rejected_entries"]
        lens = {c: len(x.msgs) for c, x in o.ctxs.items()}
        assert _observe(o, lens) == _observe(lib, lens), f"step {step} {op}{args}"
        for c, n in lens.items():
            assert lib.message_state(c, n) == -1
    # the stream exercised what it is meant to
    assert ok["prefill_done"] > 100 and ok["released"] > 20 and ok.get("fork", 0) > 10, ok
    assert all(ok.get(op, 0) > 0 for op in OPS), ok


def _drive_oracle(o, seed, live, steps):
    drv, chk = RandomDriver(seed, live), Checker(o, o.free_pages())
    for _ in range(steps):
        op, args = drv.next(o)
        snap = chk.before(op)
        try:
            rep = getattr(o, op)(*args)
        except ValueError:
            continue
        chk.after(op, args, rep, snap)


class _LruOracle(OracleManager):
    """A planted mistake: least recently suspended first inside Suspended."""

    def _admit(self, e, rep):
        for x in self.entries:
            if x.tier == T_SUSPENDED:
                x.since = (-x.since[0], -x.since[1])
        try:
            super()._admit(e, rep)
        finally:
            for x in self.entries:
                if x.tier == T_SUSPENDED:
                    x.since = (-x.since[0], -x.since[1])


class _NoHoldOracle(OracleManager):
    """A planted mistake: KV read by a running prefill may be released."""

    def start_prefill(self, c):
        rep = super().start_prefill(c)
        for e in self.ctxs[c].held:
            e.in_use -= 1
        self.ctxs[c].held = []
        return rep


class _PinnedAlwaysOracle(OracleManager):
    """A planted mistake: every newcomer competes with Pinned KV."""

    def _admit(self, e, rep):
        saved = e.tier
        if e.tier != T_PINNED and not all(v.state == TEMPORARY for v in e.versions):
            e.tier = T_PINNED
        try:
            super()._admit(e, rep)
        finally:
            e.tier = saved


@pytest.mark.parametrize("planted", [_LruOracle, _NoHoldOracle, _PinnedAlwaysOracle])
def test_the_properties_catch_planted_mistakes(planted):
    _drive_oracle(OracleManager(16), 11, 6, 1500)        # the real model passes
    with pytest.raises(AssertionError):
        _drive_oracle(planted(16), 11, 6, 1500)


# ---------------------------------------------------------------------------
# the same C++ source under AddressSanitizer and UBSan (host compiler)
# ---------------------------------------------------------------------------



def _replay_line(m, op, args):
    try:
        r = getattr(m, op)(*args)
        st = kvt.KVT_OK
    except kvt.KvtError as e:
        r, st = None, e.status
    out = str(st)
    if r is not None:
        out += " " + " ".join(str(r[k]) for k in REPORT_KEYS)
    return out + f" free={m.free_pages()}"


def test_manager_source_is_clean_under_sanitizers(tmp_path):
    import os
    import shutil
    import subprocess
    from paper_2609_39819_amd.workloads import agent_events
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = str(tmp_path / "manager_replay")
    build = subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                            "-fno-sanitize-recover=all", "-I", os.path.join(root, "include"),
                            os.path.join(root, "paper_2609_39819_amd", "csrc", "kvt_manager.cpp"),
                            os.path.join(root, "tests", "manager_replay.cpp"), "-o", exe],
                           capture_output=True, text=True)
    if build.returncode != 0 and "asan" in build.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + build.stderr[-300:])
    assert build.returncode == 0, build.stderr[-2000:]

    streams = []
    for seed, pages, live in ((21, 24, 6), (22, 12, 5)):
        o, drv, evs = OracleManager(pages), RandomDriver(seed, live), []
        for _ in range(1500):
            op, args = drv.next(o)
            try:
                getattr(o, op)(*args)
            except ValueError:
                pass
            evs.append((op, args))
        streams.append((pages, evs))
    trace = list(agent_events(seed=5, agents=48, concurrency=12))
    streams += [(4096, trace), (1 << 15, trace)]

    text, want = [], []
    for k, (pages, evs) in enumerate(streams):
        text.append(f"pages {pages}")
        want.append("ok")
        lib = kvt.Manager(pages)
        for op, args in evs:
            text.append(" ".join([op] + [str(a) for a in args]))
            want.append(_replay_line(lib, op, args))
        ok, tot = kvt.Manager(pages).replay(kvt.Manager.encode(evs))
        summary = (f"replay ok={ok} hit={tot['hit_tokens']} miss={tot['miss_tokens']} "
                   f"admitted={tot['admitted_pages']} released={tot['released_pages']} free={lib.free_pages()}")
        lib.close()
        if k > 0:
            want.insert(len(want) - len(evs) - 1, prev_summary)
        prev_summary = summary
    want.append(prev_summary)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], input="\n".join(text) + "\n", capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stderr[-3000:]
    got = run.stdout.splitlines()
    assert len(got) == len(want)
    bad = [i for i, (g, w) in enumerate(zip(got, want)) if g != w]
    assert not bad, f"first mismatch at line {bad[0]}: {text[bad[0]]!r}: {got[bad[0]]!r} != {want[bad[0]]!r}"
