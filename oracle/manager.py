"""Plain model of the KV lifecycle manager and state-guided cache (test oracle).

TEST INFRASTRUCTURE -- see the package docstring.  Pure Python, linear scans,
no indexing structures; written from the paper's description:

* §5.2 -- lifecycle states per message version and context: Pinned; Active
  when appended or taking part in a request; Suspended once prefill is done;
  Expired when the context terminates or the message (or one before it) is
  removed or replaced; Temporary for a one-off context.  Forked children keep
  their own states for inherited messages.
* §6.1 -- shared KV takes the strongest state among the versions mapped to it
  (Pinned > Active > Suspended > Discarded = Expired or Temporary), and
  Algorithm 1 admits written-back KV: bypass Temporary; Delta = size - free;
  free Expired (Discarded), then Suspended, then Active, then Pinned only for
  a Pinned newcomer, each while Delta > 0; admit if Delta <= 0.  KV under an
  in-flight request is reclaimed only after that request.
* §6.2 -- inside the Suspended tier the most recently suspended KV goes first.

Readings of points the paper leaves open (the same ones the library states):
earliest-first inside Discarded, Active and Pinned (entries that changed
tier in one call rank by creation order, in every tier); pages taken lowest id
first; KV freed on the way stays freed if the newcomer still does not fit; a
message whose KV is gone at a request -- and every later message of its
context -- is a miss and gets a fresh version; replacing or removing a
message expires its version and every later one (a pinned one included),
the later messages getting fresh Active (Temporary if one-off) versions;
unpin during a request gives Active, in a one-off context Temporary; one_off
leaves Pinned messages Pinned (as terminate does).  Because the pages are the ones the
kernels read, KV is held from the start of the prefill that reads it to the
end of the request (in every tier); an issued request whose prefill has not
started holds nothing, and its reactivated KV is the Active tier.
"""
from __future__ import annotations

PINNED, ACTIVE, SUSPENDED, EXPIRED, TEMPORARY = 0, 1, 2, 3, 4
MAX_TOKENS = 1 << 40                # per message (the library's bound)
T_PINNED, T_ACTIVE, T_SUSPENDED, T_DISCARDED = 0, 1, 2, 3


class _Entry:
    def __init__(self, pages):
        self.pages = pages
        self.versions = []          # the message versions mapped to it (shared objects)
        self.resident = False
        self.page_ids = []
        self.in_use = 0
        self.tier = None
        self.since = (0, 0)         # (event, creation index) when the current tier was entered
        self.index = 0


class _Version:
    def __init__(self, state, tokens):
        self.state = state
        self.tokens = tokens
        self.entry = None


IDLE, ISSUED, PREFILLING, DECODING = 0, 1, 2, 3


class _Context:
    def __init__(self):
        self.msgs = []              # current _Version of each message
        self.terminated = False
        self.one_off = False
        self.phase = IDLE           # of the context's LLM request
        self.held = []              # entries its prefill and decode read


class OracleManager:
    def __init__(self, num_pages):
        self.free = set(range(num_pages))
        self.ctxs = {}
        self.entries = []           # every entry ever created
        self.event = 0              # public state-changing calls so far

    # ---- aggregate state (§6.1)
    def _tier_now(self, e):
        states = [v.state for v in e.versions]
        for t, s in ((T_PINNED, PINNED), (T_ACTIVE, ACTIVE), (T_SUSPENDED, SUSPENDED)):
            if s in states:
                return t
        return T_DISCARDED

    def _refresh(self):
        """Recompute every entry's tier; an entry whose tier changed entered it
        in the current event (entries moved in one event rank by creation)."""
        for e in self.entries:
            t = self._tier_now(e)
            if t != e.tier:
                e.tier, e.since = t, (self.event, e.index)

    def _set(self, v, state):
        if v.state != state:
            v.state = state
            self._refresh()

    def _tick(self):
        self.event += 1

    # ---- Algorithm 1 (§6.1) with MRU inside Suspended (§6.2)
    def _admit(self, e, rep):
        if e.versions and all(v.state == TEMPORARY for v in e.versions):
            rep["bypassed_entries"] += 1
            return
        delta = e.pages - len(self.free)
        order = [(T_DISCARDED, False), (T_SUSPENDED, True), (T_ACTIVE, False)]
        if e.tier == T_PINNED:
            order.append((T_PINNED, False))
        for tier, newest_first in order:
            while delta > 0:
                cands = [x for x in self.entries if x.resident and x.tier == tier and x.in_use == 0]
                if not cands:
                    break
                victim = (max if newest_first else min)(cands, key=lambda x: x.since)
                victim.resident = False
                self.free.update(victim.page_ids)
                victim.page_ids = []
                rep["released_entries"] += 1
                rep["released_pages"] += victim.pages
                delta -= victim.pages
        if delta <= 0:
            e.page_ids = sorted(self.free)[:e.pages]
            self.free.difference_update(e.page_ids)
            e.resident = True
            rep["admitted_entries"] += 1
            rep["admitted_pages"] += e.pages
        else:
            rep["rejected_entries"] += 1

    @staticmethod
    def _report():
        return dict(admitted_entries=0, admitted_pages=0, bypassed_entries=0, rejected_entries=0,
                    released_entries=0, released_pages=0, hit_tokens=0, miss_tokens=0)

    def _ctx(self, c, live=True):
        if c not in self.ctxs or (live and self.ctxs[c].terminated):
            raise ValueError("unknown or terminated context")
        return self.ctxs[c]

    @staticmethod
    def _msg(ctx, i):
        if not 0 <= i < len(ctx.msgs):
            raise ValueError("bad message index")
        return ctx.msgs[i]

    def _fresh(self, ctx, tokens):
        return _Version(TEMPORARY if ctx.one_off else ACTIVE, tokens)

    # ---- context events (§5.2)
    def spawn(self, c):
        self._tick()
        if c in self.ctxs:
            raise ValueError("context exists")
        self.ctxs[c] = _Context()

    def fork(self, parent, child):
        self._tick()
        p = self._ctx(parent)
        if p.phase != IDLE or child in self.ctxs:
            raise ValueError("fork during a request or onto an existing context")
        k = _Context()
        for v in p.msgs:
            nv = _Version(v.state, v.tokens)
            nv.entry = v.entry
            if v.entry is not None:
                v.entry.versions.append(nv)
            k.msgs.append(nv)
        self.ctxs[child] = k
        self._refresh()

    def append(self, c, tokens):
        self._tick()
        if not 1 <= tokens <= MAX_TOKENS:
            raise ValueError("bad message size")
        ctx = self._ctx(c)
        ctx.msgs.append(self._fresh(ctx, tokens))

    def one_off(self, c):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != IDLE:
            raise ValueError("one_off during a request")
        ctx.one_off = True
        for v in ctx.msgs:
            if v.state != PINNED:
                self._set(v, TEMPORARY)

    def pin(self, c, i):
        self._tick()
        ctx = self._ctx(c)
        v = self._msg(ctx, i)
        if v.state == TEMPORARY:
            raise ValueError("a Temporary message is not pinned")
        self._set(v, PINNED)

    def unpin(self, c, i):
        self._tick()
        ctx = self._ctx(c, live=False)
        v = self._msg(ctx, i)
        if v.state != PINNED:
            raise ValueError("not pinned")
        if ctx.terminated:
            self._set(v, EXPIRED)
        elif ctx.one_off:
            self._set(v, TEMPORARY)
        else:
            self._set(v, ACTIVE if ctx.phase != IDLE else SUSPENDED)

    def _expire_from(self, ctx, i):
        for j in range(i, len(ctx.msgs)):
            old = ctx.msgs[j]
            self._set(old, EXPIRED)                # stays mapped to its entry as an Expired version
            ctx.msgs[j] = self._fresh(ctx, old.tokens)

    def replace(self, c, i, tokens):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != IDLE or not 1 <= tokens <= MAX_TOKENS or not 0 <= i < len(ctx.msgs):
            raise ValueError("bad replace")
        self._expire_from(ctx, i)
        ctx.msgs[i].tokens = tokens

    def remove(self, c, i):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != IDLE or not 0 <= i < len(ctx.msgs):
            raise ValueError("bad remove")
        self._expire_from(ctx, i)
        del ctx.msgs[i]

    def terminate(self, c):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != IDLE:
            raise ValueError("terminate during a request")
        ctx.terminated = True
        for v in ctx.msgs:
            if v.state in (ACTIVE, SUSPENDED):
                self._set(v, EXPIRED)

    # ---- request boundaries
    def begin_request(self, c):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != IDLE:
            raise ValueError("already in a request")
        ctx.phase = ISSUED
        for v in ctx.msgs:
            if v.state == SUSPENDED:
                self._set(v, ACTIVE)

    def start_prefill(self, c):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != ISSUED:
            raise ValueError("no issued request")
        rep = self._report()
        ctx.phase = PREFILLING
        lost = False
        for i, v in enumerate(ctx.msgs):
            if v.entry is not None and (lost or not v.entry.resident):
                v.entry.versions.remove(v)         # this version's KV is gone
                v.entry = None
                self._refresh()
            if v.entry is None:
                lost = True
                rep["miss_tokens"] += v.tokens
            else:
                rep["hit_tokens"] += v.tokens
                v.entry.in_use += 1
                ctx.held.append(v.entry)
        return rep

    def prefill_done(self, c):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase != PREFILLING:
            raise ValueError("no prefill running")
        rep = self._report()
        ctx.phase = DECODING
        fresh = []
        for v in ctx.msgs:
            if v.entry is None:
                e = _Entry((v.tokens + 15) // 16)
                e.index = len(self.entries)
                e.versions.append(v)
                v.entry = e
                e.in_use += 1
                ctx.held.append(e)
                self.entries.append(e)
                self._refresh()
                fresh.append(e)
        for v in ctx.msgs:
            if v.state == ACTIVE:
                self._set(v, SUSPENDED)
        for e in fresh:
            self._admit(e, rep)
        return rep

    def end_request(self, c):
        self._tick()
        ctx = self._ctx(c)
        if ctx.phase == IDLE:
            raise ValueError("no request")
        for e in ctx.held:
            e.in_use -= 1
        ctx.held = []
        ctx.phase = IDLE
        for v in ctx.msgs:
            if v.state == ACTIVE:
                self._set(v, SUSPENDED)

    # ---- queries
    def free_pages(self):
        return len(self.free)

    def message_state(self, c, i):
        return self.ctxs[c].msgs[i].state

    def message_pages(self, c, i):
        v = self.ctxs[c].msgs[i]
        if v.entry is None or not v.entry.resident:
            return None
        return list(v.entry.page_ids)

    def entry_tier(self, c, i):
        v = self.ctxs[c].msgs[i]
        return None if v.entry is None else v.entry.tier
