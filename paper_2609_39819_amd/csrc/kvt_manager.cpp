// Host block manager: message lifecycle states, shared-KV aggregate state,
// state-prioritized admission and MRU eviction inside the Suspended tier,
// over a pool of KV pages.
//
// Model (paper §5.2, §6.1, §6.2):
//  * a context is an ordered list of messages; each message has a current
//    version with a lifecycle state (Pinned, Active, Suspended, Expired,
//    Temporary) and, once it took part in inference, a KV entry;
//  * an entry is a run of pages that one or more message versions map to
//    (a forked child maps its inherited messages to its parent's entries);
//    its aggregate state is the strongest state among the versions that map
//    it (Pinned > Active > Suspended > Discarded, where Expired and Temporary
//    count as Discarded), and it is Discarded only when every mapped version
//    is;
//  * new KV is written back after prefill and admitted by Algorithm 1:
//    Temporary bypasses the cache; otherwise the missing capacity is freed
//    from resident entries in the order Discarded, Suspended (most recently
//    suspended first), Active, and -- for a Pinned newcomer only -- Pinned;
//    the newcomer is admitted if that covered its size.  Entries read by an
//    in-flight request are not released until the request ends.
//
// Readings where the paper is silent (each fixed here and in the header):
//  * release order inside Discarded, Active and Pinned: the entry that
//    entered that state earliest goes first (entries that changed state in
//    one call rank by creation order, in every tier);
//  * pages are taken from the lowest-numbered free pages;
//  * entries released while making room stay released even if the newcomer
//    is still not admitted (the procedure frees before it decides);
//  * a message whose entry was evicted counts as a miss at the next request
//    and gets a fresh version to be recomputed and written back;
//  * the pages of this pool are the ones the attention kernels read, so an
//    entry is held -- not released in any tier -- from the start of the
//    prefill that reads it to the end of its request; a request that was
//    issued but has not started prefill holds nothing, so its reactivated
//    (Active) entries are what the Active step of Algorithm 1 can take.
#include <algorithm>
#include <cstdint>
#include <map>
#include <set>
#include <unordered_map>
#include <vector>

#include "kvt.h"

namespace {

enum State : int { kPinned = 0, kActive = 1, kSuspended = 2, kExpired = 3, kTemporary = 4 };
constexpr int64_t kMaxTokens = int64_t{1} << 40;   // per message; keeps page counts far from overflow
constexpr int kStates = 5;
// aggregate tiers, strongest first; Expired and Temporary both map to Discarded
enum Tier : int { kTierPinned = 0, kTierActive = 1, kTierSuspended = 2, kTierDiscarded = 3 };

struct Entry {
  int64_t pages = 0;                 // size in pages
  int64_t refs[kStates] = {0, 0, 0, 0, 0};
  int tier = kTierDiscarded;
  bool only_temporary = false;       // every mapped version is Temporary
  int64_t stamp = 0;                 // event that last moved it into its tier
  bool resident = false;
  std::vector<int32_t> page_ids;
  int64_t in_use = 0;                // in-flight requests reading it
};

struct Message {
  int state = kActive;
  int64_t entry = -1;                // -1: not materialized (no KV yet)
  int64_t tokens = 0;
};

// where a context's LLM request is: none, issued (messages reactivated),
// prefilling (hits resolved, resident entries held), decoding
enum Phase : int { kIdle = 0, kIssued = 1, kPrefilling = 2, kDecoding = 3 };

struct Context {
  std::vector<Message> msgs;
  bool terminated = false;
  bool one_off = false;
  int phase = kIdle;
  std::vector<int64_t> using_entries;   // entries this context's request holds
};

// Free pages as a two-level bitmap (a set bit is a free page; a summary bit
// marks a word with a free page), so handing out the lowest free ids and
// returning pages cost O(1) per page plus a scan of the summary.
class PageSet {
 public:
  void reset(int64_t n) {
    words_.assign((size_t)((n + 63) / 64), ~0ull);
    if (n % 64) words_.back() = (1ull << (n % 64)) - 1;
    summary_.assign((words_.size() + 63) / 64, ~0ull);
    if (words_.size() % 64) summary_.back() = (1ull << (words_.size() % 64)) - 1;
    count_ = n;
    lo_ = 0;
  }
  int64_t size() const { return count_; }
  void give(int32_t p) {
    words_[(size_t)p >> 6] |= 1ull << (p & 63);
    summary_[(size_t)p >> 12] |= 1ull << ((p >> 6) & 63);
    lo_ = std::min(lo_, (size_t)p >> 12);
    ++count_;
  }
  // the lowest free page, taken; the caller checks size() first
  int32_t take_lowest() {
    size_t s = lo_;
    while (summary_[s] == 0) ++s;
    lo_ = s;
    const size_t w = s * 64 + (size_t)__builtin_ctzll(summary_[s]);
    const int b = __builtin_ctzll(words_[w]);
    words_[w] &= words_[w] - 1;
    if (words_[w] == 0) summary_[s] &= ~(1ull << (w & 63));
    --count_;
    return (int32_t)(w * 64 + (size_t)b);
  }

 private:
  std::vector<uint64_t> words_, summary_;
  int64_t count_ = 0;
  size_t lo_ = 0;   // no summary word below it has a free page
};

}  // namespace

struct kvt_manager {
  int64_t num_pages = 0;
  PageSet free_pages;
  std::unordered_map<int64_t, Entry> entries;
  int64_t next_entry = 0;           // entry ids in creation order
  int64_t event = 0;                // API calls so far
  // releasable entries (resident, held by no request) per tier, ordered by
  // (stamp, entry id): entries that moved in one event rank by creation order
  std::set<std::pair<int64_t, int64_t>> by_tier[4];
  std::unordered_map<int64_t, Context> ctxs;

  static bool listed(const Entry& e) { return e.resident && e.in_use == 0; }

  // ---- aggregate state of an entry
  void retier(int64_t id) {
    Entry& e = entries[id];
    int t = kTierDiscarded;
    for (int s = kPinned; s <= kSuspended; ++s)
      if (e.refs[s] > 0) { t = s; break; }
    e.only_temporary = e.refs[kTemporary] > 0 && e.refs[kPinned] + e.refs[kActive] + e.refs[kSuspended] +
                                                     e.refs[kExpired] == 0;
    if (t == e.tier) return;
    if (listed(e)) by_tier[e.tier].erase({e.stamp, id});
    e.tier = t;
    e.stamp = event;
    if (listed(e)) by_tier[e.tier].insert({e.stamp, id});
  }
  // a request starts or stops reading the entry
  void hold(int64_t id) {
    Entry& e = entries[id];
    if (listed(e)) by_tier[e.tier].erase({e.stamp, id});
    e.in_use += 1;
  }
  void unhold(int64_t id) {
    Entry& e = entries[id];
    e.in_use -= 1;
    if (listed(e)) by_tier[e.tier].insert({e.stamp, id});
    maybe_erase(id);
  }
  void ref(int64_t id, int state, int delta) {
    if (id < 0) return;
    entries[id].refs[state] += delta;
    retier(id);
    maybe_erase(id);
  }
  // an entry no version maps, holding no pages and read by no request is gone
  void maybe_erase(int64_t id) {
    auto it = entries.find(id);
    if (it == entries.end()) return;
    const Entry& e = it->second;
    int64_t refs = 0;
    for (int s = 0; s < kStates; ++s) refs += e.refs[s];
    if (refs == 0 && !e.resident && e.in_use == 0) entries.erase(it);
  }
  void set_state(Message& m, int state) {
    if (m.state == state) return;
    if (m.entry >= 0) {
      entries[m.entry].refs[m.state] -= 1;
      entries[m.entry].refs[state] += 1;
      retier(m.entry);
    }
    m.state = state;
  }

  // ---- pages
  void release(int64_t id, kvt_mgr_report* rep) {
    Entry& e = entries[id];
    by_tier[e.tier].erase({e.stamp, id});
    for (int32_t p : e.page_ids) free_pages.give(p);
    e.page_ids.clear();
    e.resident = false;
    if (rep) {
      rep->released_entries += 1;
      rep->released_pages += e.pages;
    }
    maybe_erase(id);
  }
  // Algorithm 1 for a newly written-back entry
  void admit(int64_t id, kvt_mgr_report* rep) {
    Entry& r = entries[id];
    if (r.only_temporary) {                 // Temporary KV bypasses reuse storage
      rep->bypassed_entries += 1;
      return;
    }
    int64_t delta = r.pages - (int64_t)free_pages.size();
    auto free_by_tier = [&](int tier, bool newest_first) {
      while (delta > 0 && !by_tier[tier].empty()) {
        const int64_t victim = newest_first ? by_tier[tier].rbegin()->second : by_tier[tier].begin()->second;
        const int64_t freed = entries[victim].pages;
        release(victim, rep);
        delta -= freed;
      }
    };
    free_by_tier(kTierDiscarded, false);
    free_by_tier(kTierSuspended, true);     // MRU inside the Suspended tier
    free_by_tier(kTierActive, false);
    if (r.tier == kTierPinned) free_by_tier(kTierPinned, false);
    if (delta <= 0) {
      for (int64_t i = 0; i < r.pages; ++i) {
        r.page_ids.push_back(free_pages.take_lowest());
      }
      r.resident = true;
      if (listed(r)) by_tier[r.tier].insert({r.stamp, id});
      rep->admitted_entries += 1;
      rep->admitted_pages += r.pages;
    } else {
      rep->rejected_entries += 1;
    }
  }
};

namespace {

Context* find_ctx(kvt_manager* m, int64_t ctx) {
  if (m == nullptr) return nullptr;
  auto it = m->ctxs.find(ctx);
  return it == m->ctxs.end() ? nullptr : &it->second;
}

// versions of messages i.. of c expire; each later message (and i unless
// removed) gets a fresh, not yet materialized version
void expire_from(kvt_manager* m, Context& c, size_t i) {
  for (size_t j = i; j < c.msgs.size(); ++j) {
    Message& msg = c.msgs[j];
    m->set_state(msg, kExpired);               // a changed prefix makes even a pinned version stale
    msg.entry = -1;                            // the old version keeps its Expired reference
    msg.state = c.one_off ? kTemporary : kActive;
  }
}

}  // namespace

extern "C" {

kvt_manager* kvt_mgr_create(int64_t num_pages) {
  if (num_pages < 0 || num_pages > INT32_MAX) return nullptr;
  kvt_manager* m = new (std::nothrow) kvt_manager;
  if (m == nullptr) return nullptr;
  m->num_pages = num_pages;
  m->free_pages.reset(num_pages);
  return m;
}

void kvt_mgr_destroy(kvt_manager* m) { delete m; }

int64_t kvt_mgr_free_pages(const kvt_manager* m) { return m ? (int64_t)m->free_pages.size() : -1; }

int64_t kvt_mgr_live_entries(const kvt_manager* m) { return m ? (int64_t)m->entries.size() : -1; }

kvt_status kvt_mgr_spawn(kvt_manager* m, int64_t ctx) {
  if (m != nullptr) ++m->event;
  if (m == nullptr || m->ctxs.count(ctx)) return KVT_ERR_INVALID_ARG;
  m->ctxs[ctx] = Context{};
  return KVT_OK;
}

kvt_status kvt_mgr_fork(kvt_manager* m, int64_t parent, int64_t child) {
  if (m != nullptr) ++m->event;
  Context* p = find_ctx(m, parent);
  if (p == nullptr || p->terminated || p->phase != kIdle || m->ctxs.count(child)) return KVT_ERR_INVALID_ARG;
  Context c;
  c.msgs = p->msgs;                          // same entries, states copied, evolving apart from here
  for (const Message& msg : c.msgs) m->ref(msg.entry, msg.state, +1);
  m->ctxs[child] = std::move(c);
  return KVT_OK;
}

kvt_status kvt_mgr_append(kvt_manager* m, int64_t ctx, int64_t tokens) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || tokens < 1 || tokens > kMaxTokens) return KVT_ERR_INVALID_ARG;
  Message msg;
  msg.state = c->one_off ? kTemporary : kActive;
  msg.tokens = tokens;
  c->msgs.push_back(msg);
  return KVT_OK;
}

kvt_status kvt_mgr_one_off(kvt_manager* m, int64_t ctx) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || c->phase != kIdle) return KVT_ERR_INVALID_ARG;
  c->one_off = true;
  for (Message& msg : c->msgs)               // a pin keeps its protection
    if (msg.state != kPinned) m->set_state(msg, kTemporary);
  return KVT_OK;
}

kvt_status kvt_mgr_pin(kvt_manager* m, int64_t ctx, int64_t msg_index) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || msg_index < 0 || msg_index >= (int64_t)c->msgs.size())
    return KVT_ERR_INVALID_ARG;
  Message& msg = c->msgs[msg_index];
  if (msg.state == kTemporary) return KVT_ERR_INVALID_ARG;
  m->set_state(msg, kPinned);
  return KVT_OK;
}

kvt_status kvt_mgr_unpin(kvt_manager* m, int64_t ctx, int64_t msg_index) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || msg_index < 0 || msg_index >= (int64_t)c->msgs.size()) return KVT_ERR_INVALID_ARG;
  Message& msg = c->msgs[msg_index];
  if (msg.state != kPinned) return KVT_ERR_INVALID_ARG;
  m->set_state(msg, c->terminated ? kExpired : c->one_off ? kTemporary : c->phase != kIdle ? kActive : kSuspended);
  return KVT_OK;
}

kvt_status kvt_mgr_replace(kvt_manager* m, int64_t ctx, int64_t msg_index, int64_t tokens) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || c->phase != kIdle || tokens < 1 || tokens > kMaxTokens || msg_index < 0 ||
      msg_index >= (int64_t)c->msgs.size())
    return KVT_ERR_INVALID_ARG;
  expire_from(m, *c, (size_t)msg_index);
  c->msgs[msg_index].tokens = tokens;
  return KVT_OK;
}

kvt_status kvt_mgr_remove(kvt_manager* m, int64_t ctx, int64_t msg_index) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || c->phase != kIdle || msg_index < 0 || msg_index >= (int64_t)c->msgs.size())
    return KVT_ERR_INVALID_ARG;
  expire_from(m, *c, (size_t)msg_index);
  c->msgs.erase(c->msgs.begin() + msg_index);
  return KVT_OK;
}

kvt_status kvt_mgr_terminate(kvt_manager* m, int64_t ctx) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || c->phase != kIdle) return KVT_ERR_INVALID_ARG;
  c->terminated = true;
  for (Message& msg : c->msgs)
    if (msg.state == kActive || msg.state == kSuspended) m->set_state(msg, kExpired);
  return KVT_OK;
}

kvt_status kvt_mgr_begin_request(kvt_manager* m, int64_t ctx) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->terminated || c->phase != kIdle) return KVT_ERR_INVALID_ARG;
  c->phase = kIssued;
  for (Message& msg : c->msgs)               // participating again
    if (msg.state == kSuspended) m->set_state(msg, kActive);
  return KVT_OK;
}

kvt_status kvt_mgr_start_prefill(kvt_manager* m, int64_t ctx, kvt_mgr_report* rep) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->phase != kIssued || rep == nullptr) return KVT_ERR_INVALID_ARG;
  *rep = kvt_mgr_report{};
  c->phase = kPrefilling;
  bool lost = false;       // once a message misses, every later one is recomputed too
  for (Message& msg : c->msgs) {
    if (msg.entry >= 0 && (lost || !m->entries[msg.entry].resident)) {
      // evicted KV: the version is gone; a fresh one will be recomputed
      m->ref(msg.entry, msg.state, -1);
      msg.entry = -1;
    }
    if (msg.entry < 0) {
      lost = true;
      rep->miss_tokens += msg.tokens;
    } else {
      rep->hit_tokens += msg.tokens;
      m->hold(msg.entry);
      c->using_entries.push_back(msg.entry);
    }
  }
  return KVT_OK;
}

kvt_status kvt_mgr_prefill_done(kvt_manager* m, int64_t ctx, kvt_mgr_report* rep) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->phase != kPrefilling || rep == nullptr) return KVT_ERR_INVALID_ARG;
  *rep = kvt_mgr_report{};
  c->phase = kDecoding;
  std::vector<int64_t> fresh;
  for (Message& msg : c->msgs) {
    if (msg.entry >= 0) continue;
    const int64_t id = m->next_entry++;
    Entry& e = m->entries[id];
    e.pages = (msg.tokens + 15) / 16;
    e.stamp = m->event;
    msg.entry = id;
    m->ref(id, msg.state, +1);
    m->hold(id);                             // the running request decodes over it
    c->using_entries.push_back(id);
    fresh.push_back(id);
  }
  for (Message& msg : c->msgs)               // prefill complete: Active -> Suspended
    if (msg.state == kActive) m->set_state(msg, kSuspended);
  for (int64_t id : fresh) m->admit(id, rep);   // write-back in message order
  return KVT_OK;
}

kvt_status kvt_mgr_end_request(kvt_manager* m, int64_t ctx) {
  if (m != nullptr) ++m->event;
  Context* c = find_ctx(m, ctx);
  if (c == nullptr || c->phase == kIdle) return KVT_ERR_INVALID_ARG;
  for (int64_t id : c->using_entries) m->unhold(id);
  c->using_entries.clear();
  c->phase = kIdle;
  for (Message& msg : c->msgs)               // ordinary messages idle again
    if (msg.state == kActive) m->set_state(msg, kSuspended);
  return KVT_OK;
}

int64_t kvt_mgr_replay(kvt_manager* m, const int64_t* events, int64_t n, kvt_mgr_report* totals) {
  if (m == nullptr || n < 0 || (n > 0 && events == nullptr)) return -1;
  if (totals != nullptr) *totals = kvt_mgr_report{};
  int64_t ok = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t* e = events + 4 * i;
    const int64_t a = e[1], b = e[2], c = e[3];
    kvt_mgr_report rep{};
    bool with_report = false;
    kvt_status st = KVT_ERR_INVALID_ARG;
    switch (e[0]) {
      case KVT_MGR_OP_SPAWN: st = kvt_mgr_spawn(m, a); break;
      case KVT_MGR_OP_FORK: st = kvt_mgr_fork(m, a, b); break;
      case KVT_MGR_OP_APPEND: st = kvt_mgr_append(m, a, b); break;
      case KVT_MGR_OP_ONE_OFF: st = kvt_mgr_one_off(m, a); break;
      case KVT_MGR_OP_PIN: st = kvt_mgr_pin(m, a, b); break;
      case KVT_MGR_OP_UNPIN: st = kvt_mgr_unpin(m, a, b); break;
      case KVT_MGR_OP_REPLACE: st = kvt_mgr_replace(m, a, b, c); break;
      case KVT_MGR_OP_REMOVE: st = kvt_mgr_remove(m, a, b); break;
      case KVT_MGR_OP_TERMINATE: st = kvt_mgr_terminate(m, a); break;
      case KVT_MGR_OP_BEGIN_REQUEST: st = kvt_mgr_begin_request(m, a); break;
      case KVT_MGR_OP_START_PREFILL: st = kvt_mgr_start_prefill(m, a, &rep); with_report = true; break;
      case KVT_MGR_OP_PREFILL_DONE: st = kvt_mgr_prefill_done(m, a, &rep); with_report = true; break;
      case KVT_MGR_OP_END_REQUEST: st = kvt_mgr_end_request(m, a); break;
      default: break;
    }
    if (st != KVT_OK) continue;
    ++ok;
    if (with_report && totals != nullptr) {
      totals->admitted_entries += rep.admitted_entries;
      totals->admitted_pages += rep.admitted_pages;
      totals->bypassed_entries += rep.bypassed_entries;
      totals->rejected_entries += rep.rejected_entries;
      totals->released_entries += rep.released_entries;
      totals->released_pages += rep.released_pages;
      totals->hit_tokens += rep.hit_tokens;
      totals->miss_tokens += rep.miss_tokens;
    }
  }
  return ok;
}

int32_t kvt_mgr_message_state(const kvt_manager* m, int64_t ctx, int64_t msg_index) {
  Context* c = find_ctx(const_cast<kvt_manager*>(m), ctx);
  if (c == nullptr || msg_index < 0 || msg_index >= (int64_t)c->msgs.size()) return -1;
  return c->msgs[msg_index].state;
}

int64_t kvt_mgr_message_pages(const kvt_manager* m, int64_t ctx, int64_t msg_index, int32_t* pages, int64_t cap) {
  Context* c = find_ctx(const_cast<kvt_manager*>(m), ctx);
  if (c == nullptr || msg_index < 0 || msg_index >= (int64_t)c->msgs.size()) return -1;
  const Message& msg = c->msgs[msg_index];
  if (msg.entry < 0) return -1;
  const Entry& e = m->entries.at(msg.entry);
  if (!e.resident) return -1;
  const int64_t n = (int64_t)e.page_ids.size();
  if (pages != nullptr)
    for (int64_t i = 0; i < n && i < cap; ++i) pages[i] = e.page_ids[i];
  return n;
}

int32_t kvt_mgr_entry_tier(const kvt_manager* m, int64_t ctx, int64_t msg_index) {
  Context* c = find_ctx(const_cast<kvt_manager*>(m), ctx);
  if (c == nullptr || msg_index < 0 || msg_index >= (int64_t)c->msgs.size()) return -1;
  const Message& msg = c->msgs[msg_index];
  if (msg.entry < 0) return -1;
  return m->entries.at(msg.entry).tier;
}

}  // extern "C"
