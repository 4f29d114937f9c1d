// Test driver: replays block-manager calls read from stdin through the C API
// and prints each call's status and report, one line per call; at the end of
// each stream it replays the same events through kvt_mgr_replay on a fresh
// manager and prints the summed report.  Built by tests/test_manager.py with
// the host compiler and sanitizers.
//
// Input lines: "<op> <args...>" with op one of spawn fork append one_off pin
// unpin replace remove terminate begin_request start_prefill prefill_done
// end_request; the first line is "pages <n>".
#include <cstdio>
#include <cstring>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "kvt.h"

// the events since the last "pages" line, as kvt_mgr_replay takes them
static std::vector<int64_t> g_events;
static long long g_pages = 0;

// replays the collected events on a fresh manager and prints the summary
static void replay_summary() {
  if (g_events.empty()) return;
  kvt_manager* r = kvt_mgr_create(g_pages);
  kvt_mgr_report tot;
  const int64_t ok = kvt_mgr_replay(r, g_events.data(), (int64_t)g_events.size() / 4, &tot);
  std::printf("replay ok=%lld hit=%lld miss=%lld admitted=%lld released=%lld free=%lld\n", (long long)ok,
              (long long)tot.hit_tokens, (long long)tot.miss_tokens, (long long)tot.admitted_pages,
              (long long)tot.released_pages, (long long)kvt_mgr_free_pages(r));
  kvt_mgr_destroy(r);
  g_events.clear();
}

int main() {
  static const char* kOps[] = {"spawn", "fork", "append", "one_off", "pin", "unpin", "replace", "remove",
                               "terminate", "begin_request", "start_prefill", "prefill_done", "end_request"};
  std::string line;
  kvt_manager* m = nullptr;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    std::string op;
    long long a = 0, b = 0, c = 0;
    in >> op >> a >> b >> c;
    if (op == "pages") {
      replay_summary();
      kvt_mgr_destroy(m);
      m = kvt_mgr_create(a);
      g_pages = a;
      std::printf("%s\n", m ? "ok" : "null");
      continue;
    }
    for (int k = 0; k < 13; ++k)
      if (op == kOps[k]) g_events.insert(g_events.end(), {k, a, b, c});
    kvt_mgr_report rep;
    std::memset(&rep, 0xff, sizeof(rep));
    kvt_status st = KVT_ERR_INVALID_ARG;
    bool with_report = false;
    if (op == "spawn") st = kvt_mgr_spawn(m, a);
    else if (op == "fork") st = kvt_mgr_fork(m, a, b);
    else if (op == "append") st = kvt_mgr_append(m, a, b);
    else if (op == "one_off") st = kvt_mgr_one_off(m, a);
    else if (op == "pin") st = kvt_mgr_pin(m, a, b);
    else if (op == "unpin") st = kvt_mgr_unpin(m, a, b);
    else if (op == "replace") st = kvt_mgr_replace(m, a, b, c);
    else if (op == "remove") st = kvt_mgr_remove(m, a, b);
    else if (op == "terminate") st = kvt_mgr_terminate(m, a);
    else if (op == "begin_request") st = kvt_mgr_begin_request(m, a);
    else if (op == "end_request") st = kvt_mgr_end_request(m, a);
    else if (op == "start_prefill") { st = kvt_mgr_start_prefill(m, a, &rep); with_report = true; }
    else if (op == "prefill_done") { st = kvt_mgr_prefill_done(m, a, &rep); with_report = true; }
    else { std::fprintf(stderr, "unknown op %s\n", op.c_str()); return 2; }
    std::printf("%d", (int)st);
    if (with_report && st == KVT_OK)
      std::printf(" %lld %lld %lld %lld %lld %lld %lld %lld", (long long)rep.admitted_entries,
                  (long long)rep.admitted_pages, (long long)rep.bypassed_entries, (long long)rep.rejected_entries,
                  (long long)rep.released_entries, (long long)rep.released_pages, (long long)rep.hit_tokens,
                  (long long)rep.miss_tokens);
    std::printf(" free=%lld\n", (long long)kvt_mgr_free_pages(m));
  }
  replay_summary();
  kvt_mgr_destroy(m);
  return 0;
}
