// Test driver: replays block-manager calls read from stdin through the C API
// and prints each call's status and report, one line per call.  Built by
// tests/test_manager.py with the host compiler and sanitizers.
//
// Input lines: "<op> <args...>" with op one of spawn fork append one_off pin
// unpin replace remove terminate begin_request start_prefill prefill_done
// end_request; the first line is "pages <n>".
#include <cstdio>
#include <cstring>
#include <iostream>
#include <sstream>
#include <string>

#include "kvt.h"

int main() {
  std::string line;
  kvt_manager* m = nullptr;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    std::string op;
    long long a = 0, b = 0, c = 0;
    in >> op >> a >> b >> c;
    if (op == "pages") {
      kvt_mgr_destroy(m);
      m = kvt_mgr_create(a);
      std::printf("%s\n", m ? "ok" : "null");
      continue;
    }
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
  kvt_mgr_destroy(m);
  return 0;
}
