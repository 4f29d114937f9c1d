// C-ABI entry points: argument validation, work planning and launches.
//
// Every check runs on the host before the first HIP call, so a bad call
// returns an error with nothing enqueued.  Planning is host arithmetic only:
// sequences are ordered longest first, the (row tile, key split) units of
// each sequence are numbered longest first, and the kv-head index varies
// fastest over workgroup ids -- workgroups are dispatched round-robin over the
// 8 XCDs, so with 8 (or a multiple/divisor of 8) kv-heads every workgroup of
// one kv-head runs on the same XCD and its K/V stream is shared in that L2.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <functional>
#include <numeric>
#include <queue>
#include <unordered_set>
#include <vector>

#include "kvt.h"
#include "kvt_internal.h"

namespace {

thread_local int g_last_hip_error = 0;

kvt_status device_error(hipError_t e) {
  g_last_hip_error = (int)e;
  return KVT_ERR_DEVICE;
}

int elem_bytes(int32_t dtype) { return dtype == KVT_DTYPE_BF16 ? 2 : 4; }

// Number of compute units of the current device, queried once per device
// (concurrent first calls may both query; they store the same value).
int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) { (void)hipGetLastError(); return 256; }
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      n = 256;
    }
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// The kernels move 16-byte pieces of every token row, page and workspace.
bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

kvt_status check_pool(const kvt_pool* pool) {
  if (pool == nullptr || pool->k == nullptr || pool->v == nullptr) return KVT_ERR_INVALID_ARG;
  if (!aligned16(pool->k) || !aligned16(pool->v)) return KVT_ERR_INVALID_ARG;
  if (pool->num_blocks < 1 || pool->num_kv_heads < 1) return KVT_ERR_INVALID_ARG;
  if (pool->head_dim != 64 && pool->head_dim != 128) return KVT_ERR_UNSUPPORTED;
  if (pool->dtype != KVT_DTYPE_BF16 && pool->dtype != KVT_DTYPE_F32) return KVT_ERR_UNSUPPORTED;
  return KVT_OK;
}

// Validates lengths and table width; fills the total token count.
kvt_status check_seqs(const kvt_seqs* seqs, int64_t* total_tokens) {
  if (seqs == nullptr || seqs->num_seqs < 1) return KVT_ERR_INVALID_ARG;
  if (seqs->prefix_len == nullptr || seqs->suffix_len == nullptr || seqs->block_table == nullptr)
    return KVT_ERR_INVALID_ARG;
  if (seqs->max_blocks < 1) return KVT_ERR_INVALID_ARG;
  int64_t T = 0;
  for (int b = 0; b < seqs->num_seqs; ++b) {
    const int64_t P = seqs->prefix_len[b], S = seqs->suffix_len[b];
    if (P < 0 || S < 1) return KVT_ERR_INVALID_ARG;
    const int64_t L = P + S;
    if (L > INT32_MAX / 2) return KVT_ERR_INVALID_ARG;
    if ((L + kvt::kBlock - 1) / kvt::kBlock > seqs->max_blocks) return KVT_ERR_INVALID_ARG;
    T += S;
  }
  if (T > INT32_MAX / 2) return KVT_ERR_INVALID_ARG;
  *total_tokens = T;
  return KVT_OK;
}

// Query heads: a positive multiple of the kv-heads, and T * num_q_heads
// packed query rows must fit the kernels' 32-bit row indices.
bool heads_ok(const kvt_pool* pool, int32_t num_q_heads, int64_t T) {
  if (num_q_heads < 1 || num_q_heads % pool->num_kv_heads != 0) return false;
  return T * num_q_heads <= INT32_MAX;
}

// Checked mode: every used block id is inside the pool.
kvt_status check_table_ids(const kvt_pool* pool, const kvt_seqs* seqs) {
  if (seqs->block_table_host == nullptr) return KVT_OK;
  for (int b = 0; b < seqs->num_seqs; ++b) {
    const int64_t L = (int64_t)seqs->prefix_len[b] + seqs->suffix_len[b];
    const int64_t nblk = (L + kvt::kBlock - 1) / kvt::kBlock;
    const int32_t* row = seqs->block_table_host + (int64_t)b * seqs->max_blocks;
    for (int64_t i = 0; i < nblk; ++i)
      if (row[i] < 0 || (int64_t)row[i] >= pool->num_blocks) return KVT_ERR_OUT_OF_RANGE;
  }
  return KVT_OK;
}

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + bn && y < x + an;
}

// Workspace of nsplit partial results per packed row: the unnormalised
// outputs in fp32 (256-byte aligned block), then (m, l) in fp32.
size_t part_o_bytes(const kvt_pool* pool, int nsplit, int64_t rows) {
  return (((size_t)nsplit * rows * pool->head_dim * sizeof(float) + 255) / 256) * 256;
}
size_t part_bytes(const kvt_pool* pool, int nsplit, int64_t rows) {
  return part_o_bytes(pool, nsplit, rows) + (size_t)nsplit * rows * 2 * sizeof(float);
}

struct ExtendPlan {
  int nsplit = 1;
  int nsplit_shared = 0;    // cascade only: key splits of the shared part
  bool use_shared = true;   // cascade only: false = run the plain extend plan
  std::vector<int> order;   // sequences, longest key range first
  size_t ws_bytes = 0;      // workspace needed for nsplit > 1
};

int row_tiles(int32_t suffix, int group) {
  const int64_t rows = (int64_t)suffix * group;
  return (int)((rows + kvt::kExtTileRows - 1) / kvt::kExtTileRows);
}

// Cost of the combine launch that merges split partials, in us.
constexpr double kMergeLaunchUs = 4.0;
// Fixed cost of one workgroup, in key tiles: its prologue (kernel arguments,
// block-table entries and the first tile's gather, about 3.3 us) and its
// epilogue.
constexpr double kUnitTiles = 2.0;

// Finish time, in key tiles, of one extend launch: list scheduling of its
// units in launch order onto the CUs (each unit to the CU that frees first,
// as workgroups are dispatched): shared_jobs units of len_s tiles first
// (a cascade's shared part; none for a plain extend), then each sequence's
// units (jobs_p[b] row tiles of ceil(kt_p[b] / ns_p) tiles, ns_p splits
// each, of which one in `share` falls to the CUs modelled); every unit also
// pays kUnitTiles.  Callers model one kv-head's units on its share of the
// CUs (the units of the kv-heads alternate) or one XCD's (workgroups go to
// the XCDs in turn).
double list_finish(int64_t shared_jobs, double len_s, const std::vector<int64_t>& jobs_p,
                   const std::vector<int64_t>& kt_p, int ns_p, int cus, int share = 1) {
  const int64_t rounds = shared_jobs / cus, rest = shared_jobs % cus;
  std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
  for (int c = 0; c < cus; ++c) free_at.push((double)(c < rest ? rounds + 1 : rounds) * (len_s + kUnitTiles));
  double span = (double)(rest > 0 ? rounds + 1 : rounds) * (len_s + kUnitTiles);
  for (size_t b = 0; b < jobs_p.size(); ++b) {
    const double len = std::ceil((double)kt_p[b] / ns_p) + kUnitTiles;
    for (int64_t j = 0; j < (jobs_p[b] * ns_p + share - 1) / share; ++j) {
      const double t = free_at.top() + len;
      free_at.pop();
      free_at.push(t);
      span = std::max(span, t);
    }
  }
  return span;
}

// Split long key ranges only when the row tiles alone cannot fill the chip.
ExtendPlan make_plan(const kvt_pool* pool, const kvt_seqs* seqs, int32_t num_q_heads, int64_t T) {
  ExtendPlan p;
  const int B = seqs->num_seqs;
  const int G = num_q_heads / pool->num_kv_heads;
  p.order.resize(B);
  std::iota(p.order.begin(), p.order.end(), 0);
  std::stable_sort(p.order.begin(), p.order.end(), [&](int x, int y) {
    return (int64_t)seqs->prefix_len[x] + seqs->suffix_len[x] > (int64_t)seqs->prefix_len[y] + seqs->suffix_len[y];
  });
  int64_t units = 0;
  int64_t min_keys = INT64_MAX, min_len = INT64_MAX, max_len = 0;
  for (int b = 0; b < B; ++b) {
    units += (int64_t)row_tiles(seqs->suffix_len[b], G) * pool->num_kv_heads;
    min_keys = std::min<int64_t>(min_keys, (int64_t)seqs->prefix_len[b] + 1);
    const int64_t len = (int64_t)seqs->prefix_len[b] + seqs->suffix_len[b];
    min_len = std::min(min_len, len);
    max_len = std::max(max_len, len);
  }
  const int cus = device_cus();
  // Split the key range when whole rounds of workgroups over the CUs leave
  // many CUs idle: with ns splits a unit's work shrinks to 1/ns and the call
  // takes about ceil(units*ns / cus) / ns unit-times.  Take the smallest ns
  // with the best estimate if it beats no split by at least 10 %; each split
  // keeps at least 16 key tiles (1024 keys) of the shortest sequence.
  const int64_t by_keys = std::max<int64_t>(1, min_keys / (16 * kvt::kExtKeysPerTile));
  const int ns_max = (int)std::min<int64_t>(by_keys, kvt::kMaxSplits);
  auto rounds = [&](int s) { return (double)((units * s + cus - 1) / cus) / s; };
  int ns = 1;
  for (int s = 2; s <= ns_max; ++s)
    if (rounds(s) < rounds(ns) - 1e-9) ns = s;
  if (rounds(ns) > 0.9 * rounds(1)) ns = 1;
  // Ragged batches: the rule above counts units as equal and keeps 1024 keys
  // of the shortest sequence per split, so one short sequence stops the long
  // ones from splitting.  When the longest key range is more than twice the
  // shortest and the row tiles fit a few rounds of the CUs, list-schedule
  // the launch for 1, 2, 4, 8 and 16 splits (one XCD's eighth of the units
  // on its CUs, each unit's length from its sequence's key tiles) and take
  // the best finish plus partial cost if it beats the rule's choice by more
  // than a fifth.
  constexpr int kXcds = 8;
  const int xcd_cus = std::max(1, cus / kXcds);
  if (max_len > 2 * min_len && units <= 4 * (int64_t)cus) {
    const int64_t rows = T * num_q_heads;
    std::vector<int64_t> jobs(B), kt(B);
    for (int i = 0; i < B; ++i) {
      const int b = p.order[i];
      jobs[i] = (int64_t)row_tiles(seqs->suffix_len[b], G) * pool->num_kv_heads;
      kt[i] = ((int64_t)seqs->prefix_len[b] + seqs->suffix_len[b] + kvt::kExtKeysPerTile - 1) / kvt::kExtKeysPerTile;
    }
    auto cost = [&](int s) {
      double t = list_finish(0, 0.0, jobs, kt, s, xcd_cus, kXcds);
      if (s > 1) t += (2.0 * (double)part_bytes(pool, s, rows) / 5.0e6 + kMergeLaunchUs) / 1.8;
      return t;
    };
    const double rule_cost = cost(ns);
    int best = ns;
    double best_cost = rule_cost;
    for (int s = 1; s <= kvt::kMaxSplits; s *= 2) {
      const double c = cost(s);
      if (c < best_cost - 1e-9) best = s, best_cost = c;
    }
    if (best_cost < 0.8 * rule_cost) ns = best;
  }
  p.nsplit = ns;
  if (ns > 1) p.ws_bytes = part_bytes(pool, ns, T * num_q_heads);
  return p;
}

// Decode: one unit per (sequence, key split) and kv-head.  Splits are added
// while the workgroups cannot cover the CUs twice over, keeping at least 1024
// keys of the shortest sequence per split (each of the 4 waves then streams
// at least 8 tiles of 32 keys).
ExtendPlan make_decode_plan(const kvt_pool* pool, const kvt_seqs* seqs, int32_t num_q_heads) {
  ExtendPlan p;
  const int B = seqs->num_seqs;
  p.order.resize(B);
  std::iota(p.order.begin(), p.order.end(), 0);
  std::stable_sort(p.order.begin(), p.order.end(),
                   [&](int x, int y) { return seqs->prefix_len[x] > seqs->prefix_len[y]; });
  int64_t min_keys = INT64_MAX;
  for (int b = 0; b < B; ++b) min_keys = std::min<int64_t>(min_keys, (int64_t)seqs->prefix_len[b] + 1);
  const int64_t units = (int64_t)B * pool->num_kv_heads;
  const int64_t want = (2 * (int64_t)device_cus() + units - 1) / units;
  const int64_t by_keys = std::max<int64_t>(1, min_keys / 1024);
  p.nsplit = (int)std::max<int64_t>(1, std::min<int64_t>({want, by_keys, (int64_t)kvt::kMaxSplits}));
  if (p.nsplit > 1) p.ws_bytes = part_bytes(pool, p.nsplit, (int64_t)B * num_q_heads);
  return p;
}

// A shared prefix: a positive multiple of 16 no longer than any sequence's
// prefix; in checked mode every table row must list the same pages for it.
kvt_status check_shared(const kvt_seqs* seqs, int32_t shared_len) {
  if (shared_len < kvt::kBlock || shared_len % kvt::kBlock != 0) return KVT_ERR_INVALID_ARG;
  for (int b = 0; b < seqs->num_seqs; ++b)
    if (seqs->prefix_len[b] < shared_len) return KVT_ERR_INVALID_ARG;
  if (seqs->block_table_host != nullptr) {
    const int32_t* row0 = seqs->block_table_host;
    for (int b = 1; b < seqs->num_seqs; ++b)
      if (std::memcmp(row0, seqs->block_table_host + (int64_t)b * seqs->max_blocks,
                      sizeof(int32_t) * (shared_len / kvt::kBlock)) != 0)
        return KVT_ERR_INVALID_ARG;
  }
  return KVT_OK;
}

// Estimated time of one extend launch in units of one 64-key tile of one
// 256-row workgroup: the larger of the work spread over the CUs and the
// longest unit's share of its key splits, plus the split partials written
// and read back when split.  kt[b]: key tiles of sequence b, units[b]: its
// row tiles x kv-heads.
double launch_estimate(const std::vector<int64_t>& units, const std::vector<int64_t>& kt, int nsplit,
                       int64_t rows, const kvt_pool* pool, int cus) {
  // one tile of one workgroup takes about 1.8 us at full load; the partials
  // move at about 5 bytes per ns (written once, read once by the combine),
  // and the combine launch itself costs about 4 us
  constexpr double kTileUs = 1.8, kBytesPerUs = 5.0e6;
  double work = 0, longest = 0;
  for (size_t b = 0; b < units.size(); ++b) {
    work += (double)units[b] * kt[b];
    longest = std::max(longest, (double)kt[b]);
  }
  double t = std::max(work / cus, longest / nsplit) + kUnitTiles;
  if (nsplit > 1) t += (2.0 * (double)part_bytes(pool, nsplit, rows) / kBytesPerUs + kMergeLaunchUs) / kTileUs;
  return t;
}

// Cascade: the split plans of the shared part (one virtual sequence of all T
// new tokens over the shared keys, all visible) and of the private parts
// (prefix lengths less the shared prefix); the workspace holds one partial
// per split of either part.  The shared pass reads the shared keys once per
// packed row tile of the whole batch instead of once per sequence's row
// tiles, but every row then goes through partials and a merge; when the
// estimate says the plain extend is faster (long suffixes, where row tiles
// pack well anyway), the plan is the plain extend's (use_shared = false).
ExtendPlan cascade_plan(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len, int32_t num_q_heads,
                        int64_t T, int32_t mode = KVT_CASCADE_AUTO) {
  const int B = seqs->num_seqs, G = num_q_heads / pool->num_kv_heads, H = pool->num_kv_heads;
  const int KT = kvt::kExtKeysPerTile;
  std::vector<int32_t> priv(B);
  for (int b = 0; b < B; ++b) priv[b] = seqs->prefix_len[b] - shared_len;
  kvt_seqs ps = *seqs;
  ps.prefix_len = priv.data();
  ExtendPlan p = make_plan(pool, &ps, num_q_heads, T);
  const int32_t shared_prefix = shared_len - 1, all_tokens = (int32_t)T;
  kvt_seqs ss = *seqs;
  ss.num_seqs = 1;
  ss.prefix_len = &shared_prefix;
  ss.suffix_len = &all_tokens;
  p.nsplit_shared = make_plan(pool, &ss, num_q_heads, T).nsplit;

  const int cus = device_cus();
  const int64_t rows = T * num_q_heads;
  std::vector<int64_t> units(B), kt_full(B), kt_priv(B), jobs_p(B), kt_p(B);
  int64_t head_jobs = 0;   // private units of one kv-head
  for (int b = 0; b < B; ++b) {
    units[b] = (int64_t)row_tiles(seqs->suffix_len[b], G) * H;
    kt_full[b] = ((int64_t)seqs->prefix_len[b] + seqs->suffix_len[b] + KT - 1) / KT;
    kt_priv[b] = ((int64_t)priv[b] + seqs->suffix_len[b] + KT - 1) / KT;
    head_jobs += row_tiles(seqs->suffix_len[b], G);
  }
  for (int i = 0; i < B; ++i) {   // launch order, longest first; one kv-head's units
    jobs_p[i] = row_tiles(seqs->suffix_len[p.order[i]], G);
    kt_p[i] = kt_priv[p.order[i]];
  }
  const int head_cus = std::max(1, cus / H);
  const int64_t shared_jobs = (int64_t)row_tiles((int32_t)T, G) * H * p.nsplit_shared;
  const double kt_shared = (double)((shared_len + KT - 1) / KT);
  const double len_s = std::ceil(kt_shared / p.nsplit_shared);
  // In one launch the private units can fill what the shared part leaves
  // idle: when one kv-head's private units fit one round of its CUs, their
  // split count is the one (trying 1, 2, 4, 8, 16 until the estimate rises)
  // with the earliest list-scheduled finish plus partial cost.
  auto partial_cost = [&](int ns_p) {
    return (2.0 * (double)part_bytes(pool, p.nsplit_shared + ns_p, rows) / 5.0e6 + kMergeLaunchUs) / 1.8;
  };
  double t_shared = 0;
  if (head_jobs <= head_cus) {
    const int64_t head_shared = shared_jobs / H;
    int best = 1;
    double best_t = list_finish(head_shared, len_s, jobs_p, kt_p, 1, head_cus) + partial_cost(1);
    for (int ns = 2; ns <= kvt::kMaxSplits; ns *= 2) {
      const double t = list_finish(head_shared, len_s, jobs_p, kt_p, ns, head_cus) + partial_cost(ns);
      if (t >= best_t - 1e-9) break;
      best = ns, best_t = t;
    }
    p.nsplit = best;
    t_shared = best_t;
  } else {
    // many private units: the work of both parts spread over the CUs, or
    // the longest unit of either
    double work = (double)shared_jobs * len_s, longest = len_s;
    for (int b = 0; b < B; ++b) {
      work += (double)units[b] * kt_priv[b];
      longest = std::max(longest, (double)kt_priv[b] / p.nsplit);
    }
    t_shared = std::max(work / cus, longest) + kUnitTiles + partial_cost(p.nsplit);
  }
  p.ws_bytes = part_bytes(pool, p.nsplit_shared + p.nsplit, rows);
  if (mode == KVT_CASCADE_SHARED_PASS) return p;

  const ExtendPlan plain = make_plan(pool, seqs, num_q_heads, T);
  if (mode == KVT_CASCADE_PLAIN) {
    ExtendPlan q = plain;
    q.use_shared = false;
    return q;
  }
  const double t_plain = launch_estimate(units, kt_full, plain.nsplit, rows, pool, cus);
  if (t_shared < t_plain) return p;
  ExtendPlan q = plain;
  q.use_shared = false;
  return q;
}

bool mode_ok(int32_t mode) {
  return mode == KVT_CASCADE_AUTO || mode == KVT_CASCADE_SHARED_PASS || mode == KVT_CASCADE_PLAIN;
}

// out must not overlap q or a pool; lse must not overlap out.
kvt_status check_outputs(const kvt_pool* pool, const void* q, int32_t num_q_heads, const void* out,
                         const float* lse, int64_t T) {
  if (!aligned16(q) || !aligned16(out) || ((uintptr_t)lse & 3) != 0) return KVT_ERR_INVALID_ARG;
  const size_t es = elem_bytes(pool->dtype);
  const size_t tok_bytes = (size_t)T * num_q_heads * pool->head_dim * es;
  const size_t pool_bytes = (size_t)pool->num_blocks * pool->num_kv_heads * kvt::kBlock * pool->head_dim * es;
  if (overlaps(out, tok_bytes, q, tok_bytes) || overlaps(out, tok_bytes, pool->k, pool_bytes) ||
      overlaps(out, tok_bytes, pool->v, pool_bytes))
    return KVT_ERR_INVALID_ARG;
  if (lse != nullptr && overlaps(lse, (size_t)T * num_q_heads * sizeof(float), out, tok_bytes))
    return KVT_ERR_INVALID_ARG;
  return KVT_OK;
}

// Launch arguments common to extend and decode.
kvt::ExtendArgs base_args(const kvt_pool* pool, const kvt_seqs* seqs, const void* q, int32_t num_q_heads,
                          float scale, void* out, float* lse, int64_t T, const ExtendPlan& plan, void* workspace) {
  kvt::ExtendArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q;
  a.k_pool = pool->k;
  a.v_pool = pool->v;
  a.out = out;
  a.lse = lse;
  a.block_table = seqs->block_table;
  a.num_blocks = pool->num_blocks;
  a.max_blocks = seqs->max_blocks;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = pool->num_kv_heads;
  a.group = num_q_heads / pool->num_kv_heads;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.kbeg = 0;
  a.kend = INT32_MAX;
  a.direct = plan.nsplit == 1 ? 1 : 0;
  a.part_base = 0;
  a.nsplit = plan.nsplit;
  a.total_rows = (int32_t)T;
  a.second = INT32_MAX;   // one group of sequences
  a.kbeg2 = 0;
  a.kend2 = INT32_MAX;
  a.nsplit2 = 1;
  a.part_base2 = 0;
  if (plan.nsplit > 1) {
    a.part_o = reinterpret_cast<float*>(workspace);
    a.part_ml = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                         part_o_bytes(pool, plan.nsplit, T * num_q_heads));
  }
  return a;
}

// Merge of the per-split partial results into out (and lse).
kvt_status combine(const kvt::ExtendArgs& a, const kvt_pool* pool, void* out, float* lse, int64_t T,
                   int32_t num_q_heads, int nsplit, hipStream_t s) {
  kvt::CombineArgs c;
  c.part_o = a.part_o;
  c.part_ml = a.part_ml;
  c.out = out;
  c.lse = lse;
  c.rows = T * num_q_heads;
  c.nsplit = nsplit;
  const hipError_t e = kvt::launch_combine(c, pool->dtype, pool->head_dim, s);
  return e == hipSuccess ? KVT_OK : device_error(e);
}

// The argument checks of kvt_extend_attention (and its no-alloc variant);
// fills the total token count.
kvt_status check_extend(const kvt_pool* pool, const kvt_seqs* seqs, const void* q, int32_t num_q_heads, float scale,
                        const void* out, const float* lse, int64_t* T) {
  kvt_status st = check_pool(pool);
  if (st != KVT_OK) return st;
  if ((st = check_seqs(seqs, T)) != KVT_OK) return st;
  if (q == nullptr || out == nullptr) return KVT_ERR_INVALID_ARG;
  if (!heads_ok(pool, num_q_heads, *T)) return KVT_ERR_INVALID_ARG;
  if (!(scale > 0.f) || !std::isfinite(scale)) return KVT_ERR_INVALID_ARG;
  if ((st = check_table_ids(pool, seqs)) != KVT_OK) return st;
  return check_outputs(pool, q, num_q_heads, out, lse, *T);
}

// Launches of one extend call under `plan` (partials in `workspace` when split).
kvt_status launch_extend_plan(const kvt_pool* pool, const kvt_seqs* seqs, const void* q, int32_t num_q_heads,
                              float scale, void* out, float* lse, int64_t T, const ExtendPlan& plan,
                              void* workspace, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int G = num_q_heads / pool->num_kv_heads;
  std::vector<int32_t> row_off(seqs->num_seqs + 1, 0);
  for (int b = 0; b < seqs->num_seqs; ++b) row_off[b + 1] = row_off[b] + seqs->suffix_len[b];

  kvt::ExtendArgs a = base_args(pool, seqs, q, num_q_heads, scale, out, lse, T, plan, workspace);
  for (size_t c0 = 0; c0 < plan.order.size(); c0 += kvt::kSeqsPerLaunch) {
    const int n = (int)std::min<size_t>(kvt::kSeqsPerLaunch, plan.order.size() - c0);
    a.nseq = n;
    int32_t units = 0;
    for (int i = 0; i < n; ++i) {
      const int b = plan.order[c0 + i];
      a.seq[i] = kvt::SeqDesc{b, seqs->prefix_len[b], seqs->suffix_len[b], row_off[b]};
      a.unit_begin[i] = units;
      units += row_tiles(seqs->suffix_len[b], G) * plan.nsplit;
    }
    a.unit_begin[n] = units;
    const int64_t grid = (int64_t)units * pool->num_kv_heads;
    if (grid > INT32_MAX) return KVT_ERR_INVALID_ARG;
    const hipError_t e = kvt::launch_extend(a, pool->dtype, pool->head_dim, (int)grid, s);
    if (e != hipSuccess) return device_error(e);
  }
  return plan.nsplit > 1 ? combine(a, pool, out, lse, T, num_q_heads, plan.nsplit, s) : KVT_OK;
}

}  // namespace

extern "C" {

const char* kvt_status_str(kvt_status s) {
  switch (s) {
    case KVT_OK: return "ok";
    case KVT_ERR_INVALID_ARG: return "invalid argument";
    case KVT_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case KVT_ERR_OUT_OF_RANGE: return "block id out of range or duplicate append target";
    case KVT_ERR_WORKSPACE: return "workspace too small";
    case KVT_ERR_DEVICE: return "HIP launch failed";
    case KVT_ERR_SCRATCH_LIMIT: return "split partials exceed the static scratch (KVT_NOALLOC_SCRATCH_BYTES)";
  }
  return "unknown status";
}

int kvt_last_hip_error(void) { return g_last_hip_error; }

kvt_status kvt_append_kv(const kvt_pool* pool, const kvt_seqs* seqs, const void* k_new, const void* v_new,
                         void* stream) {
  kvt_status st = check_pool(pool);
  if (st != KVT_OK) return st;
  int64_t T = 0;
  if ((st = check_seqs(seqs, &T)) != KVT_OK) return st;
  if (k_new == nullptr || v_new == nullptr || !aligned16(k_new) || !aligned16(v_new)) return KVT_ERR_INVALID_ARG;
  if ((st = check_table_ids(pool, seqs)) != KVT_OK) return st;
  const size_t pool_bytes = (size_t)pool->num_blocks * pool->num_kv_heads * kvt::kBlock * pool->head_dim *
                            elem_bytes(pool->dtype);
  const size_t new_bytes = (size_t)T * pool->num_kv_heads * pool->head_dim * elem_bytes(pool->dtype);
  for (const void* src : {k_new, v_new})
    for (const void* dst : {(const void*)pool->k, (const void*)pool->v})
      if (overlaps(src, new_bytes, dst, pool_bytes)) return KVT_ERR_INVALID_ARG;
  if (seqs->block_table_host != nullptr) {
    // two new tokens may not target one (block, slot)
    std::unordered_set<int64_t> seen;
    seen.reserve((size_t)T * 2);
    for (int b = 0; b < seqs->num_seqs; ++b) {
      const int32_t* row = seqs->block_table_host + (int64_t)b * seqs->max_blocks;
      for (int32_t t = 0; t < seqs->suffix_len[b]; ++t) {
        const int64_t pos = (int64_t)seqs->prefix_len[b] + t;
        const int64_t key = (int64_t)row[pos / kvt::kBlock] * kvt::kBlock + pos % kvt::kBlock;
        if (!seen.insert(key).second) return KVT_ERR_OUT_OF_RANGE;
      }
    }
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  kvt::AppendArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_pool = pool->k;
  a.v_pool = pool->v;
  a.block_table = seqs->block_table;
  a.num_blocks = pool->num_blocks;
  a.max_blocks = seqs->max_blocks;
  a.num_kv_heads = pool->num_kv_heads;
  int32_t row = 0;
  for (int b0 = 0; b0 < seqs->num_seqs; b0 += kvt::kSeqsPerLaunch) {
    const int n = std::min(kvt::kSeqsPerLaunch, seqs->num_seqs - b0);
    a.nseq = n;
    a.row_begin = row;
    for (int i = 0; i < n; ++i) {
      const int b = b0 + i;
      a.seq[i] = kvt::SeqDesc{b, seqs->prefix_len[b], seqs->suffix_len[b], row};
      row += seqs->suffix_len[b];
    }
    a.rows = row - a.row_begin;
    const hipError_t e = kvt::launch_append(a, pool->dtype, pool->head_dim, s);
    if (e != hipSuccess) return device_error(e);
  }
  return KVT_OK;
}

size_t kvt_extend_workspace_bytes(const kvt_pool* pool, const kvt_seqs* seqs, int32_t num_q_heads) {
  if (check_pool(pool) != KVT_OK) return 0;
  int64_t T = 0;
  if (check_seqs(seqs, &T) != KVT_OK) return 0;
  if (!heads_ok(pool, num_q_heads, T)) return 0;
  return make_plan(pool, seqs, num_q_heads, T).ws_bytes;
}

kvt_status kvt_extend_attention(const kvt_pool* pool, const kvt_seqs* seqs, const void* q, int32_t num_q_heads,
                                float scale, void* out, float* lse, void* workspace, size_t workspace_bytes,
                                void* stream) {
  int64_t T = 0;
  const kvt_status st = check_extend(pool, seqs, q, num_q_heads, scale, out, lse, &T);
  if (st != KVT_OK) return st;
  ExtendPlan plan = make_plan(pool, seqs, num_q_heads, T);
  if (plan.nsplit > 1) {
    if (workspace == nullptr && workspace_bytes == 0) {
      plan.nsplit = 1;   // no scratch offered: run unsplit
    } else if (workspace == nullptr || workspace_bytes < plan.ws_bytes) {
      return KVT_ERR_WORKSPACE;
    } else if (!aligned16(workspace)) {
      return KVT_ERR_INVALID_ARG;
    }
  }
  return launch_extend_plan(pool, seqs, q, num_q_heads, scale, out, lse, T, plan, workspace, stream);
}

kvt_status kvt_extend_attention_noalloc(const kvt_pool* pool, const kvt_seqs* seqs, const void* q,
                                        int32_t num_q_heads, float scale, void* out, float* lse, void* stream) {
  int64_t T = 0;
  const kvt_status st = check_extend(pool, seqs, q, num_q_heads, scale, out, lse, &T);
  if (st != KVT_OK) return st;
  // the same plan as kvt_extend_attention with a large enough workspace, so
  // both give the same bits; partials go to the static scratch
  const ExtendPlan plan = make_plan(pool, seqs, num_q_heads, T);
  void* ws = nullptr;
  if (plan.nsplit > 1) {
    if (plan.ws_bytes > (size_t)KVT_NOALLOC_SCRATCH_BYTES) return KVT_ERR_SCRATCH_LIMIT;
    const hipError_t e = kvt::noalloc_scratch(&ws);
    if (e != hipSuccess) return device_error(e);
  }
  return launch_extend_plan(pool, seqs, q, num_q_heads, scale, out, lse, T, plan, ws, stream);
}

kvt_status kvt_copy_blocks(const kvt_pool* pool, const int32_t* block_ids, const int32_t* block_ids_host,
                           int64_t num_ids, void* host, int32_t direction, void* stream) {
  kvt_status st = check_pool(pool);
  if (st != KVT_OK) return st;
  if (num_ids < 0 || (num_ids > 0 && (block_ids == nullptr || host == nullptr))) return KVT_ERR_INVALID_ARG;
  if (direction != KVT_COPY_TO_HOST && direction != KVT_COPY_TO_DEVICE) return KVT_ERR_INVALID_ARG;
  if (num_ids == 0) return KVT_OK;
  const int64_t page_bytes = (int64_t)pool->num_kv_heads * kvt::kBlock * pool->head_dim * elem_bytes(pool->dtype);
  if (num_ids > (INT64_MAX / 4) / (2 * page_bytes)) return KVT_ERR_INVALID_ARG;
  if (block_ids_host != nullptr) {
    std::unordered_set<int32_t> seen;
    for (int64_t i = 0; i < num_ids; ++i) {
      const int32_t id = block_ids_host[i];
      if (id < 0 || id >= pool->num_blocks) return KVT_ERR_OUT_OF_RANGE;
      // two host pages landing on one pool page would race
      if (direction == KVT_COPY_TO_DEVICE && !seen.insert(id).second) return KVT_ERR_OUT_OF_RANGE;
    }
  }
  // the host side must be pinned memory the device can address
  hipPointerAttribute_t attr;
  std::memset(&attr, 0, sizeof(attr));
  if (hipPointerGetAttributes(&attr, host) != hipSuccess) {
    (void)hipGetLastError();
    return KVT_ERR_INVALID_ARG;
  }
  if (attr.type != hipMemoryTypeHost) return KVT_ERR_INVALID_ARG;
  void* host_dev = attr.devicePointer != nullptr ? attr.devicePointer : host;

  kvt::CopyArgs a;
  a.k_pool = pool->k;
  a.v_pool = pool->v;
  a.ids = block_ids;
  a.n = num_ids;
  a.host = host_dev;
  a.page_bytes = page_bytes;
  a.num_blocks = pool->num_blocks;
  a.to_host = direction == KVT_COPY_TO_HOST ? 1 : 0;
  const int64_t pieces = num_ids * 2 * page_bytes / 16;
  const int grid = (int)std::min<int64_t>((pieces + 255) / 256, 8192);
  const hipError_t e = kvt::launch_copy_blocks(a, grid, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? KVT_OK : device_error(e);
}

size_t kvt_cascade_workspace_bytes_ex(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                      int32_t mode, int32_t num_q_heads) {
  if (check_pool(pool) != KVT_OK) return 0;
  int64_t T = 0;
  if (check_seqs(seqs, &T) != KVT_OK) return 0;
  if (!heads_ok(pool, num_q_heads, T)) return 0;
  if (check_shared(seqs, shared_len) != KVT_OK || !mode_ok(mode)) return 0;
  return cascade_plan(pool, seqs, shared_len, num_q_heads, T, mode).ws_bytes;
}

size_t kvt_cascade_workspace_bytes(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                   int32_t num_q_heads) {
  return kvt_cascade_workspace_bytes_ex(pool, seqs, shared_len, KVT_CASCADE_AUTO, num_q_heads);
}

int32_t kvt_cascade_uses_shared_pass(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                     int32_t num_q_heads) {
  if (check_pool(pool) != KVT_OK) return -1;
  int64_t T = 0;
  if (check_seqs(seqs, &T) != KVT_OK) return -1;
  if (!heads_ok(pool, num_q_heads, T)) return -1;
  if (check_shared(seqs, shared_len) != KVT_OK) return -1;
  return cascade_plan(pool, seqs, shared_len, num_q_heads, T).use_shared ? 1 : 0;
}

kvt_status kvt_cascade_extend_attention(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                        const void* q, int32_t num_q_heads, float scale, void* out, float* lse,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  return kvt_cascade_extend_attention_ex(pool, seqs, shared_len, KVT_CASCADE_AUTO, q, num_q_heads, scale, out, lse,
                                         workspace, workspace_bytes, stream);
}

kvt_status kvt_cascade_extend_attention_ex(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                           int32_t mode, const void* q, int32_t num_q_heads, float scale, void* out,
                                           float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  kvt_status st = check_pool(pool);
  if (st != KVT_OK) return st;
  int64_t T = 0;
  if ((st = check_seqs(seqs, &T)) != KVT_OK) return st;
  if ((st = check_shared(seqs, shared_len)) != KVT_OK) return st;
  if (!mode_ok(mode)) return KVT_ERR_INVALID_ARG;
  if (workspace == nullptr && workspace_bytes == 0)   // no scratch: the plain extend computes the same
    return kvt_extend_attention(pool, seqs, q, num_q_heads, scale, out, lse, nullptr, 0, stream);
  if (q == nullptr || out == nullptr) return KVT_ERR_INVALID_ARG;
  if (!heads_ok(pool, num_q_heads, T)) return KVT_ERR_INVALID_ARG;
  if (!(scale > 0.f) || !std::isfinite(scale)) return KVT_ERR_INVALID_ARG;
  if ((st = check_table_ids(pool, seqs)) != KVT_OK) return st;
  if ((st = check_outputs(pool, q, num_q_heads, out, lse, T)) != KVT_OK) return st;
  const ExtendPlan plan = cascade_plan(pool, seqs, shared_len, num_q_heads, T, mode);
  if (workspace == nullptr || workspace_bytes < plan.ws_bytes) return KVT_ERR_WORKSPACE;
  if (!aligned16(workspace)) return KVT_ERR_INVALID_ARG;
  if (!plan.use_shared)   // the plain extend is estimated faster: same result, same bits as kvt_extend_attention
    return launch_extend_plan(pool, seqs, q, num_q_heads, scale, out, lse, T, plan, workspace, stream);

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int G = num_q_heads / pool->num_kv_heads;
  const int nparts = plan.nsplit_shared + plan.nsplit;
  ExtendPlan parts = plan;
  parts.nsplit = nparts;                       // partial buffers: the shared part's splits, then the private ones
  kvt::ExtendArgs a = base_args(pool, seqs, q, num_q_heads, scale, out, lse, T, parts, workspace);
  a.direct = 0;

  // One launch for both parts, the shared part's (longer) units first, so
  // the private parts' units fill the CUs the shared part leaves idle at
  // its end.  Shared part (sequence 0 of the first launch): every new token
  // of the batch against keys [0, shared_len), all of them visible (one
  // virtual sequence whose causal limits start at shared_len - 1), read
  // through the first sequence's table row, with its own key splits.
  // Private parts (the second group): each sequence over keys
  // [shared_len, P_b + i], causal.  Sequences beyond one launch's
  // descriptors go to further launches of private parts only.
  a.nsplit = plan.nsplit_shared;
  a.part_base = 0;
  a.kbeg = 0;
  a.kend = shared_len;
  a.kbeg2 = shared_len;
  a.kend2 = INT32_MAX;
  a.nsplit2 = plan.nsplit;
  a.part_base2 = plan.nsplit_shared;
  std::vector<int32_t> row_off(seqs->num_seqs + 1, 0);
  for (int b = 0; b < seqs->num_seqs; ++b) row_off[b + 1] = row_off[b] + seqs->suffix_len[b];
  size_t c0 = 0;
  for (bool first = true; first || c0 < plan.order.size(); first = false) {
    int n = 0;
    int32_t units = 0;
    if (first) {
      a.seq[0] = kvt::SeqDesc{plan.order[0], shared_len - 1, (int32_t)T, 0};
      a.unit_begin[0] = 0;
      units = row_tiles((int32_t)T, G) * plan.nsplit_shared;
      n = 1;
    }
    a.second = first ? 1 : 0;
    for (; n < kvt::kSeqsPerLaunch && c0 < plan.order.size(); ++n, ++c0) {
      const int b = plan.order[c0];
      a.seq[n] = kvt::SeqDesc{b, seqs->prefix_len[b], seqs->suffix_len[b], row_off[b]};
      a.unit_begin[n] = units;
      units += row_tiles(seqs->suffix_len[b], G) * plan.nsplit;
    }
    a.nseq = n;
    a.unit_begin[n] = units;
    const int64_t grid = (int64_t)units * pool->num_kv_heads;
    if (grid > INT32_MAX) return KVT_ERR_INVALID_ARG;
    const hipError_t e = kvt::launch_extend(a, pool->dtype, pool->head_dim, (int)grid, s);
    if (e != hipSuccess) return device_error(e);
  }
  return combine(a, pool, out, lse, T, num_q_heads, nparts, s);
}

size_t kvt_decode_workspace_bytes(const kvt_pool* pool, const kvt_seqs* seqs, int32_t num_q_heads) {
  if (check_pool(pool) != KVT_OK) return 0;
  int64_t T = 0;
  if (check_seqs(seqs, &T) != KVT_OK || T != seqs->num_seqs) return 0;
  if (!heads_ok(pool, num_q_heads, T)) return 0;
  if (num_q_heads / pool->num_kv_heads > kvt::kDecMaxGroup) return 0;
  return make_decode_plan(pool, seqs, num_q_heads).ws_bytes;
}

kvt_status kvt_decode_attention(const kvt_pool* pool, const kvt_seqs* seqs, const void* q, int32_t num_q_heads,
                                float scale, void* out, float* lse, void* workspace, size_t workspace_bytes,
                                void* stream) {
  kvt_status st = check_pool(pool);
  if (st != KVT_OK) return st;
  int64_t T = 0;
  if ((st = check_seqs(seqs, &T)) != KVT_OK) return st;
  if (T != seqs->num_seqs) return KVT_ERR_INVALID_ARG;   // one new token per sequence
  if (q == nullptr || out == nullptr) return KVT_ERR_INVALID_ARG;
  if (!heads_ok(pool, num_q_heads, T)) return KVT_ERR_INVALID_ARG;
  if (num_q_heads / pool->num_kv_heads > kvt::kDecMaxGroup) return KVT_ERR_UNSUPPORTED;
  if (!(scale > 0.f) || !std::isfinite(scale)) return KVT_ERR_INVALID_ARG;
  if ((st = check_table_ids(pool, seqs)) != KVT_OK) return st;
  if ((st = check_outputs(pool, q, num_q_heads, out, lse, T)) != KVT_OK) return st;

  ExtendPlan plan = make_decode_plan(pool, seqs, num_q_heads);
  if (plan.nsplit > 1) {
    if (workspace == nullptr && workspace_bytes == 0) {
      plan.nsplit = 1;
    } else if (workspace == nullptr || workspace_bytes < plan.ws_bytes) {
      return KVT_ERR_WORKSPACE;
    } else if (!aligned16(workspace)) {
      return KVT_ERR_INVALID_ARG;
    }
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  kvt::ExtendArgs a = base_args(pool, seqs, q, num_q_heads, scale, out, lse, T, plan, workspace);
  for (size_t c0 = 0; c0 < plan.order.size(); c0 += kvt::kSeqsPerLaunch) {
    const int n = (int)std::min<size_t>(kvt::kSeqsPerLaunch, plan.order.size() - c0);
    a.nseq = n;
    for (int i = 0; i < n; ++i) {
      const int b = plan.order[c0 + i];
      a.seq[i] = kvt::SeqDesc{b, seqs->prefix_len[b], 1, b};   // row of sequence b is b
      a.unit_begin[i] = i * plan.nsplit;
    }
    a.unit_begin[n] = n * plan.nsplit;
    const int64_t grid = (int64_t)n * plan.nsplit * pool->num_kv_heads;
    const hipError_t e = kvt::launch_decode(a, pool->dtype, pool->head_dim, (int)grid, s);
    if (e != hipSuccess) return device_error(e);
  }
  return plan.nsplit > 1 ? combine(a, pool, out, lse, T, num_q_heads, plan.nsplit, s) : KVT_OK;
}

}  // extern "C"
