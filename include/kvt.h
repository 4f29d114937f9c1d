/*
 * kvt.h -- paged-KV extend attention for AMD MI355X (gfx950).
 *
 * The computation a prefix hit leaves to do in a ReAct turn: KV reuse exists
 * so that a long reusable prefix is not prefilled again (paper §1, §2.2); the
 * S new tokens of the turn attend causally over the P reused positions plus
 * themselves, and their K/V are written into freshly allocated cache pages
 * once the tokens have taken part in inference (§5.1, §6.2).  A forked
 * context shares its parent's pages (§5.2, §6.1); a replaced middle message
 * invalidates the cached suffix, which is recomputed as a longer suffix over
 * a shorter reused prefix (§5.1).
 *
 * Conventions shared by every call
 * --------------------------------
 * Pool: K and V of ONE layer, each [num_blocks][num_kv_heads][16][head_dim],
 *   contiguous, head_dim fastest.  Page (block) size is 16 tokens.
 * Sequences: B >= 1.  Sequence b reuses P_b >= 0 positions already in the
 *   pool and adds S_b >= 1 new tokens at logical positions P_b .. P_b+S_b-1.
 *   Logical position p of sequence b lives at slot p % 16 of physical block
 *   block_table[b * max_blocks + p / 16].  Table entries past the last used
 *   block are ignored (they may hold -1).
 * Packed token rows: every per-token tensor (q, out, lse, k_new, v_new)
 *   stores sequence b's new tokens at rows off_b .. off_b+S_b-1 with
 *   off_b = S_0 + ... + S_{b-1}; T = sum_b S_b.
 * GQA: query head h reads kv-head h / (Hq / Hkv) (consecutive head groups).
 * Dtypes: q, out, k_new, v_new and both pools share the pool dtype.  bf16
 *   inputs feed bf16 MFMA directly; fp32 inputs are rounded to bf16 (RNE) in
 *   registers and take the same path.  Softmax and accumulation are fp32.
 * Ownership: every buffer belongs to the caller.  The library allocates no
 *   device memory and keeps no state between calls except a cached device
 *   property and, for kvt_extend_attention_noalloc only, one static scratch
 *   array per GPU (KVT_NOALLOC_SCRATCH_BYTES) and its looked-up address;
 *   calls are reentrant, except that no-alloc calls overlapping on one GPU
 *   share that scratch.
 * Asynchrony: KVT_OK means the work is enqueued on `stream` (a hipStream_t;
 *   NULL = the default stream).  Device-side faults surface at the caller's
 *   next synchronisation.  Pool pages read or written by a call must not be
 *   freed or reused until the stream has passed the call.
 * Errors: every argument check runs on the host before any HIP call; on a
 *   non-OK return nothing has been enqueued.  KVT_ERR_DEVICE reports a failed
 *   launch; kvt_last_hip_error() then returns the hipError_t (per thread).
 * Unchecked block ids: without a host mirror of the block table (checked
 *   mode off), an out-of-range id is never dereferenced: extend clamps it to
 *   the last page of the pool and append skips it; the result is then
 *   unspecified, not a fault.
 */
#ifndef KVT_H_
#define KVT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVT_BLOCK_SIZE 16

typedef enum {
  KVT_OK = 0,
  KVT_ERR_INVALID_ARG = 1,   /* null pointer, bad length, table too narrow, aliasing */
  KVT_ERR_UNSUPPORTED = 2,   /* head_dim not in {64,128}, unknown dtype */
  KVT_ERR_OUT_OF_RANGE = 3,  /* checked mode: block id outside [0,num_blocks) or duplicate append slot */
  KVT_ERR_WORKSPACE = 4,     /* non-null workspace smaller than kvt_extend_workspace_bytes() */
  KVT_ERR_DEVICE = 5,        /* HIP launch failure; see kvt_last_hip_error() */
  KVT_ERR_SCRATCH_LIMIT = 6  /* kvt_extend_attention_noalloc: partials exceed KVT_NOALLOC_SCRATCH_BYTES */
} kvt_status;

typedef enum { KVT_DTYPE_BF16 = 0, KVT_DTYPE_F32 = 1 } kvt_dtype;

/* The paged KV pool of one layer. */
typedef struct {
  void*   k;             /* device, [num_blocks][num_kv_heads][16][head_dim] */
  void*   v;             /* device, same shape and dtype as k */
  int64_t num_blocks;    /* >= 1; 64-bit: 2^20 bf16 blocks span 32 GiB */
  int32_t num_kv_heads;  /* Hkv >= 1 */
  int32_t head_dim;      /* D in {64, 128} */
  int32_t dtype;         /* kvt_dtype of k, v and every per-token tensor */
} kvt_pool;

/* The sequences of one call. */
typedef struct {
  int32_t        num_seqs;          /* B >= 1 */
  const int32_t* prefix_len;        /* HOST [B], P_b >= 0: positions already in the pool */
  const int32_t* suffix_len;        /* HOST [B], S_b >= 1: new tokens of this call */
  const int32_t* block_table;       /* DEVICE [B][max_blocks], row-major physical block ids */
  const int32_t* block_table_host;  /* HOST copy of block_table, or NULL; non-NULL turns on checked mode */
  int32_t        max_blocks;        /* row stride; ceil((P_b+S_b)/16) <= max_blocks for every b */
} kvt_seqs;

/*
 * kvt_append_kv -- write the new tokens' K/V into their pages.
 *
 * For every b, t < S_b, kv-head g, with p = P_b + t:
 *   k_pool[block_table[b][p/16]][g][p%16][:] = k_new[off_b + t][g][:]  (same for v)
 * a bitwise copy.  k_new, v_new: device [T][Hkv][D] in the pool dtype; they
 * and the pools must be 16-byte aligned (else KVT_ERR_INVALID_ARG).
 * No other pool byte is written.  Targets must be distinct across the call
 * (checked mode rejects a repeated (block, slot) with KVT_ERR_OUT_OF_RANGE);
 * blocks shared by several sequences (a fork) are read-only here as long as
 * no sequence's new positions fall in them.
 */
kvt_status kvt_append_kv(const kvt_pool* pool, const kvt_seqs* seqs,
                         const void* k_new, const void* v_new, void* stream);

/*
 * kvt_extend_attention -- causal attention of the new tokens over prefix + suffix.
 *
 * For every b, new token i < S_b, query head h (g = h / (Hq/Hkv)):
 *   s_j = scale * <q[off_b+i][h], K_b[j]>,  j = 0 .. P_b + i  (own position included)
 *   out[off_b+i][h] = sum_j softmax(s)_j V_b[j]
 *   lse[off_b+i][h] = ln sum_j exp(s_j)            (natural log; optional)
 * K_b/V_b are read through the block table; both the reused prefix and this
 * call's suffix come from the pool, so kvt_append_kv for the same tokens must
 * be enqueued first (same stream, or otherwise ordered before this call).
 *
 * q: device [T][Hq][D]; out: device [T][Hq][D] (may not overlap q or a pool);
 * lse: device float [T][Hq] or NULL.  num_q_heads must be a multiple of Hkv,
 * and T * num_q_heads at most INT32_MAX (else KVT_ERR_INVALID_ARG).
 * q, out, the pools and the workspace must be 16-byte aligned, lse 4-byte
 * aligned (else KVT_ERR_INVALID_ARG); fresh device allocations are.
 * scale: finite and > 0 (usually 1/sqrt(D)).
 * workspace: device scratch for split-key partial results.  Pass NULL/0 to
 * run without splitting; otherwise workspace_bytes must be at least
 * kvt_extend_workspace_bytes() for the same arguments (else
 * KVT_ERR_WORKSPACE).  The split decision depends only on the lengths and
 * shapes, so results are bit-reproducible for given arguments.
 */
kvt_status kvt_extend_attention(const kvt_pool* pool, const kvt_seqs* seqs,
                                const void* q, int32_t num_q_heads, float scale,
                                void* out, float* lse,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Workspace that lets kvt_extend_attention split long key ranges over more
 * workgroups (short suffixes, small batches).  0 when no split is planned or
 * the arguments are invalid.  Host-only; enqueues nothing. */
size_t kvt_extend_workspace_bytes(const kvt_pool* pool, const kvt_seqs* seqs, int32_t num_q_heads);

/* Size of the static scratch array of kvt_extend_attention_noalloc (64 MiB),
 * held by each GPU the library runs on until the process ends. */
#define KVT_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * kvt_extend_attention_noalloc -- kvt_extend_attention for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): no workspace argument, and no
 * device allocation of any kind.
 *
 * Same arguments (less the workspace), checks and result as
 * kvt_extend_attention with a workspace of kvt_extend_workspace_bytes(): the
 * same split plan runs, so out and lse are bit-identical to that call.  The
 * split partials go to a static array of KVT_NOALLOC_SCRATCH_BYTES that each
 * GPU holds (looked up by its symbol address on the first call on that
 * device).  A call whose plan needs more (kvt_extend_workspace_bytes() >
 * KVT_NOALLOC_SCRATCH_BYTES) returns KVT_ERR_SCRATCH_LIMIT with nothing
 * enqueued; an unsplit plan needs none.  Every call on one GPU shares that
 * GPU's array, which keeps the last call's contents: two no-alloc calls that
 * overlap on one GPU (different streams, no ordering between them) race and
 * must not be issued; nothing in the array needs clearing between calls.
 */
kvt_status kvt_extend_attention_noalloc(const kvt_pool* pool, const kvt_seqs* seqs,
                                        const void* q, int32_t num_q_heads, float scale,
                                        void* out, float* lse, void* stream);

/*
 * kvt_cascade_extend_attention -- kvt_extend_attention for a batch whose
 * sequences share their first shared_len positions (forked sub-agents reuse
 * the parent's KV: paper sections 2.1 and 5.2, shared-KV state section 6.1).
 *
 * Same result as kvt_extend_attention on the same arguments, computed in
 * three steps: every new token of the batch attends over the shared keys
 * [0, shared_len) at once (one pass over the shared pages for the whole
 * batch), each sequence attends over its private keys [shared_len, P_b + i],
 * and the two partial results merge by their log-sum-exp weights.  The
 * first two steps share one kernel launch (the private parts' work fills
 * the CUs the shared part leaves idle), the merge is a second launch.
 *
 * shared_len: a positive multiple of 16, at most every prefix_len[b]; the
 * first shared_len/16 block-table entries must be the same pages in every
 * row (checked mode verifies it; otherwise the result is unspecified).
 * Violations give KVT_ERR_INVALID_ARG.  workspace: device scratch of at
 * least kvt_cascade_workspace_bytes() for the same arguments (else
 * KVT_ERR_WORKSPACE); NULL/0 runs the call as kvt_extend_attention without
 * a workspace.  Other arguments as for kvt_extend_attention.
 */
kvt_status kvt_cascade_extend_attention(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                        const void* q, int32_t num_q_heads, float scale,
                                        void* out, float* lse,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* Workspace of kvt_cascade_extend_attention: (key splits of the shared
 * part + key splits of the private parts) partial results per row, or
 * kvt_extend_workspace_bytes() when the call runs as the plain extend (see
 * kvt_cascade_uses_shared_pass).  0 when the arguments are invalid.
 * Host-only; enqueues nothing. */
size_t kvt_cascade_workspace_bytes(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                   int32_t num_q_heads);

/* Plan choice of the _ex cascade calls.  AUTO: the estimate below picks
 * (what kvt_cascade_extend_attention and kvt_cascade_workspace_bytes do);
 * SHARED_PASS: always the three-step cascade; PLAIN: always the plain extend
 * plan.  Any other value gives KVT_ERR_INVALID_ARG (0 bytes). */
typedef enum { KVT_CASCADE_AUTO = 0, KVT_CASCADE_SHARED_PASS = 1, KVT_CASCADE_PLAIN = 2 } kvt_cascade_mode;
kvt_status kvt_cascade_extend_attention_ex(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                           int32_t mode, const void* q, int32_t num_q_heads, float scale,
                                           void* out, float* lse,
                                           void* workspace, size_t workspace_bytes, void* stream);
size_t kvt_cascade_workspace_bytes_ex(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                      int32_t mode, int32_t num_q_heads);

/* Whether kvt_cascade_extend_attention with a workspace runs the three-step
 * cascade (1) or the plain extend plan (0), which it does when a host
 * estimate (key tiles of work over the CUs plus the partial results the
 * cascade writes and merges) says the plain extend is faster: with long
 * suffixes every sequence's row tiles are nearly full, so the shared pass
 * saves little key traffic and its partials cost more.  The result is the
 * same either way; the plain plan gives the same bits as
 * kvt_extend_attention.  -1 for invalid arguments.  Host-only. */
int32_t kvt_cascade_uses_shared_pass(const kvt_pool* pool, const kvt_seqs* seqs, int32_t shared_len,
                                     int32_t num_q_heads);

/*
 * kvt_decode_attention -- one decoding step: attention of each sequence's
 * single new token over its whole cache (paper section 5.2: once a request's
 * prefill completes, LLM decoding proceeds token by token over the same KV).
 *
 * The same operation as kvt_extend_attention with S_b = 1 for every b (the
 * new token at position P_b sees keys 0..P_b, its own K/V appended first by
 * kvt_append_kv):
 *   out[b][h] = sum_j softmax(scale * <q[b][h], K_b[j]>)_j V_b[j],  j = 0 .. P_b
 *   lse[b][h] = ln sum_j exp(scale * <q[b][h], K_b[j]>)            (optional)
 * Row b of q/out/lse is sequence b.  Built for large batches whose cost is
 * streaming every sequence's K/V once from HBM.
 *
 * Arguments as for kvt_extend_attention, and: every suffix_len[b] must be 1
 * (else KVT_ERR_INVALID_ARG); Hq/Hkv must be at most 32 (else
 * KVT_ERR_UNSUPPORTED).  workspace: device scratch for key-split partial
 * results; NULL/0 runs unsplit, otherwise at least
 * kvt_decode_workspace_bytes() for the same arguments (else
 * KVT_ERR_WORKSPACE).  Results are bit-reproducible for given arguments.
 */
kvt_status kvt_decode_attention(const kvt_pool* pool, const kvt_seqs* seqs,
                                const void* q, int32_t num_q_heads, float scale,
                                void* out, float* lse,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Workspace that lets kvt_decode_attention split each sequence's keys over
 * several workgroups (small batches).  0 when no split is planned or the
 * arguments are invalid.  Host-only; enqueues nothing. */
size_t kvt_decode_workspace_bytes(const kvt_pool* pool, const kvt_seqs* seqs, int32_t num_q_heads);

/* Direction of kvt_copy_blocks. */
typedef enum {
  KVT_COPY_TO_HOST = 0,     /* pool pages -> host buffer (offload)  */
  KVT_COPY_TO_DEVICE = 1    /* host buffer -> pool pages (reload)   */
} kvt_copy_direction;

/*
 * kvt_copy_blocks -- move a list of pages between the HBM pools and host
 * memory (the GPU <-> host tier of the multi-tier KV cache: pages leave HBM
 * under memory pressure and come back for reuse; paper sections 6 and 7).
 *
 * For i < num_ids, with page = block_ids[i]:
 *   KVT_COPY_TO_HOST:   host[i][0] = K pool page, host[i][1] = V pool page
 *   KVT_COPY_TO_DEVICE: the reverse
 * where host is a packed [num_ids][2][Hkv][16][D] array of the pool dtype.
 *
 * block_ids: DEVICE int32 [num_ids].  block_ids_host: optional HOST mirror;
 * when given, every id must lie in [0, num_blocks) and, for
 * KVT_COPY_TO_DEVICE, appear once (else KVT_ERR_OUT_OF_RANGE).  Without it an
 * id outside the pool is skipped (never dereferenced).
 * host: pinned host memory allocated through HIP (hipHostMalloc or
 * equivalent), at least num_ids * 2 * Hkv * 16 * D * elem bytes; other
 * memory gives KVT_ERR_INVALID_ARG.  The GPU reads/writes it directly over
 * the host link; it must stay allocated until the stream passes the call.
 * num_ids = 0 is a no-op.  Enqueued on `stream`; nothing is allocated.
 */
kvt_status kvt_copy_blocks(const kvt_pool* pool, const int32_t* block_ids, const int32_t* block_ids_host,
                           int64_t num_ids, void* host, int32_t direction, void* stream);

/* ------------------------------------------------------------------------
 * Host block manager (CPU only; no HIP calls).
 *
 * Lifecycle states of message versions (paper section 5.2), the aggregate
 * state of shared KV (section 6.1), state-prioritized admission
 * (Algorithm 1) and MRU eviction inside the Suspended tier (section 6.2),
 * over a pool of num_pages KV pages whose ids it hands out for the block
 * tables.  A context is an ordered list of messages; a message's current
 * version has a state and, once it took part in inference, a KV entry of
 * ceil(tokens / 16) pages.  Forked contexts map their inherited messages to
 * the parent's entries.  An entry's tier is the strongest state among the
 * versions that map it: Pinned > Active > Suspended > Discarded (Expired and
 * Temporary).  Newly written-back entries are admitted in message order:
 * Temporary-only entries bypass the cache; otherwise the missing pages are
 * freed from resident entries not read by an in-flight request, Discarded
 * first (earliest discarded first), then Suspended (most recently suspended
 * first), then Active (earliest first), then -- for a Pinned newcomer only --
 * Pinned (earliest first); the newcomer is admitted if that covered it
 * (entries freed on the way stay freed); entries that changed tier in the
 * same call rank by creation order.  Pages come from the lowest free ids.
 * At a request, a message whose entry is gone -- and every later message of
 * the context -- is a miss and gets a fresh version to recompute.
 * Not thread-safe: one caller at a time per manager.
 * ---------------------------------------------------------------------- */
typedef struct kvt_manager kvt_manager;

/* Lifecycle states as returned by kvt_mgr_message_state. */
enum { KVT_PINNED = 0, KVT_ACTIVE = 1, KVT_SUSPENDED = 2, KVT_EXPIRED = 3, KVT_TEMPORARY = 4 };
/* Entry tiers as returned by kvt_mgr_entry_tier. */
enum { KVT_TIER_PINNED = 0, KVT_TIER_ACTIVE = 1, KVT_TIER_SUSPENDED = 2, KVT_TIER_DISCARDED = 3 };

/* What one request-boundary call did. */
typedef struct {
  int64_t admitted_entries, admitted_pages;   /* written back into the cache          */
  int64_t bypassed_entries;                    /* Temporary KV, not stored             */
  int64_t rejected_entries;                    /* not enough releasable capacity       */
  int64_t released_entries, released_pages;    /* evicted or reclaimed to make room    */
  int64_t hit_tokens, miss_tokens;             /* kvt_mgr_start_prefill: reused / to recompute */
} kvt_mgr_report;

/* A manager over pages 0 .. num_pages-1 (all free).  NULL on a bad size. */
kvt_manager* kvt_mgr_create(int64_t num_pages);
void kvt_mgr_destroy(kvt_manager* m);
int64_t kvt_mgr_free_pages(const kvt_manager* m);
int64_t kvt_mgr_live_entries(const kvt_manager* m);

/* Context events (KVT_ERR_INVALID_ARG on an unknown or terminated context,
 * a bad message index, or an event the state does not allow: fork, one_off,
 * replace, remove and terminate only between requests). */
kvt_status kvt_mgr_spawn(kvt_manager* m, int64_t ctx);
kvt_status kvt_mgr_fork(kvt_manager* m, int64_t parent, int64_t child);  /* child maps the parent's entries */
kvt_status kvt_mgr_append(kvt_manager* m, int64_t ctx, int64_t tokens);   /* new message, Active (Temporary if one-off) */
kvt_status kvt_mgr_one_off(kvt_manager* m, int64_t ctx);                  /* existing and later messages Temporary; Pinned stay */
kvt_status kvt_mgr_pin(kvt_manager* m, int64_t ctx, int64_t msg_index);     /* not a Temporary message */
kvt_status kvt_mgr_unpin(kvt_manager* m, int64_t ctx, int64_t msg_index);  /* -> Suspended; Active in a request, Temporary if one-off, Expired if terminated */
kvt_status kvt_mgr_replace(kvt_manager* m, int64_t ctx, int64_t msg_index, int64_t tokens);
kvt_status kvt_mgr_remove(kvt_manager* m, int64_t ctx, int64_t msg_index);
    /* replace/remove: the versions of msg_index and of every later message expire; the
       message (replace) and the later ones get fresh versions, Active (Temporary if one-off) */
kvt_status kvt_mgr_terminate(kvt_manager* m, int64_t ctx);               /* ordinary messages expire; Pinned stay */

/* A request's boundaries, in this order.
 *   begin_request: the LLM call is issued; Suspended messages become Active
 *     again.  Nothing is held yet: until its prefill starts, the request's
 *     entries are Active-tier KV that admission may take (Algorithm 1's
 *     Active step).
 *   start_prefill: hits and misses are resolved against what is resident
 *     now (report: hit_tokens, miss_tokens); the context's resident entries
 *     are held until end_request, since the kernels read their pages.
 *   prefill_done: every message without KV gets an entry, Active messages
 *     become Suspended, and the new entries are admitted in message order
 *     (report: admitted / bypassed / rejected / released).
 *   end_request: the held entries become releasable; Active messages become
 *     Suspended.  Allowed from any phase after begin (an abort). */
kvt_status kvt_mgr_begin_request(kvt_manager* m, int64_t ctx);
kvt_status kvt_mgr_start_prefill(kvt_manager* m, int64_t ctx, kvt_mgr_report* report);
kvt_status kvt_mgr_prefill_done(kvt_manager* m, int64_t ctx, kvt_mgr_report* report);
kvt_status kvt_mgr_end_request(kvt_manager* m, int64_t ctx);

/* Trace replay, for callers that drive the manager from a recorded event
 * trace (the paper evaluates on replayed agent traces, section 8.1): n
 * events, each four int64 {op, a, b, c}, op one of KVT_MGR_OP_* and a, b, c
 * the arguments of that call in order (context, then index / child /
 * tokens, then tokens; unused ones ignored).  Each event runs exactly as the
 * matching call; a failing event is skipped.  The reports of start_prefill
 * and prefill_done are summed into totals (NULL: not reported).  Returns
 * the number of events that returned KVT_OK, or -1 for a NULL manager, a
 * NULL event array with n > 0, or n < 0. */
enum {
  KVT_MGR_OP_SPAWN = 0, KVT_MGR_OP_FORK = 1, KVT_MGR_OP_APPEND = 2, KVT_MGR_OP_ONE_OFF = 3, KVT_MGR_OP_PIN = 4,
  KVT_MGR_OP_UNPIN = 5, KVT_MGR_OP_REPLACE = 6, KVT_MGR_OP_REMOVE = 7, KVT_MGR_OP_TERMINATE = 8,
  KVT_MGR_OP_BEGIN_REQUEST = 9, KVT_MGR_OP_START_PREFILL = 10, KVT_MGR_OP_PREFILL_DONE = 11,
  KVT_MGR_OP_END_REQUEST = 12
};
int64_t kvt_mgr_replay(kvt_manager* m, const int64_t* events, int64_t n, kvt_mgr_report* totals);

/* Queries (-1 for an unknown context or index).  message_pages: the page
 * ids of the message's resident entry (up to cap written; pages may be NULL
 * to ask for the count), their count, or -1 if it has none resident.
 * Token counts (append, replace) are 1 .. 2^40. */
int32_t kvt_mgr_message_state(const kvt_manager* m, int64_t ctx, int64_t msg_index);
int32_t kvt_mgr_entry_tier(const kvt_manager* m, int64_t ctx, int64_t msg_index);
int64_t kvt_mgr_message_pages(const kvt_manager* m, int64_t ctx, int64_t msg_index, int32_t* pages, int64_t cap);

/* Static English text for a status code (never NULL). */
const char* kvt_status_str(kvt_status s);

/* hipError_t of the last KVT_ERR_DEVICE returned on this thread (0 if none). */
int kvt_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVT_H_ */
