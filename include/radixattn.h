/*
 * radixattn.h -- C ABI of the RadixAttention hot path on MI355X (gfx950).
 *
 * Two halves:
 *
 *  1. Host radix cache (section 3 of the SGLang paper, "RadixAttention", and
 *     Algorithm 1, cache-aware scheduling with continuous batching): a radix
 *     tree mapping token sequences to slots of a token-granular KV pool (one
 *     token per page), reference counters that protect what running requests
 *     use, LRU eviction of unreferenced leaves, and the shared slot pool.
 *     Not thread-safe per handle: one scheduler thread drives it, as the paper
 *     keeps the tree on the CPU.
 *
 *  2. Device attention over that pool.  K and V live in two caller-owned
 *     device arrays [S, Hkv, D] (bf16, row-major); request r reads position j
 *     of its context from slot req_to_token[req_pool_idx[r] * rtt_stride + j].
 *     extend: prefill of new tokens over a cached prefix plus causal attention
 *     among themselves.  decode: one query token per request over its whole
 *     context.  Every device call is asynchronous on the caller's HIP stream
 *     and allocates no device memory; all pointers are device pointers unless
 *     stated.  Results match float64 softmax attention (see the oracle) within
 *     bf16 rounding.
 *
 * Conventions.  Tokens and slots are int32 (S < 2^31).  Host lengths are
 * int64.  Node handles are int64 ids; the root is 0; ids are never reused
 * (after 2^31 - 1 nodes a match or insert returns RA_ENOMEM, no effect).
 * Every call returns RA_OK or a negative status and never throws; the text of
 * the last error on the calling thread is available from ra_last_error().  A
 * failing call changes nothing, with one exception: when the host runs out of
 * memory inside a tree or router operation, the call returns RA_ENOMEM and
 * the handle may be left part-way through it (destroy it).  Query head h uses
 * key/value head
 * h / (Hq / Hkv) (contiguous groups).
 */
#ifndef RADIXATTN_H
#define RADIXATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  RA_OK = 0,
  RA_EINVAL = -1, /* bad argument, unknown node, counter underflow, bad slot */
  RA_ENOMEM = -2, /* pool has fewer free slots than asked (no effect), or host memory ran out */
  RA_EHIP = -3    /* a HIP launch failed; message holds hipGetErrorString */
};

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* ra_last_error(void);

/* ===================================================================== */
/* Host radix cache (section 3; Algorithm 1).                            */
/* ===================================================================== */

typedef struct ra_cache ra_cache;

/* Creates a cache over a pool of `pool_slots` slots.  The free slots form a
 * FIFO queue initialised to `initial_free_order` (a permutation of
 * [0, pool_slots), copied), or to 0, 1, ... when it is NULL.  EINVAL if the
 * order is not a permutation. */
int ra_cache_create(int64_t pool_slots, const int32_t* initial_free_order, ra_cache** out);
void ra_cache_destroy(ra_cache* c);

/* Longest cached prefix of tokens[0..n) (Algorithm 1, match_prefix).
 * Writes its slots to out_slots (capacity n; may be NULL), its length to
 * *out_len and the node covering exactly that prefix to *out_node (0 when
 * nothing matches).  A match ending inside an edge splits it there.  Every
 * node on the walked path becomes most recently used. */
int ra_match_prefix(ra_cache* c, const int32_t* tokens, int64_t n, int32_t* out_slots,
                    int64_t* out_len, int64_t* out_node);

/* Lock / unlock the root-to-node path for a running request (section 3:
 * a node with a non-zero counter is never evicted).  *out_delta receives the
 * change of the evictable token count: <= 0 for inc, >= 0 for dec (Algorithm
 * 1 adds it to the available size).  dec on a path with a zero counter is
 * EINVAL.  out_delta may be NULL. */
int ra_inc_ref(ra_cache* c, int64_t node, int64_t* out_delta);
int ra_dec_ref(ra_cache* c, int64_t node, int64_t* out_delta);

/* Pool (Algorithm 1, P.alloc).  Pops n slots from the front of the free queue
 * into out_slots, or returns ENOMEM with no effect if fewer are free. */
int ra_alloc_slots(ra_cache* c, int64_t n, int32_t* out_slots);
/* Appends slots to the free queue in order.  EINVAL (no effect) if any slot
 * is out of range, already free, or repeated. */
int ra_free_slots(ra_cache* c, const int32_t* slots, int64_t n);

/* Inserts a finished sequence tokens[0..n) -> slots[0..n) (Algorithm 1,
 * T.insert).  Cached positions keep their slots; a caller slot that differs
 * from the cached one at the same position is returned to the pool.  Splits
 * an edge where the sequence diverges inside it.  *out_cached = positions
 * that were already cached, *out_node = node ending at position n (either may
 * be NULL).  The new leaf is unreferenced (evictable).  EINVAL (no effect)
 * for n >= 2^31, a new slot that is out of range or free, or differing
 * caller slots that are out of range, free or repeated. */
int ra_insert(ra_cache* c, const int32_t* tokens, const int32_t* slots, int64_t n,
              int64_t* out_cached, int64_t* out_node);

/* Evicts least recently used unreferenced leaves (ties: smaller node id)
 * until at least n_tokens slots were freed or nothing is evictable; whole
 * leaves only, so it may free more.  Freed slots join the back of the free
 * queue.  *out_freed = slots freed (may be NULL). */
int ra_evict(ra_cache* c, int64_t n_tokens, int64_t* out_freed);

int64_t ra_evictable_size(const ra_cache* c); /* tokens in unreferenced nodes */
int64_t ra_available_size(const ra_cache* c); /* free slots */
int64_t ra_cached_tokens(const ra_cache* c);  /* tokens held by the tree */
int64_t ra_num_nodes(const ra_cache* c);      /* live nodes, root included */

/* Canonical dump for exact comparisons: [clock, n_nodes, n_free, then per
 * live node in id order: id, parent (-1 for root), ref, stamp, len, len
 * tokens, len slots; then the free queue front to back].  *out_len gets the
 * number of int64 words; with buf == NULL only the length is reported;
 * EINVAL if cap is too small. */
int ra_snapshot(const ra_cache* c, int64_t* buf, int64_t cap, int64_t* out_len);

/* Eviction log, for a router that mirrors this tree (Appendix A.4: workers
 * commit their evictions to a queue the router applies later).  While
 * enabled, every leaf ra_evict frees appends one entry: the tokens of its
 * root-to-leaf path and the leaf's own length (the evicted suffix of that
 * path).  Disabling drops the pending entries. */
int ra_cache_log_evictions(ra_cache* c, int32_t enable);
/* Pops the oldest entry: tokens[0..*out_path_len) = its path,
 * *out_evicted_len = the evicted suffix length.  An empty log gives
 * *out_path_len = -1 and RA_OK.  EINVAL if cap < the path length (the entry
 * stays queued; *out_path_len reports the size needed). */
int ra_eviction_log_pop(ra_cache* c, int32_t* tokens, int64_t cap, int64_t* out_path_len,
                        int64_t* out_evicted_len);

/* ===================================================================== */
/* Host: data-parallel router meta-tree (Appendix A.4).                  */
/* ===================================================================== */

/* A trie over the token sequences of up to 64 replica workers; every node
 * records which workers hold its prefix.  Host memory only, not thread-safe
 * per handle (one router thread).  The view is what the caller reports:
 * inserts at dispatch, evictions when the caller commits them, so between
 * commits it may still credit a worker with a prefix it has dropped. */
typedef struct ra_router ra_router;

int ra_router_create(int32_t n_workers, ra_router** out); /* 1 <= n_workers <= 64 */
void ra_router_destroy(ra_router* r);
/* out_len[w] (n_workers entries) = the longest prefix of tokens[0..n) that
 * worker w holds in the router's view. */
int ra_router_match(const ra_router* r, const int32_t* tokens, int64_t n, int64_t* out_len);
/* Records that worker holds tokens[0..n) (splits nodes where needed). */
int ra_router_insert(ra_router* r, int32_t worker, const int32_t* tokens, int64_t n);
/* Commits one eviction of the worker: it dropped the last evicted_len tokens
 * of the path tokens[0..path_len) and everything below them.  Ranges the
 * router never recorded are ignored.  Nodes no worker holds are freed. */
int ra_router_evict(ra_router* r, int32_t worker, const int32_t* tokens, int64_t path_len,
                    int64_t evicted_len);
int64_t ra_router_num_nodes(const ra_router* r);                   /* live nodes, root included */
int64_t ra_router_held_tokens(const ra_router* r, int32_t worker); /* -1 for a bad worker */

/* ===================================================================== */
/* Device: KV pool and attention (gfx950 HIP kernels).                   */
/* ===================================================================== */

/* Scatter of new tokens' K and V into their pool slots (page size one,
 * section 3): k_pool[slots[i]] = k_new[i], v_pool[slots[i]] = v_new[i], each
 * row Hkv * D bf16.  Slots outside [0, pool_slots) are skipped.  Pointers
 * must be 16-byte aligned. */
int ra_store_kv(const int32_t* slots, const void* k_new, const void* v_new, int64_t n_tokens,
                void* k_pool, void* v_pool, int64_t pool_slots, int32_t hkv, int32_t d,
                hipStream_t stream);

/* Extend attention (prefill of new tokens over a cached prefix; Appendix A.1
 * defines prefill, section 3 the reuse of a prefix's KV cache).
 *   q      [total_tokens, Hq, D] bf16, rows of request r at extend_start[r] ..
 *   k_new, v_new [total_tokens, Hkv, D] bf16, the new tokens' K and V (same rows)
 *   k_pool, v_pool [pool_slots, Hkv, D] bf16; prefix position j < P_r of
 *          request r is read from slot req_to_token[req_pool_idx[r] *
 *          rtt_stride + j]; req_to_token is int32 [rtt_rows, rtt_stride]
 *   prefix_lens, extend_lens, extend_start, req_pool_idx: int32 [B]
 *   max_extend_len: host upper bound of extend_lens (sizes the grid; every
 *          extend_lens[r] must be <= it: rows past it are never written)
 *   out    [sum E, Hq, D] bf16
 * New token i of request r (position P_r + i) attends positions 0 .. P_r + i.
 * Requires Hq % Hkv == 0, G = Hq / Hkv in {1, 2, 4, 8, 16}, D in {64, 128}.
 * Device-side bounds: table rows, prefix lengths, token rows and slots are
 * clamped into their arrays (out-of-range inputs give undefined values, never
 * an out-of-bounds access). */
int ra_extend_attention(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                        const void* k_pool, const void* v_pool, int64_t pool_slots,
                        const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                        const int32_t* req_pool_idx, const int32_t* prefix_lens,
                        const int32_t* extend_lens, const int32_t* extend_start, int32_t batch,
                        int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                        void* out, hipStream_t stream);

/* Extend attention with key splits, for batches whose work items would not
 * fill the chip (few requests or a head shard; the same operation as
 * ra_extend_attention, section 3 and Appendix A.1).  Each item's keys are cut
 * into runs of whole tiles processed in parallel; each run writes its rows'
 * output normalised over its keys (fp32) and their log-sum-exp to
 * `workspace`, and a second kernel merges them.  num_splits = 0 picks the
 * count (1 when the items already fill the chip); num_splits > 0 asks for
 * that many (at most 16; items too short for them use fewer).  workspace
 * (16-byte aligned, owned by the caller, contents undefined on return) must
 * hold ra_extend_workspace_bytes(...) bytes for the same arguments, which is
 * 0 when the call does not split: then workspace may be NULL.  Other arguments,
 * layouts and bounds as ra_extend_attention; RA_EINVAL for a negative
 * num_splits or a short workspace. */
int32_t ra_extend_num_splits(int32_t batch, int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t num_splits);
size_t ra_extend_workspace_bytes(int64_t total_tokens, int32_t batch, int32_t max_extend_len, int32_t hq,
                                 int32_t hkv, int32_t d, int32_t num_splits);
int ra_extend_attention_split(const void* q, const void* k_new, const void* v_new, int64_t total_tokens,
                              const void* k_pool, const void* v_pool, int64_t pool_slots,
                              const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                              const int32_t* req_pool_idx, const int32_t* prefix_lens,
                              const int32_t* extend_lens, const int32_t* extend_start, int32_t batch,
                              int32_t max_extend_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                              int32_t num_splits, void* workspace, size_t workspace_bytes, void* out,
                              hipStream_t stream);

/* Decode attention: query r ([B, Hq, D] bf16) at position L_r - 1 over
 * positions 0 .. L_r - 1 (its own K/V already stored), seq_lens = L_r >= 1.
 * Long contexts are cut into KV chunks processed in parallel; each chunk
 * writes a normalised partial output and its log-sum-exp to `workspace`, and
 * a second pass merges them.  num_splits = 0 picks the chunking; otherwise the
 * context is cut into at most num_splits chunks.  max_seq_len bounds seq_lens
 * (0 means rtt_stride).  workspace must hold ra_decode_workspace_bytes(...)
 * bytes for the same arguments (NULL allowed when that is 0).  Lengths above
 * max_seq_len are clamped to it.  Same head, table and slot rules as extend;
 * G = Hq / Hkv may be any value from 1 to 16. */
size_t ra_decode_workspace_bytes(int32_t batch, int32_t hq, int32_t hkv, int32_t d,
                                 int32_t max_seq_len, int32_t num_splits);
int ra_decode_attention(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                        const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                        const int32_t* req_pool_idx,
                        const int32_t* seq_lens, int32_t batch, int32_t max_seq_len, int32_t hq,
                        int32_t hkv, int32_t d, float scale, int32_t num_splits, void* workspace,
                        size_t workspace_bytes, void* out, hipStream_t stream);

/* The chunk length (tokens) decode uses for these arguments. */
int32_t ra_decode_chunk_len(int32_t batch, int32_t hkv, int32_t max_seq_len, int32_t num_splits);

/* Decode attention that allocates nothing, for callers that cannot allocate
 * device memory or pass a workspace (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation).  Same arguments, results
 * and rules as ra_decode_attention without the workspace: the split partials
 * live in a library-owned device array of ra_decode_noalloc_max_scratch_bytes()
 * bytes (128 MiB) per device, set up on the first call that needs it on a
 * device and held until the process ends.  A batch whose
 * ra_decode_workspace_bytes(...) exceeds that maximum is rejected with
 * RA_EINVAL and nothing is launched.  No hipMalloc, hipFree or allocating
 * library call.  Every call on a device shares that device's array (no part
 * of it needs to start at zero; each call writes every entry it reads), so
 * calls that overlap on one device -- on different streams or host threads
 * -- race; serialise them. */
size_t ra_decode_noalloc_max_scratch_bytes(void);
int ra_decode_attention_noalloc(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                                const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                                const int32_t* req_pool_idx, const int32_t* seq_lens, int32_t batch,
                                int32_t max_seq_len, int32_t hq, int32_t hkv, int32_t d, float scale,
                                int32_t num_splits, void* out, hipStream_t stream);

/* Shared-prefix decode.  With RadixAttention, requests that share a prefix
 * hold the same pool slots for it (section 3), so a decode batch of requests
 * on common branches of the radix tree reads the same K/V rows many times.
 * ra_decode_share_plan (host, plain host pointers) finds those shared runs
 * from the requests' slot rows: it sorts the requests by slot row, takes the
 * tree of common-prefix intervals of neighbours, and turns every node with at
 * least two requests and at least min_shared new positions into a shared
 * segment; each request's rest is private.  Segments are cut into chunks of
 * at most chunk_len positions and their requests into blocks of at most
 * members_per_item (1 .. 16); every (chunk, block) is one work item,
 * longest first.  chunk_len = 0 picks the longest of 4096, 2048, 1024, 512
 * and 256 that still gives at least min_items items (e.g. two work-items'
 * worth of waves per SIMD divided by Hkv; the shortest if none does).
 *   req_to_token [rtt_rows, rtt_stride], req_pool_idx [B], seq_lens [B]:
 *          host copies of the arrays ra_decode_attention takes (L clamped to
 *          [0, rtt_stride]; a request with L = 0 gets no item and
 *          ra_decode_attention_shared leaves its output rows as they were:
 *          decode requires L >= 1); RA_EINVAL for a
 *          table row outside [0, rtt_rows)
 *   plan:  int32 output of plan_capacity words; *plan_len receives the
 *          length needed.  plan = NULL only queries the length; a shorter
 *          buffer is RA_EINVAL.
 * Plan layout: header of 16 words {n_items, n_member_entries, n_parts, B,
 * members_per_item, rows per kv head, chunk length, 0...}, n_items items of 8 words
 * {table row, first position, end position, first member entry, members,
 * 0, 0, 0}, n_member_entries pairs {request, partial index or -1 for a
 * request whose only item writes its output}, part_off [B + 1] (request b's
 * partials are part_off[b] .. part_off[b+1]-1).
 *
 * ra_decode_attention_shared computes ra_decode_attention's output (query r
 * over positions 0 .. L_r - 1) from such a plan, copied by the caller to
 * device memory (`plan`, plan_len words, with the header's counts passed as
 * n_items, n_member_entries, n_parts and members_per_item): one wave per
 * (item, kv head) reads the item's K/V rows once for all its members' query
 * heads (members_per_item x Hq / Hkv <= 64 MFMA columns), writes outputs of
 * requests with one item directly and normalised partials with their
 * log-sum-exp otherwise, and a second kernel merges each request's partials.
 * workspace (16-byte aligned, caller-owned, contents undefined on return)
 * must hold ra_decode_shared_workspace_bytes(n_parts, Hq, D) bytes.  Other
 * arguments and layouts as ra_decode_attention; RA_EINVAL when plan_len does
 * not match the counts.  Device-side bounds as ra_decode_attention: table
 * rows, positions, requests and partial indices of the plan are clamped into
 * their arrays. */
int ra_decode_share_plan(const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride,
                         const int32_t* req_pool_idx, const int32_t* seq_lens, int32_t batch,
                         int32_t members_per_item, int32_t min_shared, int32_t chunk_len, int32_t min_items,
                         int32_t* plan, int64_t plan_capacity, int64_t* plan_len);
size_t ra_decode_shared_workspace_bytes(int32_t n_parts, int32_t hq, int32_t d);
int ra_decode_attention_shared(const void* q, const void* k_pool, const void* v_pool, int64_t pool_slots,
                               const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int32_t batch,
                               int32_t hq, int32_t hkv, int32_t d, float scale, const int32_t* plan,
                               int64_t plan_len, int32_t n_items, int32_t n_member_entries, int32_t n_parts,
                               int32_t members_per_item, void* workspace, size_t workspace_bytes, void* out,
                               hipStream_t stream);

/* Batch validation (a debug aid).  The kernels keep every access inside
 * the arrays by clamping: a table row outside [0, rtt_rows) reads row 0, a
 * length above its bound is cut, a slot outside [0, pool_slots) reads the
 * last slot -- so a caller bug gives plausible but wrong output.  This call
 * reads the same device arrays and reports such values instead.
 * Extend (prefix_lens, extend_lens, extend_start non-NULL, seq_lens NULL):
 * req_pool_idx in [0, rtt_rows), prefix_lens in [0, rtt_stride],
 * extend_lens in [0, max_extend_len], extend_start + extend_lens within
 * [0, total_tokens], and every prefix slot req_to_token[row, j < P] in
 * [0, pool_slots).  Decode (seq_lens non-NULL, the three extend arrays
 * NULL): req_pool_idx as above, seq_lens in [1, max_seq_len] and every slot
 * req_to_token[row, j < L] in [0, pool_slots).  Runs a small kernel on
 * `stream`, waits for the stream, and returns RA_OK or RA_EINVAL with a
 * message naming the first bad request, the field and, for slots, the
 * position.  Not for graph capture.  Uses one library-owned device word per
 * device; concurrent calls on one device are serialised. */
int ra_check_batch(const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int64_t pool_slots,
                   const int32_t* req_pool_idx, int32_t batch, const int32_t* prefix_lens,
                   const int32_t* extend_lens, const int32_t* extend_start, int64_t total_tokens,
                   int32_t max_extend_len, const int32_t* seq_lens, int32_t max_seq_len, hipStream_t stream);

/* Debug switch for the whole library: while enabled (non-zero), every
 * ra_extend_attention(_split), ra_decode_attention(_noalloc) and
 * ra_mixed_attention call runs ra_check_batch on its batch first
 * (synchronising the stream) and returns its error without launching
 * anything; ra_mixed_attention_shared checks its extend half (the shared
 * decode's plan entries are clamped on the device).  Off by default. */
int ra_set_debug_checks(int32_t enable);

/* Mixed continuous batch (section 3: continuous batching merges new and
 * running requests into one batch; Algorithm 1, B.merge and B.run): the
 * extend requests and the decode requests of one batch in one call, over the
 * same pool and slot table.  Arguments are those of ra_extend_attention
 * (q_ext .. out_ext) and ra_decode_attention (q_dec .. out_dec).  The
 * MFMA-bound extend runs on `stream`, the HBM-bound decode on a library-owned
 * companion stream of the same device (default priority) that first waits
 * for all work already queued on `stream`; `stream` then waits for the
 * decode, so later work on `stream` sees both outputs.  No host
 * synchronisation and no device allocation.  Either part may be empty
 * (n_ext == 0 or n_dec == 0).  Not safe to call concurrently from several
 * host threads on one device. */
int ra_mixed_attention(const void* q_ext, const void* k_new, const void* v_new, int64_t total_tokens,
                       const int32_t* req_pool_idx_ext, const int32_t* prefix_lens,
                       const int32_t* extend_lens, const int32_t* extend_start, int32_t n_ext,
                       int32_t max_extend_len, void* out_ext, const void* q_dec,
                       const int32_t* req_pool_idx_dec, const int32_t* seq_lens, int32_t n_dec,
                       int32_t max_seq_len, int32_t num_splits, void* workspace, size_t workspace_bytes,
                       void* out_dec, const void* k_pool, const void* v_pool, int64_t pool_slots,
                       const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int32_t hq,
                       int32_t hkv, int32_t d, float scale, hipStream_t stream);

/* The same mixed batch with the decode half computed from a shared-prefix
 * plan (ra_decode_share_plan, ra_decode_attention_shared): q_dec [n_dec, Hq,
 * D], the plan's device words and header counts, its workspace and out_dec
 * as ra_decode_attention_shared takes them.  Streams, ordering and the
 * all-or-nothing argument checks as ra_mixed_attention. */
int ra_mixed_attention_shared(const void* q_ext, const void* k_new, const void* v_new, int64_t total_tokens,
                              const int32_t* req_pool_idx_ext, const int32_t* prefix_lens,
                              const int32_t* extend_lens, const int32_t* extend_start, int32_t n_ext,
                              int32_t max_extend_len, void* out_ext, const void* q_dec, int32_t n_dec,
                              const int32_t* plan, int64_t plan_len, int32_t n_items, int32_t n_member_entries,
                              int32_t n_parts, int32_t members_per_item, void* workspace, size_t workspace_bytes,
                              void* out_dec, const void* k_pool, const void* v_pool, int64_t pool_slots,
                              const int32_t* req_to_token, int64_t rtt_rows, int64_t rtt_stride, int32_t hq,
                              int32_t hkv, int32_t d, float scale, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RADIXATTN_H */
