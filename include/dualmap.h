/*
 * dualmap.h -- C ABI of the DualMap routing engine for AMD Instinct MI355X
 * (gfx950).
 *
 * DualMap (arXiv 2602.06502) maps every request to two candidate instances
 * with two independent hash functions over its prompt prefix, placed on two
 * consistent-hash rings, and picks one with an SLO-aware rule that keeps the
 * cache-affine candidate unless its expected TTFT breaks the SLO (Sec. 3.2);
 * overloaded instances hand queued requests to the other member of their
 * pair (Sec. 3.3); instances join and leave with only local remapping
 * (Sec. 3.4).  This library runs that path as HIP kernels on one GPU.
 *
 * Conventions shared by every entry point
 *   - Array arguments are caller-owned DEVICE memory unless marked "host".
 *     The library never frees them; they must stay valid until the work is
 *     complete (dm_sync returns).
 *   - Calls are ordered on the stream given to dm_create.  Argument errors
 *     are detected on the host, return DM_EINVAL at once and change no state.
 *     Errors found by kernels (malformed offsets, a full index table, more
 *     migrations than the output holds) set a device status word that the
 *     next dm_sync returns (and clears).
 *   - Integers: token ids are read as u32; block keys, ring positions and
 *     ring keys are u64; loads and times are int64 (microseconds for times).
 *   - No entry point throws or aborts; dm_last_error gives a message for the
 *     last failing call on a context.
 *   - A context is not thread safe: one host thread at a time.
 */
#ifndef DUALMAP_H
#define DUALMAP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dm_ctx dm_ctx;

typedef enum {
    DM_OK = 0,
    DM_EINVAL = 1,  /* bad argument (host check) or malformed input (device) */
    DM_ENOMEM = 2,  /* device or host allocation failed                      */
    DM_EFULL = 3,   /* index table past its load limit / migrations > cap    */
    DM_ESTATE = 4,  /* call out of order (e.g. routing before rings exist)   */
    DM_EDEVICE = 5  /* HIP runtime error                                     */
} dm_status;

/* Engine configuration.  The hash functions f1, f2 of Sec. 3.2 are left
 * unnamed by the paper; this engine uses, per function s, NH block digests
 * keyed from a SplitMix64 stream seeded by seed[s], chained across blocks by
 * an affine step with an odd multiplier, and finalised by the SplitMix64 mix
 * xor seed[s].  Block b's key covers tokens [0, (b+1)*block_size). */
typedef struct {
    uint32_t block_size;        /* B: tokens per KV block; power of two, 4..64      */
    uint32_t key_blocks;        /* K: ring keys hash the first K full blocks, 1..64  */
    uint64_t seed[2];           /* seeds of f1 (ring 1) and f2 (ring 2)              */
    uint32_t vnodes;            /* V >= 1 virtual nodes per instance on each ring    */
    uint32_t max_slots;         /* instance ids are < max_slots; 1..4096             */
    uint32_t index_log2_slots;  /* per-instance table holds 2^k keys, 4 <= k <= 30;  */
                                /*   inserts fail (DM_EFULL) past 2^(k-1) keys       */
    uint32_t reserved;          /* must be 0                                         */
    int64_t ttft_base_us;       /* TTFT(us) = base + per_token * uncached tokens     */
    int64_t ttft_per_token_us;  /*          + floor(load / queue_div)   (Sec. 3.2)   */
    int64_t queue_div;          /* power of two >= 1                                 */
    int64_t slo_us;             /* TTFT SLO; "exceeds" means >, "meets" means <=     */
} dm_config;

/* Create a context on the current HIP device, ordered on hip_stream (a
 * hipStream_t; NULL = the default stream).  Allocates the per-instance index
 * tables (max_slots * 2^index_log2_slots * 8 bytes) up front.  *out is set
 * only on DM_OK. */
dm_status dm_create(const dm_config* cfg, void* hip_stream, dm_ctx** out);

/* Free a context and everything it owns (waits for its stream first). */
void dm_destroy(dm_ctx* ctx);

/* Set the live instance set to ids[0..n) (host array, distinct, each
 * < max_slots, n >= 1) and build both consistent-hash rings (Sec. 3.4): each
 * live instance gets V virtual nodes per ring at positions mixed from
 * (id, v) and the ring's seed; a ring key belongs to the first virtual node
 * at or after it, wrapping past the top (the (A,B] -> B rule of Sec. A.1.3).
 * Index tables keep their contents. */
dm_status dm_build_rings(dm_ctx* ctx, const uint32_t* ids, uint32_t n);

/* Copy ring s (0 or 1) to host memory: *len entries sorted by position.
 * pos/id may be NULL to query the length only; otherwise they hold cap
 * entries.  Synchronises the stream. */
dm_status dm_ring_export(dm_ctx* ctx, int s, uint64_t* pos_host, uint32_t* id_host,
                         uint64_t cap, uint64_t* len);

/* Add n block keys (device array) to instance id's cached-block index (the
 * per-instance KV metadata of Sec. A.3.2) with set semantics.  Keys 0 and 1
 * are stored as 2^63 and 2^63 + 1 (0 and 1 mark empty and erased slots).
 * A table holds at most 2^(index_log2_slots - 1) keys; keys past that are
 * dropped and dm_sync reports DM_EFULL. */
dm_status dm_index_insert(dm_ctx* ctx, uint32_t id, const uint64_t* keys, uint64_t n);

/* Remove n keys (device array) from instance id's index; absent keys are
 * ignored.  Erased slots stay occupied until dm_index_clear. */
dm_status dm_index_erase(dm_ctx* ctx, uint32_t id, const uint64_t* keys, uint64_t n);

/* Empty instance id's index (and drop its keys from dm_kv_save's record). */
dm_status dm_index_clear(dm_ctx* ctx, uint32_t id);

/* KV save with least-recently-used eviction: the serving step after routing
 * (the KV query and save of Sec. A.3.2), on the device.  Request r of a
 * served batch (offsets: device int64 [n + 1], non-decreasing, the batch's
 * prompts as in dm_route_batch; block_keys: device u64, every full block's
 * f1 key request-major, e.g. dm_route_out.block_keys) is served by inst[r]
 * (device u32 [n], e.g. dm_route_out.chosen after any migrations).  Every
 * block is touched on that instance, deepest block first, at time
 * clock + start_r + (nfull_r - 1 - b) for block b (start_r: full blocks of
 * the requests before r), so a prefix's blocks are always more recent than
 * its descendants and caches stay prefix-closed.  Each instance's cache
 * becomes the cap most recently touched distinct keys (cap = 0: unbounded;
 * cap <= 2^(k-1)) among those saved before and those sent now; keys that
 * leave are erased from its index and keys that join are inserted.  The
 * counts go to *added_host / *removed_host (host, optional).  The caller
 * advances its clock by the batch's full blocks; times must stay below
 * 2^40.  The record of saved keys is the library's: keys inserted with
 * dm_index_insert are not in it, and erasing saved keys with
 * dm_index_erase leaves them recorded.  Synchronises.  DM_EINVAL (nothing
 * changed) for offsets that decrease or are negative, or an instance id >=
 * max_slots, both checked on the device before any other work. */
dm_status dm_kv_save(dm_ctx* ctx, const int64_t* offsets, uint64_t n, const uint64_t* block_keys,
                     const uint32_t* inst, uint64_t clock, uint64_t cap, uint64_t* added_host,
                     uint64_t* removed_host);

/* Number of keys held by instance id's index (host out).  Synchronises. */
dm_status dm_index_size(dm_ctx* ctx, uint32_t id, uint64_t* n_host);

/* Outputs of dm_route_batch (device arrays; all required except
 * block_keys). */
typedef struct {
    uint64_t* key;        /* [2n] ring keys: f1 at [r], f2 at [n + r]               */
    uint32_t* cand;       /* [2n] candidates c1 at [r], c2 at [n + r]               */
    uint32_t* match;      /* [2n] cached leading blocks on c1 / c2                  */
    uint32_t* chosen;     /* [n]  selected instance                                 */
    int64_t* ttft_us;     /* [n]  estimated TTFT on the selected instance           */
    uint8_t* flags;       /* [n]  bit0 left the cache-affine candidate for the SLO, */
                          /*      bit1 both candidates' TTFT exceed the SLO (the    */
                          /*      rebalance trigger of Sec. A.1.2), bit2 equal      */
                          /*      match, bit3 second candidate adjusted             */
    uint64_t* block_keys; /* NULL, or [sum over r of floor(len_r / B)] every full    */
                          /*      block's f1 key, request-major (the keys a KV     */
                          /*      save inserts)                                    */
    uint32_t* key_len;    /* NULL, or [n] blocks the ring keys hash (K_r)           */
} dm_route_out;

/* Route a batch of n requests (Sec. 3.2, Sec. A.1.1).  tokens holds n_tokens
 * int32 token ids; request r's prompt is tokens[offsets[r] .. offsets[r+1])
 * (offsets int64, n + 1 entries, 0 <= offsets[0] <= ... <= offsets[n] <=
 * n_tokens).  Offsets are checked on the device: if they break that rule,
 * no token outside [0, n_tokens) and no block key past the batch's block
 * count is touched, every request is treated as having no full block (ring
 * keys 0, match 0), and dm_sync returns DM_EINVAL.  For every request:
 *   1. chained f1/f2 block keys; ring keys x_s = key of the first K_r
 *      blocks, K_r = min(K, full blocks) (no full block: the empty-prefix
 *      key), or with the hotness tree on (dm_keylen_enable) the length the
 *      tree gives;
 *   2. c1 = owner of x1 on ring 1, c2 = owner of x2 on ring 2; if they
 *      coincide c2 becomes the next live id after c1 in cyclic id order
 *      (Sec. 3.2, id2 = (id1 + 1) mod n for dense ids);
 *   3. match_c = number of leading full blocks whose f1 keys are all in
 *      candidate c's index (index snapshot: not updated within the batch);
 *   4. TTFT_c = base + per_token * (len - B * match_c) + floor(L[c] / div);
 *   5. selection in request order with loads L = loads[] updated after each
 *      request (L[chosen] += its uncached tokens): equal match -> the
 *      less-loaded candidate (ties c1); otherwise the candidate with more
 *      cached blocks unless its TTFT exceeds the SLO, then the other one if
 *      strictly less loaded.
 * loads: device int64 [max_slots], read and updated in place.  Requires
 * rings (DM_ESTATE otherwise).  The call does not wait for the device: its
 * work arrays are sized from n and n_tokens (they grow, synchronising once,
 * only when a batch needs more than any before it).  n = 0 is a no-op; n must be at most
 * 1,041,203,200 (DM_EINVAL): the selection indexes its per-request slots in
 * 32 bits.  Match lengths are 32-bit: a request with 2^32 or more full
 * blocks sets the device status word (DM_EINVAL from dm_sync). */
dm_status dm_route_batch(dm_ctx* ctx, const int32_t* tokens, uint64_t n_tokens,
                         const int64_t* offsets, uint64_t n, int64_t* loads,
                         const dm_route_out* out);

/* dm_route_batch for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Same arguments, results and device-side checks as dm_route_batch; the
 * caller still provides every input and output.  Work arrays come from a
 * static area of 64 MiB per GPU that the library holds until the process
 * ends, instead of the context's growable scratch: the call allocates and
 * frees nothing.  The batch is planned on the host first; if its work
 * arrays do not fit (about 550 bytes per request plus, when block_keys is
 * NULL, 8 bytes per n_tokens / B), the call returns DM_EINVAL with the
 * sizes in dm_last_error and launches nothing.  Runs unpipelined on the
 * context's stream (after any pipelined batch).  Every call on one GPU
 * shares that GPU's area: calls that overlap on one GPU (other contexts,
 * other host threads, unordered streams) race.  DM_EDEVICE if the area
 * could not be located on this device. */
dm_status dm_route_batch_noalloc(dm_ctx* ctx, const int32_t* tokens, uint64_t n_tokens,
                                 const int64_t* offsets, uint64_t n, int64_t* loads,
                                 const dm_route_out* out);

/* Pending-request queues, CSR over instance slots (device arrays).  Queue i
 * is records [qoff[i], qoff[i+1]) head first; record q costs unc_here[q]
 * uncached tokens on i and unc_alt[q] on its alternative candidate alt[q]
 * (the other member of its dual-mapping pair); base_work[i] is pending work
 * ahead of queue i.
 *
 * Decode-bottleneck telemetry (Sec. A.7), optional: prefill_interval[i] is
 * the time in microseconds since instance i last completed a prefill.  An
 * instance with a non-empty queue whose interval exceeds
 * decode_threshold_us is taken to be stalled in decode, and every TTFT the
 * pass estimates on it (as source or as target) gets its interval added as
 * the decode-delay estimate.  NULL: no correction.  Intervals must lie in
 * [0, 2^40] (the pass reports DM_EINVAL through dm_sync otherwise, its
 * outputs then undefined); the threshold must not be negative (host
 * check).  The paper's deployment uses a threshold of 3 s. */
typedef struct {
    const int64_t* qoff;       /* [max_slots + 1], qoff[0] = 0, non-decreasing */
    const uint64_t* rec_id;    /* [Q] caller's record ids                      */
    const uint32_t* unc_here;  /* [Q]                                          */
    const uint32_t* alt;       /* [Q] each < max_slots                         */
    const uint32_t* unc_alt;   /* [Q]                                          */
    const int64_t* base_work;  /* [max_slots]                                  */
    const int64_t* prefill_interval;  /* [max_slots] or NULL                   */
    int64_t decode_threshold_us;      /* read only with prefill_interval       */
} dm_queues;

/* Writable queues, the output of the queue operations below: device arrays
 * with room for cap records (qoff [max_slots + 1], base_work [max_slots]).
 * They must not overlap the input queues' arrays. */
typedef struct {
    int64_t* qoff;
    uint64_t* rec_id;
    uint32_t* unc_here;
    uint32_t* alt;
    uint32_t* unc_alt;
    int64_t* base_work;
    uint64_t cap;
} dm_queue_out;

/* Queue operations: the serving state the rebalancing pass reads, kept on
 * the device.  Each reads queues q and writes the result to out (DM_EFULL,
 * nothing written, if it holds more than out->cap records; DM_EINVAL,
 * nothing written, if q's offsets are not in order within [0, qoff[S]] or
 * q has 2^32 records or more).  All synchronise.
 *   dm_queue_append: a routed batch (offsets as given to dm_route_batch;
 *     routed->cand, match and chosen of its result) joins the queues:
 *     request r, id rec_base + r, at the tail of chosen[r]'s queue in
 *     request order, with len - B * match uncached tokens there and on the
 *     other candidate, its alternative.  Base work unchanged.  DM_EINVAL
 *     for a chosen id >= max_slots.
 *   dm_queue_migrate: a migration list (e.g. dm_rebalance's, its first m
 *     entries) applied in order: each record leaves its source's queue (the
 *     others keep their order) and joins its target's tail with the pair's
 *     roles swapped (its alternative becomes the source).  DM_EINVAL if a
 *     record is not queued on its source, appears twice, or is id 2^64 - 1,
 *     or an id is >= max_slots.
 *   dm_queue_drain: units[i] (device int64 [max_slots], >= 0) of service on
 *     instance i: its base work first, then whole records from the head; a
 *     partly served head keeps the rest of its uncached tokens. */
dm_status dm_queue_append(dm_ctx* ctx, const dm_queues* q, const int64_t* offsets, uint64_t n,
                          const dm_route_out* routed, uint64_t rec_base,
                          const dm_queue_out* out);
dm_status dm_queue_migrate(dm_ctx* ctx, const dm_queues* q, const uint64_t* rec_id,
                           const uint32_t* from, const uint32_t* to, uint64_t m,
                           const dm_queue_out* out);
dm_status dm_queue_drain(dm_ctx* ctx, const dm_queues* q, const int64_t* units,
                         const dm_queue_out* out);

/* Queued records re-priced against the caches as they are now (Sec. 3.3;
 * Sec. A.3.2: each TTFT the rebalancing pass evaluates rests on a KV-cache
 * query on the record's instance and one on its backup).  Record id r
 * (< n_ids) has the f1 block-key chain chain_keys[chain_off[r] ..
 * chain_off[r+1]) (block keys as dm_route_batch emits them; device u64
 * [n_keys]) and a prompt of prompt_len[r] tokens (device int64 [n_ids];
 * chain_off device int64 [n_ids + 1]).  out receives q with each record's
 * unc_here and unc_alt recomputed as prompt_len - B * (leading chain blocks
 * cached on its instance / on its alternative); order, ids, alternatives
 * and base work are unchanged.  DM_EINVAL, nothing written, for a queued id
 * >= n_ids, a chain outside [0, n_keys) or with more blocks than its prompt
 * holds, a prompt outside [0, 2^32) or an alternative >= max_slots.
 * Synchronises.  The caches must not change during the call. */
dm_status dm_queue_reprobe(dm_ctx* ctx, const dm_queues* q, const int64_t* chain_off,
                           const uint64_t* chain_keys, uint64_t n_keys, const int64_t* prompt_len,
                           uint64_t n_ids, const dm_queue_out* out);

/* Migration list of dm_rebalance (device arrays of cap entries). */
typedef struct {
    uint64_t* rec_id;
    uint32_t* from;
    uint32_t* to;
    int64_t* benefit_us;  /* TTFT on the source minus TTFT on the target, at pass start */
    int64_t* ttft_to_us;  /* TTFT on the target with its load when the record moved    */
    uint64_t* count;      /* [1] number of migrations (may exceed cap: DM_EFULL)       */
} dm_migrations;

/* One non-recursive, single-round hotspot rebalancing pass (Sec. 3.3,
 * Eq. of the migration benefit; Sec. A.1.2).  The TTFT of the record at
 * queue position p of instance i waits behind base_work[i] and the records
 * ahead of it (plus the decode-delay estimate of a stalled instance, see
 * dm_queues).  Instance i is overloaded when some queued TTFT exceeds the
 * SLO (judged at pass start).  Overloaded sources are taken heaviest load
 * first (ties: lower id); within a source, records with benefit B > 0 whose
 * alternative is not overloaded go in order of descending B (ties: nearer
 * the head first).  Before each record the source stops if every queued
 * TTFT meets the SLO; the record moves iff its TTFT on the target with the
 * target's current load is below the SLO.  Migrations are listed in the
 * order they happen.  loads_out[i] (device int64 [max_slots]) receives the
 * final load: base work + queued uncached tokens + received records. */
dm_status dm_rebalance(dm_ctx* ctx, const dm_queues* q, int64_t* loads_out,
                       const dm_migrations* out, uint64_t cap);

/* Change membership (Sec. 3.4; Sec. A.1.3): add ids add[0..n_add), remove
 * rm[0..n_rm) (host arrays), rebuild both rings, and check the remap of n
 * ring keys per ring (keys: device u64 [2n], ring 1 keys then ring 2 keys,
 * e.g. dm_route_out.key).  old_owner/new_owner (device u32 [2n]) get each
 * key's owner before and after; moved (device u64 [2]) counts changed owners
 * per ring; violations (device u64 [1]) counts changes that neither leave a
 * removed instance nor land on an added one (zero for consistent hashing).
 * Removed and added instances' indexes are emptied.  DM_EINVAL (and no
 * change) if an added id is live or out of range, a removed id is not live,
 * either list repeats an id, or the new set would be empty. */
dm_status dm_scale(dm_ctx* ctx, const uint32_t* add, uint32_t n_add, const uint32_t* rm,
                   uint32_t n_rm, const uint64_t* keys, uint64_t n, uint32_t* old_owner,
                   uint32_t* new_owner, uint64_t* moved, uint64_t* violations);

/* Instrumentation.  With on != 0, dm_route_batch records HIP events around
 * its stages; dm_route_stage_ms waits for the last batch and writes up to n
 * stage times in milliseconds to ms_host, averaged over the batches routed
 * since timing was (re)enabled (the last 64 at most): [0] ring keys,
 * candidates and request groups (prefix hashing, ring lookup, ordering,
 * grouping), [1] full chains and longest cached prefixes (group leaders,
 * then every other request), [2] record packing and in-order selection
 * (with pipelining: from the end of the batch's stage [1] to the end of its
 * selection, so it includes waiting for the previous batch's selection),
 * [3] per-request block offsets and the offsets check.
 * dm_route_stage_ms returns DM_ESTATE if timing is off or no batch was
 * timed. */
dm_status dm_set_timing(dm_ctx* ctx, int on);
dm_status dm_route_stage_ms(dm_ctx* ctx, float* ms_host, int n);

/* Pipelined routing of consecutive batches.  The selection stage is a chain
 * in request order over shared loads (Sec. 3.2) and runs as one wave, while
 * hashing and probing use the whole GPU.  With on != 0, dm_route_batch runs
 * on three streams owned by the context: hashing, probing and record
 * packing on a work stream restricted to all compute units but one, the
 * selection walk on a stream restricted to that one unit, and the
 * per-request epilogue (chosen, TTFT, flags) on a third stream (where the
 * runtime refuses compute-unit masks, the streams are unrestricted).  A
 * batch's work starts after the work queued on the context's stream before
 * the call; its selection starts once its records are packed and the
 * previous batch's selection is done, so batches are still decided in
 * order.  The context's stream is not made to wait, so the next batch's
 * hashing and probing overlap this batch's selection.  At most two batches
 * are in flight: a batch's work also waits for the epilogue of the batch
 * two before it.
 *
 * Until the batch's selection and epilogue have run (dm_sync, or any call
 * that orders the context's stream after them, below), the batch's tokens,
 * offsets, output arrays and the loads must stay valid and unmodified.
 * Consecutive batches need distinct output arrays; a batch may reuse those
 * of the batch two before it.  The same loads array may be passed to every
 * batch.
 *
 * dm_sync waits for all streams.  Every other call except dm_route_batch,
 * dm_set_timing and dm_route_stage_ms first orders the context's stream
 * after the last epilogue.  Turning pipelining off does the same.  Returns
 * DM_EDEVICE if the streams or their events cannot be created. */
dm_status dm_set_pipelining(dm_ctx* ctx, int on);

/* Adaptive hash-key length (Sec. 3.2, "How long prefix is appropriate for
 * the hash key?"; Sec. A.1.1).  The prefix hotness tree: nodes are prompt
 * prefixes of d >= K full blocks (named by the f1 key of their last block),
 * the depth-K prefixes its roots; the tree is kept as the set of its
 * extended nodes (those with children).  While it is on, a request's ring
 * keys hash K_r blocks: the smallest d >= K whose prefix is not extended,
 * at most its full blocks (fewer than K full blocks: all of them).  Every
 * routed request joins the current window with its prefixes of depth >= K.
 *
 * dm_keylen_enable turns the tree on with room for max_nodes extended
 * prefixes and a window record of max_window_blocks prefixes (the tree
 * starts empty, i.e. every K_r is min(K, full blocks)); max_nodes = 0 turns
 * it off.  Prefixes past the record's room are dropped and dm_sync reports
 * DM_EFULL; closing such a window returns DM_EFULL and leaves the tree
 * unchanged.  With the tree on, the routing computes every request's block
 * keys (as for block_keys) to record them.
 *
 * dm_keylen_window closes the window.  With W requests in it and n live
 * instances, a prefix's traffic ratio rho is the share of the window's
 * requests that carry it.  A leaf with rho > 2/n becomes extended (its
 * requests will hash one block more and spread over more candidate pairs),
 * an extended node with rho < 1/n stops being extended, and the rule is
 * applied until it changes nothing, so a hot prefix grows in one close to
 * where its requests part.  As a prefix's count never exceeds its
 * parent's, the new tree is the set of prefixes (depth >= K) with
 * rho > 2/n, or already extended with rho >= 1/n.  An empty window changes
 * nothing.  DM_EFULL if the new tree would hold more than max_nodes
 * extended prefixes (the tree is then unchanged); the next window starts
 * empty either way.  dm_keylen_export writes up to cap extended prefixes,
 * ascending (canonical keys: k, or k + 2^63 for k < 2), to keys_host and
 * their count to *n_host.  All three synchronise with the context's
 * streams.  DM_ESTATE if the tree is off (window, export) or no ring exists
 * (window). */
dm_status dm_keylen_enable(dm_ctx* ctx, uint64_t max_nodes, uint64_t max_window_blocks);
dm_status dm_keylen_window(dm_ctx* ctx);
dm_status dm_keylen_export(dm_ctx* ctx, uint64_t* keys_host, uint64_t cap, uint64_t* n_host);

/* Selection rule between the two candidates of every request.  The
 * SLO-aware rule is DualMap's (Sec. 3.2) and the default; the others are the
 * single-criterion variants of the ablation study (Sec. 4.3):
 *   DM_POLICY_CACHE_AFFINITY  the candidate with more cached blocks (equal
 *                             hits: the less-loaded one, ties c1);
 *   DM_POLICY_LEAST_LOADED    the candidate with the smaller load (ties c1);
 *   DM_POLICY_MIN_TTFT        the candidate with the smaller estimated TTFT
 *                             (ties c1).
 * The ablation's "no rebalance" variant is the SLO-aware rule with no
 * dm_rebalance calls.  Every rule updates the loads in request order as the
 * SLO-aware one does; flag bit0 marks a chosen candidate with fewer cached
 * blocks than the other (under the SLO-aware rule exactly its switches for
 * the SLO).  The minimum-TTFT rule always takes the one-request-at-a-time
 * selection path.  Applies to batches routed after the call; DM_EINVAL for
 * an unknown rule. */
typedef enum {
    DM_POLICY_SLO_AWARE = 0,
    DM_POLICY_CACHE_AFFINITY = 1,
    DM_POLICY_LEAST_LOADED = 2,
    DM_POLICY_MIN_TTFT = 3
} dm_policy;
dm_status dm_set_policy(dm_ctx* ctx, int policy);

/* Wait for all work on the context's stream (and, with pipelining, on its
 * work, selection and epilogue streams); return and clear the first
 * device-side error since the last dm_sync. */
dm_status dm_sync(dm_ctx* ctx);

/* Message of the last failing call on ctx ("" if none); valid until the next
 * call on ctx. */
const char* dm_last_error(const dm_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* DUALMAP_H */
