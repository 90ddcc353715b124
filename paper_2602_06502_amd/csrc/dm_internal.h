// Internal declarations of the DualMap HIP engine (gfx950).  Not part of the
// public ABI: include/dualmap.h is.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "dualmap.h"

namespace dm {

constexpr int kWave = 64;
constexpr int kScratchSlots = 10;  // context work buffers, one per use
// Scratch slots.  Routing uses starts, probe, select, keys, sort, scan and
// members;
// a rebalancing pass reuses probe, rebalance and select (it runs after the
// batches before it have finished).
constexpr int kSlotStarts = 0, kSlotProbe = 1, kSlotRebalance = 2, kSlotSelect = 3, kSlotKeys = 4,
              kSlotRing = 5, kSlotSort = 6, kSlotScan = 7, kSlotPurge = 8, kSlotMembers = 9;
constexpr uint32_t kMaxSlots = 4096;
constexpr uint64_t kEmpty = 0;      // index slot never used
constexpr uint64_t kTomb = 1;       // index slot erased
constexpr uint32_t kBucket = 8;     // slots per probe bucket (one 64-byte line)

// Device status word bits (reported by dm_sync).
constexpr uint32_t kErrInval = 1u;
constexpr uint32_t kErrFull = 2u;
// Largest batch dm_route_batch takes: the selection gives each block of 2048
// requests room for 66 windows of two sets of 64 lanes and indexes those
// lanes in 32 bits.
constexpr uint64_t kSelBlock = 2048, kSelWindowsPerBlock = 66;
constexpr uint64_t kMaxRouteBatch = (0xFFFFFFFFull / (kSelWindowsPerBlock * 2 * 64)) * kSelBlock;

// Hash parameters of both functions, computed on the host at dm_create.
// For function s: key words kk[s][0..B), odd multiplier P, its inverse
// Q = P^-1 mod 2^64, chain start H0, and per-lane powers P^(l+1), Q^(l+1)
// for l = 0..63 used by the wave-parallel chain.
struct HashParams {
    uint64_t seed[2];
    uint64_t P[2];
    uint64_t Q[2];
    uint64_t H0[2];
    uint64_t ppow[2][kWave];
    uint64_t qpow[2][kWave];
    uint32_t kk[2][64];
};

// One consistent-hash ring: positions ascending, owner ids, and a radix
// directory dir[k] = first index whose position >= k << (64 - dbits).
struct Ring {
    uint64_t* pos = nullptr;
    uint32_t* id = nullptr;
    uint32_t* dir = nullptr;
    uint64_t cap = 0;      // entries allocated
    uint32_t dcap = 0;     // directory entries allocated
    uint64_t len = 0;
    uint32_t dbits = 1;
};

struct RingView {
    const uint64_t* pos;
    const uint32_t* id;
    const uint32_t* dir;
    uint64_t len;
    uint32_t dbits;
};

// Growable device scratch.
struct Scratch {
    void* p = nullptr;
    size_t bytes = 0;
};

// Fixed work area for calls that must not allocate: every scratch slot is a
// region carved from it before the call's first launch, sized by the call's
// plan; a request past its region fails instead of growing.
struct Arena {
    bool on = false;
    uint8_t* base = nullptr;
    size_t off[kScratchSlots] = {};
    size_t len[kScratchSlots] = {};
};

// Adaptive hash-key length (Sec. 3.2): the prefix hotness tree as the set of
// its extended prefixes (canonical f1 key of each prefix's last block), in
// an open-addressing table of 8-slot buckets (double-buffered: a window's
// close builds the next one), and the window's record: every prefix of
// depth >= K of every routed request.
struct KeyLen {
    bool on = false;
    uint64_t max_nodes = 0;       // most extended prefixes
    uint64_t cap = 0;             // window record entries
    uint32_t log2 = 0;            // table slots 2^log2 (>= 2 max_nodes, >= 64)
    uint64_t* tab[2] = {nullptr, nullptr};
    int cur = 0;
    uint64_t* list = nullptr;     // [max_nodes] extended prefixes, ascending
    uint64_t n_ext = 0;
    uint64_t* log = nullptr;      // [cap] the window's record
    uint32_t* roots = nullptr;    // [cap / 32 + 1] bit i: record entry i is a request's root
    unsigned long long* log_n = nullptr;  // entries the window produced (may pass cap)
    uint64_t win = 0;             // requests routed in the current window
};

// Record of the keys saved through dm_kv_save: (instance, key, time of the
// latest touch) per entry, one flat array.
struct KvRecord {
    uint64_t* key = nullptr;
    uint64_t* t = nullptr;
    uint32_t* inst = nullptr;
    uint64_t n = 0, cap = 0;
};

}  // namespace dm

struct dm_ctx {
    dm_config cfg;
    hipStream_t stream = nullptr;       // launches go here (pipelined routing swaps it)
    hipStream_t home_stream = nullptr;  // the stream given to dm_create
    int device = 0;
    int n_cu = 0;           // compute units of the device
    std::string err;

    // live set (host) and cyclic next-live table (device)
    std::vector<uint8_t> live;
    uint32_t n_live = 0;
    uint32_t* d_next_live = nullptr;  // [max_slots]
    uint32_t* d_live_ids = nullptr;   // [max_slots] ascending live ids
    uint32_t* d_dense = nullptr;      // [max_slots] live id -> its index in d_live_ids
    uint8_t* d_flag_add = nullptr;    // [max_slots] scale: added this call
    uint8_t* d_flag_rm = nullptr;     // [max_slots] scale: removed this call

    dm::HashParams hp{};
    dm::HashParams* d_hp = nullptr;

    dm::Ring ring[2][2];   // [buffer][s]
    int cur = 0;           // active ring buffer

    uint64_t* d_tables = nullptr;  // [max_slots << log2slots]
    uint64_t* d_counts = nullptr;  // [2 * max_slots] live keys, then occupied slots
    uint32_t* d_status = nullptr;  // device status word

    dm::Scratch scratch[dm::kScratchSlots];
    dm::Arena arena;                  // set only for the duration of an allocation-free call
    uint8_t* noalloc_area = nullptr;  // this device's static work area (dm_noalloc.hip)
    uint32_t shift_div = 0;        // log2(queue_div)
    // Distance between the two selection work-array sets (by batch parity).
    // It only grows, and only once every stream is idle, so a set in use by
    // a batch in flight never overlaps the other set.
    size_t sel_stride = 0;

    // stage timing of dm_route_batch: one set of 5 events per batch, in a
    // ring (recorded only when enabled)
    static constexpr int kTimingRing = 64;
    bool timing = false;
    std::vector<hipEvent_t> tev;  // [kTimingRing * 5]
    uint64_t tcount = 0;          // batches recorded since timing was enabled

    // Pipelined routing.  Per batch: hashing, probing and record packing on
    // work_stream (every compute unit but one), the serial selection on
    // sel_stream (that one unit), the output epilogue on out_stream.  A
    // batch's selection follows its packing and the previous selection; a
    // batch's work first waits for the batch two back to finish, so at most
    // two batches' outputs and work arrays (by batch parity) are in use.
    bool pipelined = false;
    uint32_t policy = DM_POLICY_SLO_AWARE;  // selection rule of later batches
    dm::KeyLen kl;                          // adaptive hash-key length
    dm::KvRecord kv;                        // keys saved through dm_kv_save
    hipStream_t work_stream = nullptr, sel_stream = nullptr, out_stream = nullptr;
    hipEvent_t in_ready = nullptr;                 // caller's stream: inputs of the batch
    hipEvent_t prep_done = nullptr;                // work stream: records packed
    hipEvent_t sel_done = nullptr;                 // selection stream: selection done
    hipEvent_t out_done[2] = {nullptr, nullptr};   // output stream, by batch parity
    uint64_t batches = 0;                          // pipelined batches routed
};

namespace dm {

// ---------------------------------------------------------------------------
// Host helpers (dm_api.hip)
// ---------------------------------------------------------------------------
dm_status fail(dm_ctx* c, dm_status s, const std::string& msg);
dm_status hip_fail(dm_ctx* c, hipError_t e, const char* what);
void* scratch_get(dm_ctx* c, int slot, size_t bytes, hipError_t* e);
// Wait for the context's stream and, with pipelining, its other streams.
hipError_t sync_streams(dm_ctx* c);

inline RingView view(const Ring& r) { return RingView{r.pos, r.id, r.dir, r.len, r.dbits}; }

template <typename T>
inline bool aligned(const T* p)
{
    return (reinterpret_cast<uintptr_t>(p) % alignof(T)) == 0;
}

// Host checks of dm_route_batch's arguments (what = the calling entry
// point's name, for the message).
dm_status route_args_check(dm_ctx* c, const int32_t* tokens, uint64_t n_tokens,
                           const int64_t* offsets, uint64_t n, int64_t* loads,
                           const dm_route_out* out, const char* what);

// Grid of a grid-stride loop over n items, at least one block, at most cap.
inline uint32_t grid_for(uint64_t n, int threads, uint32_t cap = 65536)
{
    uint64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    return (uint32_t)(g > cap ? cap : g);
}

// ---------------------------------------------------------------------------
// Launchers (one per kernel family), all asynchronous on c->stream.
// ---------------------------------------------------------------------------

// Scratch bytes of each route stage for a batch of n requests (the
// launchers request exactly these, so a plan made from them up front holds).
uint64_t scan_scratch_bytes(uint64_t n);
uint64_t sort_scratch_bytes(uint64_t n);
uint64_t sort_scan_len(uint64_t n);  // length of the sort's digit-count scans
uint64_t probe_scratch_bytes(uint64_t n);
uint64_t member_scratch_bytes(uint64_t n);
uint64_t select_scratch_bytes(uint64_t n);
// Per-slot scratch of one unpipelined dm_route_batch (bytes[kScratchSlots]).
void route_scratch_plan(const dm_ctx* c, uint64_t n, uint64_t n_tokens, bool keys_in_scratch,
                        size_t* bytes);

// dm_noalloc.hip: this device's static work area (looked up once per device
// by dm_create) and its size.
hipError_t noalloc_attach(dm_ctx* c);
size_t noalloc_capacity();

// dm_scan.hip: exclusive prefix sums.
hipError_t exclusive_scan_u64(dm_ctx* c, const uint64_t* in, uint64_t n, uint64_t* out,
                              uint64_t* total_out);
// block_starts also checks the offsets (0 <= offsets[0] <= ... <= offsets[n]
// <= n_tokens) and sets *bad (zeroed beforehand) when they break that rule;
// such requests count no full block.
hipError_t block_starts(dm_ctx* c, const int64_t* offsets, uint64_t n, uint64_t n_tokens,
                        uint64_t* starts, uint32_t* bad);

// dm_sort.hip: stable LSD radix sort of (u64 key, u32 value) pairs on the
// low `bits` bits of the key (bits multiple of 8).  Sorted data ends in
// keys/vals; ktmp/vtmp are same-sized work arrays.  vals and vtmp may both
// be null: keys only.
hipError_t radix_sort_kv(dm_ctx* c, uint64_t* keys, uint32_t* vals, uint64_t* ktmp,
                         uint32_t* vtmp, uint64_t n, int bits);

// dm_ring.hip
hipError_t ring_build(dm_ctx* c, Ring& r, int s, const uint32_t* d_live_ids, uint32_t n_live);
hipError_t ring_remap(dm_ctx* c, const Ring old_r[2], const Ring new_r[2], const uint64_t* keys,
                      uint64_t n, uint32_t* old_owner, uint32_t* new_owner, uint64_t* moved,
                      uint64_t* violations);

// dm_index.hip
hipError_t index_insert(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n);
hipError_t index_erase(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n);
// Lists of several instances at once: keys[seg[i] .. seg[i+1]) are instance
// i's (seg: device [max_slots + 1], seg_host its host copy).  The insert
// runs as one kernel when every table has room for its keys, else table by
// table as index_insert.
hipError_t index_erase_many(dm_ctx* c, const uint64_t* keys, const uint64_t* seg, uint64_t n);
hipError_t index_insert_many(dm_ctx* c, const uint64_t* keys, const uint64_t* seg,
                             const uint64_t* seg_host, uint64_t n);
hipError_t index_clear(dm_ctx* c, uint32_t id);
// the tables of n instances (host list) emptied by one launch
hipError_t index_clear_many(dm_ctx* c, const uint32_t* ids_host, uint32_t n);

// Requests grouped by equal ring keys (dm_probe.hip): group_of[r] is
// request r's group, leader[g] is group g's leader request, *groups = G.
struct GroupView {
    const uint32_t* group_of;
    const uint32_t* leader;
    const uint64_t* groups;
};

// dm_hash.hip.  With *bad set (malformed offsets) every request has no full
// block: ring keys 0, match 0, no block key.
//   hash_prefix: both ring keys of every request (key_out[r], key_out[n+r]),
//     hashing only the first min(K, full blocks) blocks;
//   hash_leaders: every group leader's full f1 chain into hkeys (at
//     bstart[r]) and its longest cached prefix on both candidates (match);
//   hash_members: every other request's full f1 chain, compared with its
//     leader's keys as it is computed, and its longest cached prefix from
//     that comparison and probes past the first disagreement; its keys are
//     stored into hkeys only when write_keys is set.
//   hash_prefix with the hotness tree on: requests whose depth-K prefix is
//     extended are listed (ext_list, *ext_count zeroed beforehand) for
//     hash_extend, which walks them down the tree to K_r and rewrites their
//     ring keys.  key_len (optional) gets every request's K_r.
//   nh0 (optional, [n * K]): hash_prefix keeps there the f1 digests of
//     every request's blocks below min(K, full blocks), and hash_members
//     takes them instead of reading those tokens again.
//   keylen_record: every request's prefixes of depth >= K (its f1 block
//     keys from block K - 1 on, in hkeys at bstart[r]) join the window.
hipError_t hash_prefix(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                       const uint32_t* bad, uint64_t* key_out, uint32_t* key_len,
                       uint32_t* ext_list, unsigned long long* ext_count, uint64_t* nh0);
hipError_t hash_extend(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                       const uint32_t* bad, uint64_t* key_out, uint32_t* key_len,
                       const uint32_t* ext_list, const unsigned long long* ext_count);
hipError_t hash_leaders(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                        const uint64_t* bstart, const uint32_t* bad, const GroupView& gv,
                        const uint32_t* cand, uint64_t* hkeys, uint32_t* match);
hipError_t hash_members(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                        const uint64_t* bstart, const uint32_t* bad, const GroupView& gv,
                        const uint32_t* cand, uint64_t* hkeys, bool write_keys, uint32_t* match,
                        const uint64_t* nh0);

// dm_keylen.hip: the hotness tree's set-up, window close and export
// (host entry points; they synchronise), and its release.
dm_status keylen_enable(dm_ctx* c, uint64_t max_nodes, uint64_t max_window_blocks);
hipError_t keylen_record(dm_ctx* c, uint64_t n, const uint64_t* bstart, const uint64_t* hkeys,
                         uint64_t* work);
uint64_t keylen_record_bytes(uint64_t n);
dm_status keylen_window(dm_ctx* c);
dm_status keylen_export(dm_ctx* c, uint64_t* keys_host, uint64_t cap, uint64_t* n_host);
void keylen_free(dm_ctx* c);

// dm_kv.hip: KV save with LRU eviction (host entry point; synchronises),
// the record's entries of emptied instances dropped (d_gone: device u8 flags
// per instance slot), and the record's release.
dm_status kv_save(dm_ctx* c, const int64_t* offsets, uint64_t n, const uint64_t* block_keys,
                  const uint32_t* inst, uint64_t clock, uint64_t cap, uint64_t* added,
                  uint64_t* removed);
hipError_t kv_forget(dm_ctx* c, const uint8_t* d_gone);
void kv_free(dm_ctx* c);

// dm_queue.hip: queued requests, CSR to CSR (host entry points; they
// synchronise).  The output arrays must not overlap the input's.
dm_status queue_append(dm_ctx* c, const dm_queues* q, const int64_t* offsets, uint64_t n,
                       const dm_route_out* routed, uint64_t rec_base, const dm_queue_out* out);
dm_status queue_migrate(dm_ctx* c, const dm_queues* q, const uint64_t* mrec,
                        const uint32_t* msrc, const uint32_t* mdst, uint64_t m,
                        const dm_queue_out* out);
dm_status queue_drain(dm_ctx* c, const dm_queues* q, const int64_t* units,
                      const dm_queue_out* out);
dm_status queue_reprobe(dm_ctx* c, const dm_queues* q, const int64_t* coff, const uint64_t* keys,
                        uint64_t n_keys, const int64_t* plen, uint64_t n_ids,
                        const dm_queue_out* out);

// dm_probe.hip: candidates on the current rings (cand, fix-up flag bit 3),
// then requests ordered by their first ring key and grouped (gv).
hipError_t lookup_group(dm_ctx* c, uint64_t n, const uint64_t* key, const uint64_t* bstart,
                        const uint32_t* bad, uint32_t* cand, uint8_t* flags, GroupView* gv);

// dm_select.hip: SLO-aware choice in request order; chosen, ttft_us and
// flags bits 0-2 written, loads updated.  select_prepare packs the batch's
// records (no loads needed); select_run takes the loads' base and plan, walks
// the batch on ss and writes the outputs on os (after an event when os is
// another stream).  par picks one of two work-array sets.  select_batch is
// both on one stream.
hipError_t select_prepare(dm_ctx* c, hipStream_t st, const int64_t* offsets, uint64_t n,
                          const dm_route_out* out, int par);
hipError_t select_run(dm_ctx* c, hipStream_t ss, hipStream_t os, hipEvent_t sel_done,
                      const int64_t* offsets, uint64_t n, const dm_route_out* out,
                      int64_t* loads, int par);
hipError_t select_batch(dm_ctx* c, hipStream_t st, const int64_t* offsets, uint64_t n,
                        const dm_route_out* out, int64_t* loads);

// dm_api.hip: with pipelining on, make the context's stream wait for the
// last selection (every call except dm_route_batch starts with this).
hipError_t join_selection(dm_ctx* c);

// dm_route.hip: the whole batch, stage by stage.
hipError_t route(dm_ctx* c, const int32_t* tokens, uint64_t n_tokens, const int64_t* offsets,
                 uint64_t n, int64_t* loads, const dm_route_out* out);

// dm_rebalance.hip
hipError_t rebalance(dm_ctx* c, const dm_queues* q, int64_t* loads_out, const dm_migrations* out,
                     uint64_t cap, uint64_t Q);

}  // namespace dm

// ---------------------------------------------------------------------------
// Device helpers shared by the kernels.
// ---------------------------------------------------------------------------
namespace dm {

// SplitMix64 finaliser (Steele, Lea and Flood 2014).
__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Index key: 0 and 1 are reserved for empty and erased slots.
__host__ __device__ __forceinline__ uint64_t canon_key(uint64_t k)
{
    return k >= 2 ? k : k + (1ull << 63);
}

// Home bucket of a key in a table of 2^log2slots slots (8-slot buckets).
__device__ __forceinline__ uint64_t home_bucket(uint64_t ck, uint32_t log2slots)
{
    return ck >> (64 - (log2slots - 3));
}

// Integer TTFT estimate: base + per_token * uncached + floor(load / 2^shift).
__device__ __forceinline__ int64_t ttft_us(int64_t base, int64_t per, uint32_t shift, int64_t unc,
                                           int64_t load)
{
    return base + per * unc + (load >> shift);
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src)
{
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = __shfl(lo, src);
    hi = __shfl(hi, src);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask)
{
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = __shfl_xor(lo, mask);
    hi = __shfl_xor(hi, mask);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane)
{
    uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// v moved across lanes by a DPP control (both 32-bit halves); lanes whose
// source is out of range or whose row is masked off read 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, ROW_MASK,
                                                              0xF, true);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL,
                                                              ROW_MASK, 0xF, true);
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum (mod 2^64) of a u64 over the 64 lanes of a wave; every
// lane must be active.  Register-level data movement only: shifts by 1, 2,
// 4, 8 inside each 16-lane row, then the last lane of row 0 (row 2) into
// row 1 (row 3), then the last lane of row 1 into rows 2 and 3.
__device__ __forceinline__ uint64_t wave_incl_sum_u64(uint64_t v, int /*lane*/)
{
    v += dpp_u64<0x111, 0xF>(v);  // row_shr:1
    v += dpp_u64<0x112, 0xF>(v);  // row_shr:2
    v += dpp_u64<0x114, 0xF>(v);  // row_shr:4
    v += dpp_u64<0x118, 0xF>(v);  // row_shr:8
    v += dpp_u64<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp_u64<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Sum over the 64 lanes of a wave, in every lane; every lane must be active.
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
    return readlane_u64(wave_incl_sum_u64(v, 0), kWave - 1);
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// Owner of ring key x: the first ring entry at a position >= x, wrapping to
// entry 0 past the top.  The directory bounds the search to x's bucket.
__device__ __forceinline__ uint32_t ring_owner(const RingView& r, uint64_t x)
{
    const uint64_t b = x >> (64 - r.dbits);
    uint64_t i = r.dir[b];
    const uint64_t e = r.dir[b + 1];
    while (i < e && r.pos[i] < x)
        i++;
    if (i >= r.len)
        i = 0;
    return r.id[i];
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Index probing.  A table is 2^ls slots in 8-slot (64-byte) buckets; a
// key's probe sequence starts at its home bucket (the key's top ls - 3
// bits) and walks buckets in order.  An insert takes the first empty slot
// of the sequence and slots never return to empty, so a bucket's empty
// slots are a suffix of it: a bucket has one iff its last slot is empty,
// and such a bucket ends the key's sequence.
enum : int { kHit = 0, kMiss = 1, kNext = 2 };

typedef unsigned long long v2u64 __attribute__((ext_vector_type(2), aligned(16)));

// Home bucket of a canonical key in a 2^ls-slot table (ls <= 30).
__device__ __forceinline__ uint32_t home32(uint64_t ck, uint32_t ls)
{
    return (uint32_t)(ck >> 32) >> (35 - ls);
}

// One bucket: the key is there, the bucket ends the sequence without it, or
// go on to the next bucket.
__device__ __forceinline__ int bucket_probe(const uint64_t* tab, uint32_t bkt, uint64_t key)
{
    const v2u64* line = reinterpret_cast<const v2u64*>(tab + (uint64_t)bkt * kBucket);
    const v2u64 s0 = line[0], s1 = line[1], s2 = line[2], s3 = line[3];
    const bool hit = s0.x == key || s0.y == key || s1.x == key || s1.y == key || s2.x == key ||
                     s2.y == key || s3.x == key || s3.y == key;
    return hit ? kHit : (s3.y == kEmpty ? kMiss : kNext);
}

// Is canonical key ck in the table?  Walks its probe sequence.
__device__ __forceinline__ bool table_has(const uint64_t* tab, uint32_t ls, uint64_t ck)
{
    const uint32_t nbk = 1u << (ls - 3);
    uint32_t b = home32(ck, ls);
    for (uint32_t step = 0; step < nbk; step++) {
        const int r = bucket_probe(tab, b, ck);
        if (r != kNext)
            return r == kHit;
        b = (b + 1) & (nbk - 1);
    }
    return false;
}

}  // namespace dm
