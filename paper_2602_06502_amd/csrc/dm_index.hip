// Per-instance cached-block index (the KV metadata of Sec. A.3.2): one
// open-addressing table of 2^k u64 keys per instance slot, probed a bucket
// of 8 slots (one 64-byte line) at a time, buckets in linear order from the
// key's home bucket.  Slot 0 = empty, 1 = erased; stored keys are >= 2.
// An insert takes the first empty slot of the probe sequence, so an empty
// slot seen during a lookup proves the key absent.
//
// Capacity: a table never holds more than 2^(k-1) occupied slots.  A thread
// reserves a unit of the occupied count before it claims an empty slot and
// gives it back if the claim loses (another thread stored the same or a
// different key there).  A reservation refused at the limit is not final,
// since reservations still in flight may be given back: the key goes to an
// overflow list, and once the insert kernel has finished a single wave
// settles the list in order (present already, stored while room is left,
// else dropped with DM_EFULL).  So a batch that fits is stored whole, and a
// batch that does not fills the table to exactly the limit.
#include <algorithm>
#include <vector>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kPurgeSlot = kSlotPurge;  // table rebuild work area

struct TableRef {
    uint64_t* slots;
    uint64_t* live;      // live key count
    uint64_t* occupied;  // non-empty slots (live + erased)
    uint32_t log2slots;
    uint64_t limit;      // maximum occupied slots
};

// Overflow list: a count and the keys (room for every key of the batch).
struct Overflow {
    unsigned long long* count;
    uint64_t* keys;
};

// Insert of one canonical key (>= 2); set semantics.  With an overflow list,
// a key whose reservation is refused at the limit is appended to it;
// without one the key is dropped with kErrFull.
__device__ __forceinline__ void insert_one(const TableRef& t, uint64_t k, uint32_t* status,
                                           const Overflow* ovf)
{
    const uint64_t nbk = 1ull << (t.log2slots - 3);
    uint64_t b = home_bucket(k, t.log2slots);
    bool done = false;
    for (uint64_t step = 0; step < nbk && !done; step++, b = (b + 1) & (nbk - 1)) {
        for (uint32_t s = 0; s < kBucket && !done; s++) {
            uint64_t* slot = t.slots + b * kBucket + s;
            uint64_t v = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (v == k) {
                done = true;
            } else if (v == kEmpty) {
                const unsigned long long held =
                    atomicAdd((unsigned long long*)t.occupied, 1ull);
                if (held >= t.limit) {
                    atomicAdd((unsigned long long*)t.occupied, ~0ull);  // give back
                    if (ovf) {
                        const unsigned long long at = atomicAdd(ovf->count, 1ull);
                        ovf->keys[at] = k;
                    } else {
                        atomicOr(status, kErrFull);
                    }
                    return;
                }
                const unsigned long long prev = atomicCAS(
                    (unsigned long long*)slot, (unsigned long long)kEmpty, (unsigned long long)k);
                if (prev == kEmpty) {
                    atomicAdd((unsigned long long*)t.live, 1ull);
                    done = true;
                } else {
                    atomicAdd((unsigned long long*)t.occupied, ~0ull);  // claim lost
                    done = prev == k;  // else another key took the slot: keep walking
                }
            }
        }
    }
    if (!done)
        atomicOr(status, kErrFull);  // every slot scanned: table full
}

__global__ void insert_kernel(TableRef t, const uint64_t* __restrict__ keys, uint64_t n,
                              uint32_t* __restrict__ status, Overflow ovf)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        insert_one(t, canon_key(keys[i]), status, &ovf);
}

// Is canonical key k stored?  Walks k's probe sequence to its first empty slot.
__device__ bool contains(const TableRef& t, uint64_t k)
{
    const uint64_t nbk = 1ull << (t.log2slots - 3);
    uint64_t b = home_bucket(k, t.log2slots);
    for (uint64_t step = 0; step < nbk; step++, b = (b + 1) & (nbk - 1))
        for (uint32_t s = 0; s < kBucket; s++) {
            const uint64_t v = __hip_atomic_load(t.slots + b * kBucket + s, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
            if (v == k)
                return true;
            if (v == kEmpty)
                return false;
        }
    return false;
}

// The overflow list in list order, by one wave after the insert kernel:
// every lane looks up its key, then the absent ones are stored one lane
// at a time while the table has room; the rest are dropped with kErrFull.
// Nothing else writes the table meanwhile, so the counts are exact here.
__global__ void overflow_kernel(TableRef t, Overflow ovf, uint32_t* __restrict__ status)
{
    const int lane = lane_id();
    const uint64_t m = *ovf.count;
    for (uint64_t base = 0; base < m; base += kWave) {
        const uint64_t i = base + lane;
        const uint64_t k = i < m ? ovf.keys[i] : 0;
        bool need = i < m && !contains(t, k);
        if (!__any(need))
            continue;
        for (int j = 0; j < kWave; j++) {
            // lanes in order: an earlier lane may have stored the same key
            if (lane == j && need) {
                if (contains(t, k)) {
                    need = false;
                } else if (__hip_atomic_load(t.occupied, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT) >= t.limit) {
                    atomicOr(status, kErrFull);
                } else {
                    insert_one(t, k, status, nullptr);
                }
            }
            // the next lane sees this lane's store and counts
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent");
        }
    }
}

// Erased slots are never reused by inserts (an empty slot must keep proving
// absence), so churn fills a table with them.  Before an insert of n keys
// that could push the occupied count past the limit while erased slots
// exist, the table is rebuilt: live keys gathered, slots cleared, keys
// reinserted.  The decision is taken on the device (plan[0]); every kernel
// of the rebuild returns at once when it is not needed.
__global__ void purge_plan_kernel(TableRef t, uint64_t n, unsigned long long* plan)
{
    const uint64_t occ = *t.occupied, live = *t.live;
    plan[0] = (occ + n > t.limit && occ > live) ? 1ull : 0ull;
    plan[1] = 0;  // live keys gathered
    plan[2] = 0;  // overflow list length
}

__global__ void purge_gather_kernel(TableRef t, const unsigned long long* plan,
                                    unsigned long long* cnt, uint64_t* __restrict__ out)
{
    if (!plan[0])
        return;
    const uint64_t n = 1ull << t.log2slots;
    const uint64_t lt = (1ull << lane_id()) - 1;
    for (uint64_t base = blockIdx.x * (uint64_t)blockDim.x; base < n;
         base += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t i = base + threadIdx.x;
        const uint64_t v = i < n ? t.slots[i] : kEmpty;
        const bool keep = v != kEmpty && v != kTomb;
        const uint64_t m = ballot(keep);
        uint64_t first = 0;
        if (m && lane_id() == 0)
            first = atomicAdd(cnt, (unsigned long long)__popcll(m));
        first = readlane_u64(first, 0);
        // live <= occupied <= limit, the buffer's length; bounded all the same
        const uint64_t at = first + __popcll(m & lt);
        if (keep && at < t.limit)
            out[at] = v;
    }
}

__global__ void purge_clear_kernel(TableRef t, const unsigned long long* plan)
{
    if (!plan[0])
        return;
    const uint64_t n = 1ull << t.log2slots;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        t.slots[i] = kEmpty;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *t.live = 0;
        *t.occupied = 0;
    }
}

__global__ void purge_insert_kernel(TableRef t, const unsigned long long* plan,
                                    const uint64_t* __restrict__ keys, uint32_t* __restrict__ status)
{
    if (!plan[0])
        return;
    const uint64_t n = plan[1] < t.limit ? plan[1] : t.limit;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        insert_one(t, keys[i], status, nullptr);
}

__global__ void erase_kernel(TableRef t, const uint64_t* __restrict__ keys, uint64_t n)
{
    const uint64_t nbk = 1ull << (t.log2slots - 3);
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t k = canon_key(keys[i]);
        uint64_t b = home_bucket(k, t.log2slots);
        bool done = false;
        for (uint64_t step = 0; step < nbk && !done; step++, b = (b + 1) & (nbk - 1)) {
            for (uint32_t s = 0; s < kBucket && !done; s++) {
                uint64_t* slot = t.slots + b * kBucket + s;
                const uint64_t v = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (v == kEmpty) {
                    done = true;
                } else if (v == k) {
                    const unsigned long long prev = atomicCAS(
                        (unsigned long long*)slot, (unsigned long long)k, (unsigned long long)kTomb);
                    if (prev == k)
                        atomicAdd((unsigned long long*)t.live, ~0ull);  // -1
                    done = true;
                }
            }
        }
    }
}

__global__ void clear_kernel(uint64_t* __restrict__ slots, uint64_t n, uint64_t* live,
                             uint64_t* occupied)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        slots[i] = kEmpty;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *live = 0;
        *occupied = 0;
    }
}

// Tables of several instances emptied at once: grid row y clears table
// ids[y] (and its counts).
__global__ void clear_many_kernel(uint64_t* __restrict__ tables, uint32_t log2slots,
                                  const uint32_t* __restrict__ ids, uint64_t* __restrict__ counts,
                                  uint32_t S)
{
    const uint32_t id = ids[blockIdx.y];
    uint64_t* slots = tables + ((uint64_t)id << log2slots);
    const uint64_t n = 1ull << log2slots;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        slots[i] = kEmpty;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        counts[id] = 0;      // live keys
        counts[S + id] = 0;  // occupied slots
    }
}

// Key lists of several tables at once: keys[seg[i] .. seg[i+1]) belong to
// table i (seg: device [S + 1]).  Each thread finds its key's table by
// bisection over seg.
struct Tables {
    uint64_t* slots;   // [S << log2slots]
    uint64_t* counts;  // [2 S]: live keys, then occupied slots
    uint32_t log2slots, S;
    __device__ TableRef of(uint32_t id) const
    {
        return TableRef{slots + ((uint64_t)id << log2slots), counts + id, counts + S + id,
                        log2slots, 1ull << (log2slots - 1)};
    }
};

__device__ __forceinline__ uint32_t seg_of(const uint64_t* seg, uint32_t S, uint64_t i)
{
    uint32_t lo = 0, hi = S;  // seg[lo] <= i < seg[hi]
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (seg[mid] <= i)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Adds to a table's counts, once per wave when the wave's lanes share the
// table (the counters are few words that every insert would meet on).
__device__ __forceinline__ void add_counts(const TableRef& t, uint32_t id, bool mine,
                                           unsigned long long dl, unsigned long long docc)
{
    const uint32_t id0 = __builtin_amdgcn_readfirstlane(id);
    if (ballot(id != id0) == 0) {
        const unsigned long long c = __popcll(ballot(mine));
        if (c && lane_id() == __builtin_ctzll(ballot(true))) {
            if (dl)
                atomicAdd((unsigned long long*)t.live, c * dl);
            if (docc)
                atomicAdd((unsigned long long*)t.occupied, c * docc);
        }
    } else if (mine) {
        if (dl)
            atomicAdd((unsigned long long*)t.live, dl);
        if (docc)
            atomicAdd((unsigned long long*)t.occupied, docc);
    }
}

__global__ void erase_many_kernel(Tables T, const uint64_t* __restrict__ keys,
                                  const uint64_t* __restrict__ seg, uint64_t n)
{
    for (uint64_t i0 = blockIdx.x * (uint64_t)blockDim.x; i0 < n;
         i0 += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t i = i0 + threadIdx.x;
        const bool in = i < n;
        const uint32_t id = seg_of(seg, T.S, in ? i : n - 1);
        const TableRef t = T.of(id);
        const uint64_t nbk = 1ull << (t.log2slots - 3);
        const uint64_t k = in ? canon_key(keys[i]) : kEmpty;
        uint64_t b = home_bucket(k, t.log2slots);
        bool done = !in, gone = false;
        for (uint64_t step = 0; step < nbk && !done; step++, b = (b + 1) & (nbk - 1)) {
            for (uint32_t q = 0; q < kBucket && !done; q++) {
                uint64_t* slot = t.slots + b * kBucket + q;
                const uint64_t v = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (v == kEmpty) {
                    done = true;
                } else if (v == k) {
                    const unsigned long long prev = atomicCAS(
                        (unsigned long long*)slot, (unsigned long long)k, (unsigned long long)kTomb);
                    gone = prev == k;
                    done = true;
                }
            }
        }
        add_counts(t, id, gone, ~0ull, 0);  // live - 1 per key erased
    }
}

// fits[i] = 1 when table i has room for all of its keys without a rebuild
// (else the caller inserts into it alone, with the rebuild and overflow
// handling of index_insert).
__global__ void fits_many_kernel(Tables T, const uint64_t* __restrict__ seg,
                                 uint32_t* __restrict__ fits)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < T.S; i += gridDim.x * blockDim.x) {
        const uint64_t n = seg[i + 1] - seg[i];
        fits[i] = !n || *T.of(i).occupied + n <= (1ull << (T.log2slots - 1)) ? 1u : 0u;
    }
}

// Every table has room for all of its keys (checked before), so a key takes
// the first empty slot of its sequence without reserving a unit of the
// occupied count; the counts grow by the keys stored, per wave.
__global__ void insert_many_kernel(Tables T, const uint64_t* __restrict__ keys,
                                   const uint64_t* __restrict__ seg, uint64_t n,
                                   const uint32_t* __restrict__ fits, uint32_t* __restrict__ status)
{
    for (uint64_t i0 = blockIdx.x * (uint64_t)blockDim.x; i0 < n;
         i0 += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t i = i0 + threadIdx.x;
        const bool in = i < n;
        const uint32_t id = seg_of(seg, T.S, in ? i : n - 1);
        const TableRef t = T.of(id);
        bool stored = false;
        if (in && fits[id]) {
            const uint64_t k = canon_key(keys[i]);
            const uint64_t nbk = 1ull << (t.log2slots - 3);
            uint64_t b = home_bucket(k, t.log2slots);
            bool done = false;
            for (uint64_t step = 0; step < nbk && !done; step++, b = (b + 1) & (nbk - 1)) {
                for (uint32_t q = 0; q < kBucket && !done; q++) {
                    uint64_t* slot = t.slots + b * kBucket + q;
                    const uint64_t v =
                        __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (v == k) {
                        done = true;
                    } else if (v == kEmpty) {
                        const unsigned long long prev =
                            atomicCAS((unsigned long long*)slot, (unsigned long long)kEmpty,
                                      (unsigned long long)k);
                        stored = prev == kEmpty;
                        done = stored || prev == k;  // else another key took it: walk on
                    }
                }
            }
            if (!done)
                atomicOr(status, kErrFull);
        }
        add_counts(t, id, stored, 1, 1);
    }
}

TableRef table_of(dm_ctx* c, uint32_t id)
{
    const uint32_t k = c->cfg.index_log2_slots;
    return TableRef{c->d_tables + ((uint64_t)id << k), c->d_counts + id,
                    c->d_counts + c->cfg.max_slots + id, k, 1ull << (k - 1)};
}


}  // namespace

hipError_t index_insert(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n)
{
    const TableRef t = table_of(c, id);
    hipError_t e = hipSuccess;
    // work area: plan word, gather count, overflow count, then up to `limit`
    // gathered live keys, then up to n overflow keys
    unsigned long long* w = static_cast<unsigned long long*>(
        scratch_get(c, kPurgeSlot, (t.limit + n + 3) * sizeof(uint64_t), &e));
    if (!w)
        return e;
    uint64_t* gathered = reinterpret_cast<uint64_t*>(w + 3);
    const Overflow ovf{w + 2, gathered + t.limit};
    const uint64_t nslots = 1ull << t.log2slots;
    purge_plan_kernel<<<1, 1, 0, c->stream>>>(t, n, w);
    purge_gather_kernel<<<grid_for(nslots, 256, 4096), 256, 0, c->stream>>>(t, w, w + 1, gathered);
    purge_clear_kernel<<<grid_for(nslots, 256, 4096), 256, 0, c->stream>>>(t, w);
    purge_insert_kernel<<<grid_for(t.limit, 256, 4096), 256, 0, c->stream>>>(t, w, gathered,
                                                                            c->d_status);
    insert_kernel<<<grid_for(n, 256), 256, 0, c->stream>>>(t, keys, n, c->d_status, ovf);
    overflow_kernel<<<1, kWave, 0, c->stream>>>(t, ovf, c->d_status);
    return hipGetLastError();
}

hipError_t index_erase(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n)
{
    erase_kernel<<<grid_for(n, 256), 256, 0, c->stream>>>(table_of(c, id), keys, n);
    return hipGetLastError();
}

hipError_t index_erase_many(dm_ctx* c, const uint64_t* keys, const uint64_t* seg, uint64_t n)
{
    if (n == 0)
        return hipSuccess;
    const Tables T{c->d_tables, c->d_counts, c->cfg.index_log2_slots, c->cfg.max_slots};
    erase_many_kernel<<<grid_for(n, 256), 256, 0, c->stream>>>(T, keys, seg, n);
    return hipGetLastError();
}

hipError_t index_insert_many(dm_ctx* c, const uint64_t* keys, const uint64_t* seg,
                             const uint64_t* seg_host, uint64_t n)
{
    if (n == 0)
        return hipSuccess;
    const uint32_t S = c->cfg.max_slots;
    const Tables T{c->d_tables, c->d_counts, c->cfg.index_log2_slots, S};
    hipError_t e = hipSuccess;
    // a flag per table: room for all of its keys
    uint32_t* fits = static_cast<uint32_t*>(scratch_get(c, kPurgeSlot, 4 * (size_t)S + 256, &e));
    if (!fits)
        return e;
    std::vector<uint32_t> fits_h(S);
    fits_many_kernel<<<grid_for(S, 256), 256, 0, c->stream>>>(T, seg, fits);
    insert_many_kernel<<<grid_for(n, 256), 256, 0, c->stream>>>(T, keys, seg, n, fits,
                                                                 c->d_status);
    if ((e = hipMemcpyAsync(fits_h.data(), fits, 4 * (size_t)S, hipMemcpyDeviceToHost,
                            c->stream)) != hipSuccess ||
        (e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return e;
    // tables without room: one at a time, with the rebuild and overflow handling
    for (uint32_t i = 0; i < S; i++)
        if (!fits_h[i] &&
            (e = index_insert(c, i, keys + seg_host[i], seg_host[i + 1] - seg_host[i])) !=
                hipSuccess)
            return e;
    return hipSuccess;
}

hipError_t index_clear_many(dm_ctx* c, const uint32_t* ids_host, uint32_t n)
{
    if (n == 0)
        return hipSuccess;
    hipError_t e = hipSuccess;
    uint32_t* d = static_cast<uint32_t*>(scratch_get(c, kPurgeSlot, n * sizeof(uint32_t), &e));
    if (!d)
        return e;
    if ((e = hipMemcpyAsync(d, ids_host, n * sizeof(uint32_t), hipMemcpyHostToDevice,
                            c->stream)) != hipSuccess ||
        (e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return e;
    const uint32_t k = c->cfg.index_log2_slots;
    const uint64_t per = std::max<uint64_t>(1, 4096 / n);
    dim3 grid((uint32_t)std::min<uint64_t>(per, ((1ull << k) + 255) / 256), n);
    clear_many_kernel<<<grid, 256, 0, c->stream>>>(c->d_tables, k, d, c->d_counts,
                                                   c->cfg.max_slots);
    return hipGetLastError();
}

hipError_t index_clear(dm_ctx* c, uint32_t id)
{
    const TableRef t = table_of(c, id);
    const uint64_t n = 1ull << t.log2slots;
    clear_kernel<<<grid_for(n, 256, 4096), 256, 0, c->stream>>>(t.slots, n, t.live, t.occupied);
    return hipGetLastError();
}

}  // namespace dm
