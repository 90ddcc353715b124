// Per-instance cached-block index (the KV metadata of Sec. A.3.2): one
// open-addressing table of 2^k u64 keys per instance slot, probed a bucket
// of 8 slots (one 64-byte line) at a time, buckets in linear order from the
// key's home bucket.  Slot 0 = empty, 1 = erased; stored keys are >= 2.
// An insert takes the first empty slot of the probe sequence, so an empty
// slot seen during a lookup proves the key absent.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kPurgeSlot = 8;  // table rebuild work area

struct TableRef {
    uint64_t* slots;
    uint64_t* live;      // live key count
    uint64_t* occupied;  // non-empty slots (live + erased)
    uint32_t log2slots;
    uint64_t limit;      // maximum occupied slots
};

// Insert of one canonical key (>= 2); set semantics.
__device__ __forceinline__ void insert_one(const TableRef& t, uint64_t k, uint32_t* status)
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
                if (__hip_atomic_load(t.occupied, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >=
                    t.limit) {
                    atomicOr(status, kErrFull);
                    return;
                }
                const unsigned long long prev = atomicCAS(
                    (unsigned long long*)slot, (unsigned long long)kEmpty, (unsigned long long)k);
                if (prev == kEmpty) {
                    atomicAdd((unsigned long long*)t.occupied, 1ull);
                    atomicAdd((unsigned long long*)t.live, 1ull);
                    done = true;
                } else if (prev == k) {
                    done = true;
                }
                // else another key took the slot: keep walking
            }
        }
    }
    if (!done)
        atomicOr(status, kErrFull);  // every slot scanned: table full
}

__global__ void insert_kernel(TableRef t, const uint64_t* __restrict__ keys, uint64_t n,
                              uint32_t* __restrict__ status)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        insert_one(t, canon_key(keys[i]), status);
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
    plan[1] = 0;
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
        if (keep)
            out[first + __popcll(m & lt)] = v;
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
    const uint64_t n = plan[1];
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        insert_one(t, keys[i], status);
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
    // rebuild work area: plan word, gather counter, then up to `limit` live keys
    unsigned long long* w = static_cast<unsigned long long*>(
        scratch_get(c, kPurgeSlot, (t.limit + 2) * sizeof(uint64_t), &e));
    if (!w)
        return e;
    const uint64_t nslots = 1ull << t.log2slots;
    purge_plan_kernel<<<1, 1, 0, c->stream>>>(t, n, w);
    purge_gather_kernel<<<grid_for(nslots, 256, 4096), 256, 0, c->stream>>>(
        t, w, w + 1, reinterpret_cast<uint64_t*>(w + 2));
    purge_clear_kernel<<<grid_for(nslots, 256, 4096), 256, 0, c->stream>>>(t, w);
    purge_insert_kernel<<<grid_for(t.limit, 256, 4096), 256, 0, c->stream>>>(
        t, w, reinterpret_cast<const uint64_t*>(w + 2), c->d_status);
    insert_kernel<<<grid_for(n, 256), 256, 0, c->stream>>>(table_of(c, id), keys, n, c->d_status);
    return hipGetLastError();
}

hipError_t index_erase(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n)
{
    erase_kernel<<<grid_for(n, 256), 256, 0, c->stream>>>(table_of(c, id), keys, n);
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
