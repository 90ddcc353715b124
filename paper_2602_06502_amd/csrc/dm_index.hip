// Per-instance cached-block index (the KV metadata of Sec. A.3.2): one
// open-addressing table of 2^k u64 keys per instance slot, probed a bucket
// of 8 slots (one 64-byte line) at a time, buckets in linear order from the
// key's home bucket.  Slot 0 = empty, 1 = erased; stored keys are >= 2.
// An insert takes the first empty slot of the probe sequence, so an empty
// slot seen during a lookup proves the key absent.
#include "dm_internal.h"

namespace dm {
namespace {

struct TableRef {
    uint64_t* slots;
    uint64_t* live;      // live key count
    uint64_t* occupied;  // non-empty slots (live + erased)
    uint32_t log2slots;
    uint64_t limit;      // maximum occupied slots
};

__global__ void insert_kernel(TableRef t, const uint64_t* __restrict__ keys, uint64_t n,
                              uint32_t* __restrict__ status)
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
                uint64_t v = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (v == k) {
                    done = true;
                } else if (v == kEmpty) {
                    if (__hip_atomic_load(t.occupied, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >=
                        t.limit) {
                        atomicOr(status, kErrFull);
                        done = true;
                        break;
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
