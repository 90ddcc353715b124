// Consistent-hash rings (Sec. 3.4; Sec. A.1.3): virtual-node placement,
// sorting, the bucket directory used by lookups, and the remap check of a
// membership change.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kRingSlot = kSlotRing;  // sort work arrays

// Virtual node v of live instance k on ring s sits at
// mix64(((id << 32) | v) xor mix64(seed_s)).
__global__ void vnode_kernel(const uint32_t* __restrict__ live_ids, uint32_t vnodes, uint64_t len,
                             uint64_t salt, uint64_t* __restrict__ pos, uint32_t* __restrict__ id)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < len;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t inst = live_ids[i / vnodes];
        const uint32_t v = (uint32_t)(i % vnodes);
        pos[i] = mix64((((uint64_t)inst << 32) | v) ^ salt);
        id[i] = inst;
    }
}

// dir[k] = first index whose position >= k << (64 - dbits), k = 0..2^dbits.
// Entry i (i = 0..len, i = len meaning "past the end") fills the buckets
// after its predecessor's bucket up to its own.
__global__ void directory_kernel(const uint64_t* __restrict__ pos, uint64_t len, uint32_t dbits,
                                 uint32_t* __restrict__ dir)
{
    const uint64_t nb = 1ull << dbits;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i <= len;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t lo = i == 0 ? 0 : (pos[i - 1] >> (64 - dbits)) + 1;
        const uint64_t hi = i == len ? nb : (pos[i] >> (64 - dbits));
        for (uint64_t b = lo; b <= hi; b++)
            dir[b] = (uint32_t)i;
    }
}

// Rings of up to kBucketSortMax positions are sorted by bucket instead of
// by radix passes: with 2^dbits >= len buckets on the top bits, a bucket
// holds about one position, so counting, placing and a per-bucket insertion
// sort take four launches, and the bucket counts' scan is the directory.
// Positions are distinct (bijective in (id, v)), so the order is unique.
constexpr uint64_t kBucketSortMax = 1ull << 22;

__global__ void fill_u64_kernel(uint64_t* __restrict__ p, uint64_t n)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// Virtual nodes as vnode_kernel, each counted in its bucket; rank = its
// place among its bucket's (any order: the bucket is sorted afterwards).
__global__ void vnode_count_kernel(const uint32_t* __restrict__ live_ids, uint32_t vnodes,
                                   uint64_t len, uint64_t salt, uint32_t dbits,
                                   uint64_t* __restrict__ pos, uint32_t* __restrict__ id,
                                   unsigned long long* __restrict__ cnt,
                                   uint32_t* __restrict__ rank)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < len;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t inst = live_ids[i / vnodes];
        const uint32_t v = (uint32_t)(i % vnodes);
        const uint64_t x = mix64((((uint64_t)inst << 32) | v) ^ salt);
        pos[i] = x;
        id[i] = inst;
        rank[i] = (uint32_t)atomicAdd(&cnt[x >> (64 - dbits)], 1ull);
    }
}

__global__ void bucket_place_kernel(const uint64_t* __restrict__ pos,
                                    const uint32_t* __restrict__ id,
                                    const uint32_t* __restrict__ rank, uint64_t len,
                                    uint32_t dbits, const uint64_t* __restrict__ start,
                                    uint64_t* __restrict__ out_pos, uint32_t* __restrict__ out_id)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < len;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t d = start[pos[i] >> (64 - dbits)] + rank[i];
        out_pos[d] = pos[i];
        out_id[d] = id[i];
    }
}

// Each bucket's positions in order (insertion sort; a bucket holds a few),
// and the directory: dir[b] = the bucket's first index, dir[2^dbits] = len.
__global__ void bucket_sort_kernel(uint64_t* __restrict__ pos, uint32_t* __restrict__ id,
                                   uint64_t len, uint32_t dbits,
                                   const uint64_t* __restrict__ start, uint32_t* __restrict__ dir)
{
    const uint64_t nb = 1ull << dbits;
    for (uint64_t b = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; b <= nb;
         b += (uint64_t)gridDim.x * blockDim.x) {
        if (b == nb) {
            dir[b] = (uint32_t)len;
            continue;
        }
        const uint64_t lo = start[b], hi = b + 1 < nb ? start[b + 1] : len;
        dir[b] = (uint32_t)lo;
        for (uint64_t i = lo + 1; i < hi; i++) {
            const uint64_t x = pos[i];
            const uint32_t y = id[i];
            uint64_t j = i;
            while (j > lo && pos[j - 1] > x) {
                pos[j] = pos[j - 1];
                id[j] = id[j - 1];
                j--;
            }
            pos[j] = x;
            id[j] = y;
        }
    }
}

__global__ void zero_u64_kernel(uint64_t* p, uint32_t n)
{
    if (threadIdx.x < n)
        p[threadIdx.x] = 0;
}

__global__ void remap_kernel(RingView o1, RingView o2, RingView n1, RingView n2,
                             const uint64_t* __restrict__ keys, uint64_t n,
                             const uint8_t* __restrict__ is_add, const uint8_t* __restrict__ is_rm,
                             uint32_t* __restrict__ old_owner, uint32_t* __restrict__ new_owner,
                             uint64_t* __restrict__ moved, uint64_t* __restrict__ violations)
{
    // counts gather per wave over the grid-stride loop, then per workgroup in
    // LDS: three device atomics per workgroup, not per wave
    __shared__ unsigned long long s_cnt[3];
    if (threadIdx.x < 3)
        s_cnt[threadIdx.x] = 0;
    __syncthreads();
    uint64_t c1 = 0, c2 = 0, cb = 0;
    const uint64_t total = 2 * n;
    for (uint64_t base = blockIdx.x * (uint64_t)blockDim.x; base < total;
         base += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t k = base + threadIdx.x;
        const bool ok = k < total;
        const bool second = ok && k >= n;
        bool mv = false, bad = false;
        if (ok) {
            const uint64_t x = keys[k];
            const uint32_t a = ring_owner(second ? o2 : o1, x);
            const uint32_t b = ring_owner(second ? n2 : n1, x);
            old_owner[k] = a;
            new_owner[k] = b;
            mv = a != b;
            bad = mv && !is_rm[a] && !is_add[b];
        }
        c1 += __popcll(ballot(mv && !second));
        c2 += __popcll(ballot(mv && second));
        cb += __popcll(ballot(bad));
    }
    if ((threadIdx.x & 63) == 0) {
        if (c1) atomicAdd(&s_cnt[0], (unsigned long long)c1);
        if (c2) atomicAdd(&s_cnt[1], (unsigned long long)c2);
        if (cb) atomicAdd(&s_cnt[2], (unsigned long long)cb);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        if (s_cnt[0]) atomicAdd((unsigned long long*)&moved[0], s_cnt[0]);
        if (s_cnt[1]) atomicAdd((unsigned long long*)&moved[1], s_cnt[1]);
        if (s_cnt[2]) atomicAdd((unsigned long long*)violations, s_cnt[2]);
    }
}


}  // namespace

hipError_t ring_build(dm_ctx* c, Ring& r, int s, const uint32_t* d_live_ids, uint32_t n_live)
{
    const uint64_t len = (uint64_t)n_live * c->cfg.vnodes;
    uint32_t dbits = 1;
    while ((1ull << dbits) < len && dbits < 24)
        dbits++;
    hipError_t e = hipSuccess;
    if (r.cap < len) {
        e = hipStreamSynchronize(c->stream);
        (void)hipFree(r.pos);
        (void)hipFree(r.id);
        r.pos = nullptr;
        r.id = nullptr;
        r.cap = 0;
        if (e == hipSuccess) e = hipMalloc(&r.pos, len * sizeof(uint64_t));
        if (e == hipSuccess) e = hipMalloc(&r.id, len * sizeof(uint32_t));
        if (e != hipSuccess)
            return e;
        r.cap = len;
    }
    const uint32_t dneed = (1u << dbits) + 1;
    if (r.dcap < dneed) {
        e = hipStreamSynchronize(c->stream);
        (void)hipFree(r.dir);
        r.dir = nullptr;
        r.dcap = 0;
        if (e == hipSuccess) e = hipMalloc(&r.dir, dneed * sizeof(uint32_t));
        if (e != hipSuccess)
            return e;
        r.dcap = dneed;
    }
    const uint64_t salt = mix64(c->cfg.seed[s]);
    if (len <= kBucketSortMax && (1ull << dbits) >= len) {
        const uint64_t nb = 1ull << dbits;
        const size_t lenb = (len * 8 + 255) & ~size_t(255), nbb = (nb * 8 + 255) & ~size_t(255);
        uint8_t* w = static_cast<uint8_t*>(
            scratch_get(c, kRingSlot, lenb + 2 * ((len * 4 + 255) & ~size_t(255)) + 2 * nbb + 256,
                        &e));
        if (!w)
            return e;
        uint64_t* ptmp = reinterpret_cast<uint64_t*>(w);
        uint32_t* itmp = reinterpret_cast<uint32_t*>(w + lenb);
        uint32_t* rank = reinterpret_cast<uint32_t*>(w + lenb + ((len * 4 + 255) & ~size_t(255)));
        uint64_t* cnt = reinterpret_cast<uint64_t*>(w + lenb + 2 * ((len * 4 + 255) & ~size_t(255)));
        uint64_t* start = cnt + nbb / 8;
        uint64_t* total = start + nbb / 8;
        fill_u64_kernel<<<grid_for(nb, 256, 4096), 256, 0, c->stream>>>(cnt, nb);
        vnode_count_kernel<<<grid_for(len, 256), 256, 0, c->stream>>>(
            d_live_ids, c->cfg.vnodes, len, salt, dbits, ptmp, itmp,
            reinterpret_cast<unsigned long long*>(cnt), rank);
        if ((e = hipGetLastError()) != hipSuccess ||
            (e = exclusive_scan_u64(c, cnt, nb, start, total)) != hipSuccess)
            return e;
        bucket_place_kernel<<<grid_for(len, 256), 256, 0, c->stream>>>(ptmp, itmp, rank, len,
                                                                        dbits, start, r.pos,
                                                                        r.id);
        bucket_sort_kernel<<<grid_for(nb + 1, 256), 256, 0, c->stream>>>(r.pos, r.id, len, dbits,
                                                                          start, r.dir);
        r.len = len;
        r.dbits = dbits;
        return hipGetLastError();
    }
    uint8_t* tmp = static_cast<uint8_t*>(
        scratch_get(c, kRingSlot, len * (sizeof(uint64_t) + sizeof(uint32_t)) + 64, &e));
    if (!tmp)
        return e;
    uint64_t* ktmp = reinterpret_cast<uint64_t*>(tmp);
    uint32_t* vtmp = reinterpret_cast<uint32_t*>(tmp + len * sizeof(uint64_t));
    vnode_kernel<<<grid_for(len, 256), 256, 0, c->stream>>>(d_live_ids, c->cfg.vnodes, len, salt,
                                                            r.pos, r.id);
    e = hipGetLastError();
    if (e == hipSuccess)
        e = radix_sort_kv(c, r.pos, r.id, ktmp, vtmp, len, 64);
    if (e != hipSuccess)
        return e;
    directory_kernel<<<grid_for(len + 1, 256), 256, 0, c->stream>>>(r.pos, len, dbits, r.dir);
    r.len = len;
    r.dbits = dbits;
    return hipGetLastError();
}

hipError_t ring_remap(dm_ctx* c, const Ring old_r[2], const Ring new_r[2], const uint64_t* keys,
                      uint64_t n, uint32_t* old_owner, uint32_t* new_owner, uint64_t* moved,
                      uint64_t* violations)
{
    zero_u64_kernel<<<1, 64, 0, c->stream>>>(moved, 2);
    zero_u64_kernel<<<1, 64, 0, c->stream>>>(violations, 1);
    if (n)
        remap_kernel<<<grid_for(2 * n, 256, 1024), 256, 0, c->stream>>>(
            view(old_r[0]), view(old_r[1]), view(new_r[0]), view(new_r[1]), keys, n,
            c->d_flag_add, c->d_flag_rm, old_owner, new_owner, moved, violations);
    return hipGetLastError();
}

}  // namespace dm
