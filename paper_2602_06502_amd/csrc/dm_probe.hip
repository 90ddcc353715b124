// Candidates and longest cached prefixes (Sec. 3.2; Sec. A.1.1).
//
// lookup_kernel: one thread per request finds the owners of its two ring
//   keys and applies the distinct-candidate adjustment.
// probe_kernel: the longest cached prefix on each candidate, first miss
//   exact.  Requests are first ordered by the top 16 bits of their first
//   ring key, which puts requests that share a prompt prefix (hence the
//   same candidates and the same leading block keys) side by side.  A wave
//   takes 64 consecutive requests on one of the two candidates, all lanes
//   walking their key sequences in step: lanes that share a prefix load the
//   same 64-byte bucket in the same instruction, so one line fetch serves
//   them all, and they tend to stop at the same block.  No probe past a
//   lane's first miss is issued.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeSlot = kSlotProbe;  // sort keys, request order and sort work arrays
constexpr int kOrderBits = 16;            // top bits of the first ring key used for ordering

typedef unsigned long long v2u64 __attribute__((ext_vector_type(2), aligned(16)));

__global__ void lookup_kernel(uint64_t n, uint64_t q0, uint64_t q1, const uint64_t* __restrict__ key,
                              RingView r1, RingView r2, const uint32_t* __restrict__ next_live,
                              uint32_t n_live, uint32_t* __restrict__ cand,
                              uint8_t* __restrict__ flags)
{
    for (uint64_t r = q0 + blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < q1;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t c1 = ring_owner(r1, key[r]);
        uint32_t c2 = ring_owner(r2, key[n + r]);
        uint8_t f = 0;
        if (c2 == c1) {
            f = 8;
            c2 = n_live >= 2 ? next_live[c1] : c1;
        }
        cand[r] = c1;
        cand[n + r] = c2;
        flags[r] = f;
    }
}

// keys[i] = top kOrderBits bits of request r0 + i's first ring key;
// vals[i] = r0 + i.
__global__ void order_init_kernel(const uint64_t* __restrict__ key, uint64_t r0, uint64_t m,
                                  uint64_t* __restrict__ keys, uint32_t* __restrict__ vals)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x) {
        keys[i] = key[r0 + i] >> (64 - kOrderBits);
        vals[i] = (uint32_t)(r0 + i);
    }
}

struct ProbeArgs {
    const uint64_t* hkeys;
    const uint64_t* bstart;
    const uint32_t* bad;  // malformed offsets: no block key was written
    uint64_t n;      // batch size (cand and match hold 2n entries)
    uint64_t count;  // requests in order[]
    const uint32_t* cand;
    const uint64_t* tables;
    uint32_t log2slots;
    uint32_t* match;
    const uint32_t* order;  // [count] requests ordered by first ring key prefix
    uint32_t* status;
    unsigned long long* next;  // per-XCD group counters, kCounterStride apart, zeroed
};

// Probe outcome of one key against one bucket: the key is there, the bucket
// has an empty slot (so the key is absent: the probe sequence of an insert
// would have stopped here), or neither (go on to the next bucket).  Inserts
// take a bucket's slots in order and slots never return to empty, so a
// bucket's empty slots are a suffix of it: it has one iff its last slot is.
enum : int { kHit = 0, kMiss = 1, kNext = 2 };

__device__ __forceinline__ int bucket_probe(const uint64_t* tab, uint32_t bkt, uint64_t key)
{
    const v2u64* line = reinterpret_cast<const v2u64*>(tab + (uint64_t)bkt * kBucket);
    const v2u64 s0 = line[0], s1 = line[1], s2 = line[2], s3 = line[3];
    const bool hit = s0.x == key || s0.y == key || s1.x == key || s1.y == key || s2.x == key ||
                     s2.y == key || s3.x == key || s3.y == key;
    return hit ? kHit : (s3.y == kEmpty ? kMiss : kNext);
}

// Home bucket of a canonical key in 8-slot buckets of a 2^ls-slot table
// (ls <= 30): its top ls - 3 bits.
__device__ __forceinline__ uint32_t home32(uint64_t ck, uint32_t ls)
{
    return (uint32_t)(ck >> 32) >> (35 - ls);
}

// Block keys of a lane's probe sequence are read kWin at a time into a
// window in LDS; a step needs the keys of its two blocks and of the two
// after them, so a window serves three steps and only one step in three
// waits for HBM (keys are touched once, by the probe that needs them, long
// after the hash kernel wrote them).
constexpr int kWin = 8;

typedef unsigned long long v2u64a8 __attribute__((ext_vector_type(2), aligned(8)));

// Loads hk[q, q + kWin) (zeros from index lim on) into w[0..kWin).
__device__ __forceinline__ void window_load(const uint64_t* hk, uint64_t q, uint64_t lim,
                                            uint64_t (&w)[kWin])
{
    if (q + kWin <= lim) {
        const v2u64a8* p = reinterpret_cast<const v2u64a8*>(hk + q);
#pragma unroll
        for (int k = 0; k < kWin / 2; k++) {
            const v2u64a8 v = p[k];
            w[2 * k] = v.x;
            w[2 * k + 1] = v.y;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kWin; k++)
            w[k] = q + k < lim ? hk[q + k] : 0;
    }
}

// Groups are claimed one at a time: the waves of XCD x (workgroups x, x + 8,
// ...) take claims h = x, x + 8, x + 16, ... in turn through a counter of
// their own, on a line of its own, so group lengths (unknown until probed)
// even out inside each XCD.  Claim h is request block ((h >> 4) << 3) | (h & 7)
// on candidate (h >> 3) & 1: an XCD probes both candidates of its blocks,
// one after the other (their block keys are shared through its L2), and the
// XCDs get statistically equal shares.
constexpr uint32_t kXcds = 8;
constexpr uint32_t kCounterStride = 32;  // 256 bytes

__global__ void probe_zero_kernel(unsigned long long* next)
{
    if (threadIdx.x < kXcds)
        next[threadIdx.x * kCounterStride] = 0;
}

// Longest cached prefix of every (request, candidate), first miss exact.
// A group covers the 64 requests of one block of the ordered list on one of
// their candidates.  Within a group every lane probes two
// consecutive blocks per step (slot 0: the first unresolved block kb,
// slot 1: kb + 1), the keys of the next two coming from its window; a step
// resolves up to two blocks.  The group is done when every lane has met its
// first miss or its last full block.  Block positions are relative to the
// request's first block (a request has fewer than 2^32 full blocks, as its
// 32-bit match length requires; more set the status word).
__global__ __launch_bounds__(kProbeThreads) void probe_kernel(ProbeArgs a)
{
    __shared__ uint64_t win_all[kProbeThreads / kWave][kWin][kWave];
    const int lane = lane_id();
    uint64_t (*win)[kWave] = win_all[threadIdx.x >> 6];
    const uint64_t nblk = (a.count + kWave - 1) / kWave;
    const uint64_t nclaims = 16 * ((nblk + kXcds - 1) / kXcds);
    const uint32_t xcd = blockIdx.x % kXcds;
    unsigned long long* counter = a.next + xcd * kCounterStride;
    const uint32_t nbk = 1u << (a.log2slots - 3);
    const uint32_t ls = a.log2slots;
    const bool bad = *a.bad != 0;
    const uint64_t total = bad ? 0 : a.bstart[a.n];  // block keys in hkeys
    // the claim of the next group is issued before the current one is probed
    uint64_t claim = 0;
    if (lane == 0)
        claim = atomicAdd(counter, 1ull);
    uint64_t h = xcd + kXcds * readlane_u64(claim, 0);
    while (h < nclaims) {
        if (lane == 0)
            claim = atomicAdd(counter, 1ull);
        const uint64_t blk = ((h >> 4) << 3) | (h & 7), side = (h >> 3) & 1;
        const uint64_t i = blk * kWave + lane;
        const bool valid = i < a.count;
        uint64_t k0 = 0, out = 0;
        uint32_t len = 0;
        const uint64_t* tab = a.tables;
        if (valid) {
            const uint32_t r = a.order[i];
            out = side * a.n + r;
            k0 = a.bstart[r];
            const uint64_t ke = a.bstart[(uint64_t)r + 1];
            if (ke - k0 > 0xFFFFFFFFull) {
                atomicOr(a.status, kErrInval);
                k0 = ke;
            }
            len = bad ? 0u : (uint32_t)(ke - k0);
            tab = a.tables + ((uint64_t)a.cand[out] << ls);
        }
        const uint64_t* hk = a.hkeys + k0;
        const uint64_t lim = total > k0 ? total - k0 : 0;  // keys readable from hk
        bool active = valid && len > 0;
        if (valid && !active)
            a.match[out] = 0;  // no full block
        // slot 0: block kb; slot 1: block kb + 1 (when kb + 1 < len); the
        // window holds blocks [w0, w0 + kWin)
        uint32_t kb = 0, w0 = 0, st0 = 0, st1 = 0;
        uint64_t key0 = 0, key1 = 0;
        if (active) {
            uint64_t w[kWin];
            window_load(hk, 0, lim, w);
#pragma unroll
            for (int k = 0; k < kWin; k++)
                win[k][lane] = w[k];
            key0 = canon_key(w[0]);
            key1 = canon_key(w[1]);
        }
        uint32_t b0 = home32(key0, ls), b1 = home32(key1, ls);
        while (__any(active)) {
            const bool two = kb + 1 < len;
            int r0 = kMiss, r1 = kMiss;
            if (active) {
                r0 = bucket_probe(tab, b0, key0);
                r1 = bucket_probe(tab, b1, key1);  // slot 1 past the last block: a valid, unused bucket
            }
            // the window covers blocks kb + 2 and kb + 3 (kb + 4 <= w0 + kWin)
            const uint64_t c2 = canon_key(win[kb + 2 - w0][lane]);
            const uint64_t c3 = canon_key(win[kb + 3 - w0][lane]);
            const bool h0 = r0 == kHit, h1 = two && r1 == kHit;
            const uint32_t adv = h0 ? (h1 ? 2u : 1u) : 0u;
            // next step of slot 0's sequence (slot 0 unresolved), or of slot
            // 1's sequence moving to slot 0 (block kb present)
            const uint32_t nst = h0 ? st1 + 1 : st0 + 1;
            const bool fin = active && (!h0 ? (r0 == kMiss || nst >= nbk)
                                            : (!two || r1 == kMiss || (h1 ? kb + 2 == len : nst >= nbk)));
            if (fin)
                a.match[out] = kb + adv;
            const bool go = active && !fin;
            // slot 0 unresolved: it goes on to its next bucket and slot 1 is
            // probed again; both present: the next two blocks; block kb
            // present only: slot 1's sequence continues in slot 0
            const uint64_t nk0 = !h0 ? key0 : (h1 ? c2 : key1);
            const uint64_t nk1 = !h0 ? key1 : (h1 ? c3 : c2);
            const uint32_t nb0 = !h0 ? ((b0 + 1) & (nbk - 1))
                                     : (h1 ? home32(c2, ls) : ((b1 + 1) & (nbk - 1)));
            const uint32_t nb1 = !h0 ? b1 : home32(h1 ? c3 : c2, ls);
            key0 = go ? nk0 : key0;
            key1 = go ? nk1 : key1;
            b0 = go ? nb0 : b0;
            b1 = go ? nb1 : b1;
            st0 = go ? (h1 ? 0u : nst) : st0;
            st1 = go && h0 ? 0u : st1;
            kb = go ? kb + adv : kb;
            active = go;
            // the next step reads blocks kb + 2 and kb + 3 from the window
            const bool refill = go && kb + 4 > w0 + kWin;
            if (__any(refill) && refill) {
                uint64_t w[kWin];
                window_load(hk, kb, lim, w);
                w0 = kb;
#pragma unroll
                for (int k = 0; k < kWin; k++)
                    win[k][lane] = w[k];
            }
        }
        h = xcd + kXcds * readlane_u64(claim, 0);
    }
}

}  // namespace

// Sort keys and request order (each twice, for the sort's passes), then the
// per-XCD claim counters.
uint64_t probe_scratch_bytes(uint64_t m)
{
    const size_t kbytes = ((m * sizeof(uint64_t)) + 255) & ~size_t(255);
    const size_t vbytes = ((m * sizeof(uint32_t)) + 255) & ~size_t(255);
    const size_t cbytes = kXcds * kCounterStride * sizeof(unsigned long long);
    return 2 * (kbytes + vbytes) + cbytes + 256;
}

hipError_t lookup_probe(dm_ctx* c, uint64_t n, const uint64_t* key, const uint64_t* hkeys,
                        const uint64_t* bstart, const uint32_t* bad, uint32_t* cand,
                        uint32_t* match, uint8_t* flags, uint64_t r0, uint64_t r1)
{
    hipError_t e = hipSuccess;
    hipStream_t st = c->stream;
    if (r1 <= r0)
        return hipSuccess;
    const uint64_t m = r1 - r0;
    lookup_kernel<<<grid_for(m, 256, 8192), 256, 0, st>>>(
        n, r0, r1, key, view(c->ring[c->cur][0]), view(c->ring[c->cur][1]), c->d_next_live,
        c->n_live, cand, flags);
    if (r1 > 0xFFFFFFFFull)
        return hipErrorInvalidValue;
    // requests ordered by the top bits of their first ring key (stable radix sort)
    const size_t kbytes = ((m * sizeof(uint64_t)) + 255) & ~size_t(255);
    const size_t vbytes = ((m * sizeof(uint32_t)) + 255) & ~size_t(255);
    uint8_t* w = static_cast<uint8_t*>(scratch_get(c, kProbeSlot, probe_scratch_bytes(m), &e));
    if (!w)
        return e;
    uint64_t* keys = reinterpret_cast<uint64_t*>(w);
    uint64_t* ktmp = reinterpret_cast<uint64_t*>(w + kbytes);
    uint32_t* order = reinterpret_cast<uint32_t*>(w + 2 * kbytes);
    uint32_t* vtmp = reinterpret_cast<uint32_t*>(w + 2 * kbytes + vbytes);
    unsigned long long* next =
        reinterpret_cast<unsigned long long*>(w + ((2 * (kbytes + vbytes) + 255) & ~size_t(255)));
    order_init_kernel<<<grid_for(m, 256, 8192), 256, 0, st>>>(key, r0, m, keys, order);
    if ((e = radix_sort_kv(c, keys, order, ktmp, vtmp, m, kOrderBits)) != hipSuccess)
        return e;
    if (!c->probe_grid) {
        // persistent: as many workgroups as stay resident at once
        int per_cu = 0;
        if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, probe_kernel, kProbeThreads,
                                                              0)) != hipSuccess)
            return e;
        // every XCD residue class of workgroup indices needs workgroups
        const uint32_t g = (uint32_t)std::max(1, per_cu * std::max(1, c->n_cu));
        c->probe_grid = (g + kXcds - 1) / kXcds * kXcds;
    }
    ProbeArgs pa{hkeys, bstart, bad,   n,     m,           cand, c->d_tables,
                 c->cfg.index_log2_slots, match, order, c->d_status, next};
    probe_zero_kernel<<<1, 64, 0, st>>>(next);
    probe_kernel<<<c->probe_grid, kProbeThreads, 0, st>>>(pa);
    return hipGetLastError();
}

}  // namespace dm
