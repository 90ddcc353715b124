// Candidates and longest cached prefixes (Sec. 3.2; Sec. A.1.1).
//
// lookup_kernel: one thread per request finds the owners of its two ring
//   keys and applies the distinct-candidate adjustment.
// probe_kernel: the longest cached prefix on each candidate, first miss
//   exact.  Requests are first ordered by the top 16 bits of their first
//   ring key, which puts requests that share a prompt prefix (hence the
//   same candidates and the same leading block keys) side by side.  A wave
//   takes 32 consecutive requests, lanes 0-31 probing their first
//   candidate and lanes 32-63 their second, all walking their key
//   sequences in step: lanes that share a prefix load the same 64-byte
//   bucket in the same instruction, so one line fetch serves them all.  No
//   probe past a lane's first miss is issued.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeSlot = 1;             // sort keys, request order and sort work arrays
constexpr uint32_t kProbeBlocks = 2048;   // persistent: 8,192 waves, 256 CUs x 4 SIMDs x 8
constexpr int kGroupReq = kWave / 2;      // requests per wave step (two candidates each)
constexpr int kOrderBits = 16;            // top bits of the first ring key used for ordering

typedef unsigned long long v2u64 __attribute__((ext_vector_type(2), aligned(16)));

__global__ void lookup_kernel(uint64_t n, const uint64_t* __restrict__ key, RingView r1, RingView r2,
                              const uint32_t* __restrict__ next_live, uint32_t n_live,
                              uint32_t* __restrict__ cand, uint8_t* __restrict__ flags)
{
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
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

// keys[i] = top kOrderBits bits of request i's first ring key; vals[i] = i.
__global__ void order_init_kernel(const uint64_t* __restrict__ key, uint64_t n,
                                  uint64_t* __restrict__ keys, uint32_t* __restrict__ vals)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x) {
        keys[i] = key[i] >> (64 - kOrderBits);
        vals[i] = (uint32_t)i;
    }
}

struct ProbeArgs {
    const uint64_t* hkeys;
    const uint64_t* bstart;
    uint64_t n;
    const uint32_t* cand;
    const uint64_t* tables;
    uint32_t log2slots;
    uint32_t* match;
    const uint32_t* order;  // [n] requests ordered by first ring key prefix
};

// Longest cached prefix of every (request, candidate), first miss exact.
// Wave w takes request groups w, w + W, ... of the ordered list; within a
// group every lane probes one 64-byte bucket per step while the next block
// key of its sequence is already being fetched, and the group is done when
// every lane has met its first miss or its last full block.
__global__ __launch_bounds__(kProbeThreads) void probe_kernel(ProbeArgs a)
{
    const int lane = lane_id();
    const uint64_t gw = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const uint64_t ng = (a.n + kGroupReq - 1) / kGroupReq;
    const uint64_t nbk = 1ull << (a.log2slots - 3);
    const uint64_t side = lane >= kGroupReq ? a.n : 0;  // second candidate's half of cand/match
    for (uint64_t g = gw; g < ng; g += nw) {
        const uint64_t i = g * kGroupReq + (lane & (kGroupReq - 1));
        const bool valid = i < a.n;
        uint64_t kb = 0, ke = 0, out = 0;
        const uint64_t* tab = a.tables;
        if (valid) {
            const uint32_t r = a.order[i];
            out = side + r;
            kb = a.bstart[r];
            ke = a.bstart[(uint64_t)r + 1];
            tab = a.tables + ((uint64_t)a.cand[out] << a.log2slots);
        }
        const uint64_t k0 = kb;
        bool active = valid && kb < ke;
        if (valid && !active)
            a.match[out] = 0;  // no full block
        uint64_t key = active ? canon_key(a.hkeys[kb]) : 0;
        uint64_t bkt = home_bucket(key, a.log2slots), steps = 0;
        while (__any(active)) {
            if (active) {
                const v2u64* line = reinterpret_cast<const v2u64*>(tab + bkt * kBucket);
                const v2u64 s0 = line[0], s1 = line[1], s2 = line[2], s3 = line[3];
                const uint64_t nkey = kb + 1 < ke ? a.hkeys[kb + 1] : 0;
                const bool hit = s0.x == key || s0.y == key || s1.x == key || s1.y == key ||
                                 s2.x == key || s2.y == key || s3.x == key || s3.y == key;
                const bool empty = s0.x == kEmpty || s0.y == kEmpty || s1.x == kEmpty ||
                                   s1.y == kEmpty || s2.x == kEmpty || s2.y == kEmpty ||
                                   s3.x == kEmpty || s3.y == kEmpty;
                if (hit) {
                    kb++;
                    if (kb == ke) {
                        a.match[out] = (uint32_t)(kb - k0);
                        active = false;
                    } else {
                        key = canon_key(nkey);
                        bkt = home_bucket(key, a.log2slots);
                        steps = 0;
                    }
                } else if (empty || ++steps >= nbk) {
                    a.match[out] = (uint32_t)(kb - k0);  // first miss (or scanned the whole table)
                    active = false;
                } else {
                    bkt = (bkt + 1) & (nbk - 1);
                }
            }
        }
    }
}

}  // namespace

hipError_t lookup_probe(dm_ctx* c, uint64_t n, const uint64_t* key, const uint64_t* hkeys,
                        const uint64_t* bstart, uint32_t* cand, uint32_t* match, uint8_t* flags)
{
    hipError_t e = hipSuccess;
    hipStream_t st = c->stream;
    lookup_kernel<<<grid_for(n, 256, 8192), 256, 0, st>>>(
        n, key, view(c->ring[c->cur][0]), view(c->ring[c->cur][1]), c->d_next_live, c->n_live,
        cand, flags);
    if (n > 0xFFFFFFFFull)
        return hipErrorInvalidValue;
    // requests ordered by the top bits of their first ring key (stable radix sort)
    const size_t kbytes = ((n * sizeof(uint64_t)) + 255) & ~size_t(255);
    const size_t vbytes = ((n * sizeof(uint32_t)) + 255) & ~size_t(255);
    uint8_t* w = static_cast<uint8_t*>(scratch_get(c, kProbeSlot, 2 * (kbytes + vbytes) + 256, &e));
    if (!w)
        return e;
    uint64_t* keys = reinterpret_cast<uint64_t*>(w);
    uint64_t* ktmp = reinterpret_cast<uint64_t*>(w + kbytes);
    uint32_t* order = reinterpret_cast<uint32_t*>(w + 2 * kbytes);
    uint32_t* vtmp = reinterpret_cast<uint32_t*>(w + 2 * kbytes + vbytes);
    order_init_kernel<<<grid_for(n, 256, 8192), 256, 0, st>>>(key, n, keys, order);
    if ((e = radix_sort_kv(c, keys, order, ktmp, vtmp, n, kOrderBits)) != hipSuccess)
        return e;
    ProbeArgs pa{hkeys, bstart, n, cand, c->d_tables, c->cfg.index_log2_slots, match, order};
    probe_kernel<<<kProbeBlocks, kProbeThreads, 0, st>>>(pa);
    return hipGetLastError();
}

}  // namespace dm
