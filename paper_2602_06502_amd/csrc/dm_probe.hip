// Candidates and longest cached prefixes (Sec. 3.2; Sec. A.1.1).
//
// lookup_kernel: one thread per request finds the owners of its two ring
//   keys and applies the distinct-candidate adjustment.
// probe_kernel: the longest cached prefix on each candidate, first miss
//   exact.  Every lane of a persistent grid walks its own (request,
//   candidate) key sequence, one 64-byte bucket per probe, so hundreds of
//   thousands of independent probe chains hide the latency of each; no
//   probe past the first miss is issued.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kSplitSlot = 1;            // first request of each probing wave
constexpr uint64_t kProbeWaves = 16384;  // ~2 rounds of 256 CUs x 4 SIMDs x 8 waves

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

// first[w] = first request of wave w, splitting requests so that every wave
// gets about the same share of pre[n] - pre[0] (pre: a non-decreasing prefix
// array with n + 1 entries); first[W] = n.
__global__ void fill_first_kernel(uint32_t* first, uint32_t W, uint32_t v)
{
    for (uint32_t w = blockIdx.x * blockDim.x + threadIdx.x; w <= W; w += gridDim.x * blockDim.x)
        first[w] = v;
}

__global__ void wave_split_kernel(const uint64_t* __restrict__ pre, uint64_t n, uint32_t W,
                                  uint32_t* __restrict__ first)
{
    const uint64_t lo = pre[0], span = pre[n] - pre[0];
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r <= n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        auto owner = [&](uint64_t q) -> uint64_t {
            if (q >= n)
                return W;
            const uint64_t rel = pre[q] - lo;
            if (span == 0 || rel == 0)
                return 0;
            const uint64_t w = (uint64_t)(((unsigned __int128)rel * W) / span);
            return w < W ? w : W - 1;
        };
        const uint64_t wl = r == 0 ? 0 : owner(r - 1) + 1, wh = owner(r);
        for (uint64_t w = wl; w <= wh && w <= W; w++)
            first[w] = (uint32_t)r;
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
    const uint32_t* first;  // [W + 1] request range of each wave, balanced by blocks
};

// Longest cached prefix of every (request, candidate) task, first miss exact.
// Wave w owns the tasks of requests [first[w], first[w+1]); every lane keeps
// a current task and a prefetched next one taken from the wave's task
// counter (advanced with a ballot), so a finished lane switches to work
// whose block range, table and first key are already loaded while the
// wave keeps probing.  Each probe reads one 64-byte bucket while the next
// block key is already being fetched.
__global__ __launch_bounds__(kProbeThreads) void probe_kernel(ProbeArgs a)
{
    const int lane = lane_id();
    const uint64_t lt_mask = lane ? (~0ull >> (64 - lane)) : 0ull;
    const uint64_t gw = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const uint64_t rb = a.first[gw], re = a.first[gw + 1] < a.n ? a.first[gw + 1] : a.n;
    const uint64_t T = re > rb ? 2 * (re - rb) : 0;
    const uint64_t nbk = 1ull << (a.log2slots - 3);
    uint64_t next = 0;  // wave-uniform: next unassigned task of this wave
    // current task
    bool have = false;
    uint64_t kb = 0, ke = 0, k0 = 0, key = 0, nkey = 0, bkt = 0, steps = 0, out = 0;
    const uint64_t* tab = a.tables;
    // prefetched task: stage 0 none, 1 range/table loaded, 2 first key loaded
    int pst = 0;
    uint64_t pk0 = 0, pke = 0, pout = 0, pkey = 0;
    const uint64_t* ptab = a.tables;
    for (;;) {
        // advance the prefetched task one stage (its loads land during the probe below)
        if (pst == 1) {
            if (pke == pk0) {
                a.match[pout] = 0;  // no full block: done without probing
                pst = 0;
            } else {
                pkey = a.hkeys[pk0];
                pst = 2;
            }
        }
        const uint64_t need = ballot(pst == 0);
        if (need && next < T) {
            const uint64_t t = next + __popcll(need & lt_mask);
            next += __popcll(need);
            if (pst == 0 && t < T) {
                const uint64_t r = rb + (t >> 1);
                pout = (t & 1) * a.n + r;
                pk0 = a.bstart[r];
                pke = a.bstart[r + 1];
                ptab = a.tables + ((uint64_t)a.cand[pout] << a.log2slots);
                pst = 1;
            }
        }
        // an idle lane takes its prefetched task
        if (!have && pst == 2) {
            k0 = pk0;
            kb = pk0;
            ke = pke;
            out = pout;
            tab = ptab;
            key = canon_key(pkey);
            bkt = home_bucket(key, a.log2slots);
            steps = 0;
            have = true;
            pst = 0;
        }
        if (!__any(have)) {
            if (next >= T && !__any(pst != 0))
                break;
            continue;
        }
        if (have) {
            const v2u64* line = reinterpret_cast<const v2u64*>(tab + bkt * kBucket);
            const v2u64 s0 = line[0], s1 = line[1], s2 = line[2], s3 = line[3];
            if (kb + 1 < ke)
                nkey = a.hkeys[kb + 1];
            const bool hit = s0.x == key || s0.y == key || s1.x == key || s1.y == key ||
                             s2.x == key || s2.y == key || s3.x == key || s3.y == key;
            const bool empty = s0.x == kEmpty || s0.y == kEmpty || s1.x == kEmpty ||
                               s1.y == kEmpty || s2.x == kEmpty || s2.y == kEmpty ||
                               s3.x == kEmpty || s3.y == kEmpty;
            if (hit) {
                kb++;
                if (kb == ke) {
                    a.match[out] = (uint32_t)(kb - k0);
                    have = false;
                } else {
                    key = canon_key(nkey);
                    bkt = home_bucket(key, a.log2slots);
                    steps = 0;
                }
            } else if (empty || ++steps >= nbk) {
                a.match[out] = (uint32_t)(kb - k0);  // first miss (or scanned the whole table)
                have = false;
            } else {
                bkt = (bkt + 1) & (nbk - 1);
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
    // probe waves: request ranges balanced by full blocks
    const uint64_t pw = std::min<uint64_t>(n, kProbeWaves);
    const uint32_t wpb = kProbeThreads / kWave;
    const uint32_t pgrid = (uint32_t)((pw + wpb - 1) / wpb);
    const uint32_t W = pgrid * wpb;
    uint32_t* first =
        static_cast<uint32_t*>(scratch_get(c, kSplitSlot, (W + 1) * sizeof(uint32_t), &e));
    if (!first)
        return e;
    fill_first_kernel<<<grid_for(W + 1, 256, 1024), 256, 0, st>>>(first, W, (uint32_t)n);
    wave_split_kernel<<<grid_for(n + 1, 256, 8192), 256, 0, st>>>(bstart, n, W, first);
    ProbeArgs pa{hkeys, bstart, n, cand, c->d_tables, c->cfg.index_log2_slots, match, first};
    probe_kernel<<<pgrid, kProbeThreads, 0, st>>>(pa);
    return hipGetLastError();
}

}  // namespace dm
