// dm_route_batch: batched dual-mapping routing (Sec. 3.2; Sec. A.1.1).
//
// Stage 0 (block_starts): exclusive sum of full blocks per request -> where
//   each request's block keys live.
// Stage 1 (hash_kernel): one wave per request walks the prompt 64 blocks at
//   a time, lane l owning block l of the chunk:
//     - NH digest of its block from B/4 16-byte loads;
//     - the affine chain H[b] = H[b-1] P + NH(b) for all 64 lanes at once:
//       with Q = P^-1 mod 2^64, H[c+l] = P^(l+1) (G + sum_{k<=l} NH(c+k)
//       Q^(k+1)), G carrying H of the previous chunk -- a wave prefix sum of
//       u64 instead of a serial chain;
//     - block key mix64(H xor seed), stored for every full block;
//     - in the first chunk the f2 chain over the first K blocks (one wave
//       sum) gives the second ring key.
// Stage 2 (lookup_kernel): one thread per request: owners on both rings,
//   distinct-candidate adjustment.
// Stage 3 (probe_kernel): longest cached prefix, first miss exact.  Every
//   lane of a persistent grid walks its own (request, candidate) key
//   sequence, one 64-byte bucket per probe, so hundreds of thousands of
//   independent probe chains hide the latency of each; no probe past the
//   first miss is issued.
// Stage 4 (select_kernel): the SLO-aware choice in request order.  One wave
//   holds the loads in registers (lane l keeps slot 64k + l in bank k); per
//   request only readlanes, three compares and one writelane sit on the
//   serial path.  Everything that does not depend on the loads (uncached
//   tokens, the SLO threshold on the cache-affine candidate's load) is
//   computed 64 requests at a time in parallel lanes beforehand, and the
//   outputs (TTFT, flags) afterwards from the recorded pre-update loads.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kRouteThreads = 256;
constexpr int kKeySlot = 4;  // scratch for block keys when the caller keeps none
constexpr int kSelSlot = 3;  // selection records
constexpr int kSplitSlot = 1;  // first request of each probing wave
constexpr uint64_t kProbeWaves = 16384;  // ~2 rounds of 256 CUs x 4 SIMDs x 8 waves

typedef int v4i __attribute__((ext_vector_type(4), aligned(4)));
typedef unsigned long long v2u64 __attribute__((ext_vector_type(2), aligned(16)));

// NH over the B tokens at p (4-byte aligned) with key words kk.
template <int B>
__device__ __forceinline__ uint64_t nh_block(const int32_t* p, const uint32_t* kk)
{
    uint64_t acc = 0;
#pragma unroll
    for (int j = 0; j < B; j += 4) {
        const v4i v = *reinterpret_cast<const v4i*>(p + j);
        acc += (uint64_t)((uint32_t)v.x + kk[j]) * (uint32_t)((uint32_t)v.y + kk[j + 1]);
        acc += (uint64_t)((uint32_t)v.z + kk[j + 2]) * (uint32_t)((uint32_t)v.w + kk[j + 3]);
    }
    return acc;
}

template <int B>
__device__ __forceinline__ void nh_block2(const int32_t* p, const uint32_t* k1, const uint32_t* k2,
                                          uint64_t& a1, uint64_t& a2)
{
    a1 = 0;
    a2 = 0;
#pragma unroll
    for (int j = 0; j < B; j += 4) {
        const v4i v = *reinterpret_cast<const v4i*>(p + j);
        a1 += (uint64_t)((uint32_t)v.x + k1[j]) * (uint32_t)((uint32_t)v.y + k1[j + 1]);
        a1 += (uint64_t)((uint32_t)v.z + k1[j + 2]) * (uint32_t)((uint32_t)v.w + k1[j + 3]);
        a2 += (uint64_t)((uint32_t)v.x + k2[j]) * (uint32_t)((uint32_t)v.y + k2[j + 1]);
        a2 += (uint64_t)((uint32_t)v.z + k2[j + 2]) * (uint32_t)((uint32_t)v.w + k2[j + 3]);
    }
}

struct HashArgs {
    const int32_t* tokens;
    const int64_t* offsets;
    uint64_t n;
    const HashParams* hp;
    uint32_t key_blocks;
    const uint64_t* bstart;  // [n+1]
    uint64_t* hkeys;         // [bstart[n]] f1 block keys
    uint64_t* key_out;       // [2n]
    uint32_t* status;
};

template <int B>
__global__ __launch_bounds__(kRouteThreads) void hash_kernel(HashArgs a)
{
    const int lane = lane_id();
    const uint64_t gw = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0], seed2 = hp->seed[1];
    const uint64_t H01 = hp->H0[0], H02 = hp->H0[1];
    const uint64_t q1 = hp->qpow[0][lane], p1 = hp->ppow[0][lane], q2 = hp->qpow[1][lane];
    uint32_t k1[B], k2[B];
#pragma unroll
    for (int j = 0; j < B; j++) {
        k1[j] = hp->kk[0][j];
        k2[j] = hp->kk[1][j];
    }
    for (uint64_t r = gw; r < a.n; r += nw) {
        const int64_t o0 = a.offsets[r], len = a.offsets[r + 1] - o0;
        if (o0 < 0 || len < 0) {
            if (lane == 0) {
                atomicOr(a.status, kErrInval);
                a.key_out[r] = 0;
                a.key_out[a.n + r] = 0;
            }
            continue;
        }
        const uint64_t nfull = (uint64_t)len / B;
        const uint32_t kr = (uint32_t)(nfull < a.key_blocks ? nfull : a.key_blocks);
        const int32_t* tp = a.tokens + o0;
        uint64_t* hk = a.hkeys + a.bstart[r];
        uint64_t x1 = mix64(H01 ^ seed1), x2 = mix64(H02 ^ seed2);  // empty-prefix keys
        uint64_t G = H01;
        for (uint64_t cb = 0; cb < nfull; cb += kWave) {
            const uint64_t b = cb + lane;
            const bool valid = b < nfull;
            uint64_t nh1 = 0, nh2 = 0;
            if (cb == 0) {
                if (valid)
                    nh_block2<B>(tp + b * B, k1, k2, nh1, nh2);
            } else if (valid) {
                nh1 = nh_block<B>(tp + b * B, k1);
            }
            const uint64_t S = wave_incl_sum_u64(nh1 * q1, lane);
            const uint64_t H = (G + S) * p1;
            const uint64_t h = mix64(H ^ seed1);
            if (valid)
                hk[b] = h;
            G = readlane_u64(H, kWave - 1);
            if (cb == 0) {
                x1 = readlane_u64(h, (int)kr - 1);
                const uint64_t S2 = wave_sum_u64(lane < (int)kr ? nh2 * q2 : 0);
                x2 = mix64(((H02 + S2) * hp->ppow[1][kr - 1]) ^ seed2);
            }
        }
        if (lane == 0) {
            a.key_out[r] = x1;
            a.key_out[a.n + r] = x2;
        }
    }
}

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
__global__ __launch_bounds__(kRouteThreads) void probe_kernel(ProbeArgs a)
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

// Shared by both selection kernels: the SLO-aware rule given the two
// candidates' pre-update loads.  kind bit0 = equal match, bit1 = c1 is the
// cache-affine candidate; th = the affine candidate's load below which its
// TTFT meets the SLO.
__device__ __forceinline__ bool pick_first(uint32_t kind, int64_t L1, int64_t L2, int64_t th)
{
    if (kind & 1)
        return L1 <= L2;
    if (kind & 2)
        return L1 < th || !(L2 < L1);
    return !(L2 < th || !(L1 < L2));
}

// Per-lane request record for the serial loop and the output epilogue.
struct SelRec {
    uint32_t c1, c2, kind;
    int64_t u1, u2, th;
};

__device__ __forceinline__ SelRec load_rec(const int64_t* offsets, uint64_t n, uint64_t r, bool ok,
                                           uint32_t bshift, const uint32_t* cand,
                                           const uint32_t* match, int64_t base, int64_t per,
                                           uint32_t qshift, int64_t slo)
{
    SelRec s;
    s.c1 = ok ? cand[r] : 0;
    s.c2 = ok ? cand[n + r] : 0;
    const uint32_t m1 = ok ? match[r] : 0, m2 = ok ? match[n + r] : 0;
    const int64_t len = ok ? offsets[r + 1] - offsets[r] : 0;
    s.u1 = len - ((int64_t)m1 << bshift);
    s.u2 = len - ((int64_t)m2 << bshift);
    const bool eq = m1 == m2, aff1 = m1 > m2;
    // T_a <= slo  <=>  floor(L_a / 2^q) <= slo - base - per*u_a  <=>  L_a < th
    s.th = (slo - base - per * (aff1 ? s.u1 : s.u2) + 1) * ((int64_t)1 << qshift);
    s.kind = (eq ? 1u : 0u) | (aff1 ? 2u : 0u);
    return s;
}

__device__ __forceinline__ void store_out(const SelRec& s, uint64_t r, int64_t L1, int64_t L2,
                                          uint8_t* flags, uint32_t* chosen, int64_t* ttft,
                                          int64_t base, int64_t per, uint32_t qshift, int64_t slo)
{
    const bool pick1 = pick_first(s.kind, L1, L2, s.th);
    const int64_t t1 = base + per * s.u1 + (L1 >> qshift);
    const int64_t t2 = base + per * s.u2 + (L2 >> qshift);
    uint32_t f = flags[r];
    if (t1 > slo && t2 > slo)
        f |= 2;
    if (s.kind & 1)
        f |= 4;
    else if (pick1 != ((s.kind & 2) != 0))
        f |= 1;
    chosen[r] = pick1 ? s.c1 : s.c2;
    ttft[r] = pick1 ? t1 : t2;
    flags[r] = (uint8_t)f;
}

// Serial SLO-aware selection, loads in R register banks of one wave.
template <int R>
__global__ __launch_bounds__(kWave) void select_kernel(
    const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
    const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
    uint8_t* __restrict__ flags, uint32_t* __restrict__ chosen, int64_t* __restrict__ ttft,
    int64_t* __restrict__ loads, uint32_t S, int64_t base, int64_t per, uint32_t qshift, int64_t slo,
    const uint32_t* __restrict__ plan)
{
    if (!plan[0])
        return;
    const int lane = lane_id();
    uint32_t Llo[R], Lhi[R];
#pragma unroll
    for (int k = 0; k < R; k++) {
        const uint32_t i = 64 * k + lane;
        const int64_t v = i < S ? loads[i] : 0;
        Llo[k] = (uint32_t)v;
        Lhi[k] = (uint32_t)((uint64_t)v >> 32);
    }
    auto get = [&](uint32_t c) -> int64_t {
        const uint32_t bank = c >> 6, l = c & 63;
        uint32_t lo = __builtin_amdgcn_readlane(Llo[0], l), hi = __builtin_amdgcn_readlane(Lhi[0], l);
#pragma unroll
        for (int k = 1; k < R; k++) {
            const uint32_t lo_k = __builtin_amdgcn_readlane(Llo[k], l);
            const uint32_t hi_k = __builtin_amdgcn_readlane(Lhi[k], l);
            lo = bank == (uint32_t)k ? lo_k : lo;
            hi = bank == (uint32_t)k ? hi_k : hi;
        }
        return (int64_t)(((uint64_t)hi << 32) | lo);
    };
    for (uint64_t r0 = 0; r0 < n; r0 += kWave) {
        const uint64_t r = r0 + lane;
        const bool ok = r < n;
        const SelRec s = load_rec(offsets, n, r, ok, bshift, cand, match, base, per, qshift, slo);
        int64_t myL1 = 0, myL2 = 0;
        const int cnt = (int)(n - r0 < (uint64_t)kWave ? n - r0 : kWave);
        for (int j = 0; j < cnt; j++) {
            const uint32_t C1 = __builtin_amdgcn_readlane(s.c1, j);
            const uint32_t C2 = __builtin_amdgcn_readlane(s.c2, j);
            const uint32_t K = __builtin_amdgcn_readlane(s.kind, j);
            const int64_t TH = (int64_t)readlane_u64((uint64_t)s.th, j);
            const int64_t U1 = (int64_t)readlane_u64((uint64_t)s.u1, j);
            const int64_t U2 = (int64_t)readlane_u64((uint64_t)s.u2, j);
            const int64_t L1 = get(C1), L2 = get(C2);
            const bool pick1 = pick_first(K, L1, L2, TH);
            const uint32_t ch = pick1 ? C1 : C2;
            const int64_t nv = (pick1 ? L1 : L2) + (pick1 ? U1 : U2);
            const uint32_t bank = ch >> 6, l = ch & 63;
            const bool mine = lane == (int)l;
#pragma unroll
            for (int k = 0; k < R; k++)
                if (bank == (uint32_t)k) {
                    Llo[k] = mine ? (uint32_t)nv : Llo[k];
                    Lhi[k] = mine ? (uint32_t)((uint64_t)nv >> 32) : Lhi[k];
                }
            if (lane == j) {
                myL1 = L1;
                myL2 = L2;
            }
        }
        if (ok)
            store_out(s, r, myL1, myL2, flags, chosen, ttft, base, per, qshift, slo);
    }
#pragma unroll
    for (int k = 0; k < R; k++) {
        const uint32_t i = 64 * k + lane;
        if (i < S)
            loads[i] = (int64_t)(((uint64_t)Lhi[k] << 32) | Llo[k]);
    }
}

// Same rule with loads in LDS, for slot spaces beyond the register banks.
__global__ __launch_bounds__(kWave) void select_lds_kernel(
    const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
    const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
    uint8_t* __restrict__ flags, uint32_t* __restrict__ chosen, int64_t* __restrict__ ttft,
    int64_t* __restrict__ loads, uint32_t S, int64_t base, int64_t per, uint32_t qshift, int64_t slo,
    const uint32_t* __restrict__ plan)
{
    if (!plan[0])
        return;
    __shared__ int64_t L[kMaxSlots];
    const int lane = lane_id();
    for (uint32_t i = lane; i < S; i += kWave)
        L[i] = loads[i];
    __syncthreads();
    for (uint64_t r0 = 0; r0 < n; r0 += kWave) {
        const uint64_t r = r0 + lane;
        const bool ok = r < n;
        const SelRec s = load_rec(offsets, n, r, ok, bshift, cand, match, base, per, qshift, slo);
        int64_t myL1 = 0, myL2 = 0;
        const int cnt = (int)(n - r0 < (uint64_t)kWave ? n - r0 : kWave);
        for (int j = 0; j < cnt; j++) {
            const uint32_t C1 = __builtin_amdgcn_readlane(s.c1, j);
            const uint32_t C2 = __builtin_amdgcn_readlane(s.c2, j);
            const uint32_t K = __builtin_amdgcn_readlane(s.kind, j);
            const int64_t TH = (int64_t)readlane_u64((uint64_t)s.th, j);
            const int64_t U1 = (int64_t)readlane_u64((uint64_t)s.u1, j);
            const int64_t U2 = (int64_t)readlane_u64((uint64_t)s.u2, j);
            const int64_t L1 = L[C1], L2 = L[C2];
            const bool pick1 = pick_first(K, L1, L2, TH);
            const uint32_t ch = pick1 ? C1 : C2;
            const int64_t nv = (pick1 ? L1 : L2) + (pick1 ? U1 : U2);
            __syncthreads();
            if (lane == 0)
                L[ch] = nv;
            __syncthreads();
            if (lane == j) {
                myL1 = L1;
                myL2 = L2;
            }
        }
        if (ok)
            store_out(s, r, myL1, myL2, flags, chosen, ttft, base, per, qshift, slo);
    }
    __syncthreads();
    for (uint32_t i = lane; i < S; i += kWave)
        loads[i] = L[i];
}

// ---------------------------------------------------------------------------
// Fast selection path.  When every load stays within 2^31 - 1 of the batch's
// smallest live load (checked on the device), the serial loop runs on 32-bit
// loads relative to that base, over dense live-instance indices (lane l of
// bank k holds live instance 64k + l).  Records are packed by a parallel
// kernel and fetched with scalar loads; the loop records each request's two
// pre-update loads and a parallel epilogue derives chosen, TTFT and flags.
// ---------------------------------------------------------------------------

struct SelPack {
    uint32_t w;    // d1 | d2 << 12 | kind << 24 (dense candidate indices)
    uint32_t u1;   // uncached tokens on c1
    uint32_t u2;   // uncached tokens on c2
    int32_t th;    // affine candidate's relative load bound (clamped)
};

// plan[0] = 1 for the 64-bit path; plan[1] = 1 for the 32-bit path.
// base[0] = smallest live load; grow[d] bounds how much live instance d's
// load can grow in this batch (the larger uncached count of every request
// that has it as a candidate).
__global__ __launch_bounds__(256) void sel_base_kernel(const int64_t* __restrict__ loads,
                                                       const uint32_t* __restrict__ live_ids,
                                                       uint32_t n_live, int64_t* __restrict__ base,
                                                       unsigned long long* __restrict__ grow)
{
    __shared__ int64_t smin[256];
    int64_t mn = INT64_MAX;
    for (uint32_t k = threadIdx.x; k < n_live; k += blockDim.x) {
        const int64_t v = loads[live_ids[k]];
        mn = v < mn ? v : mn;
        grow[k] = 0;
    }
    smin[threadIdx.x] = mn;
    __syncthreads();
    for (int d = 128; d > 0; d >>= 1) {
        if (threadIdx.x < d)
            smin[threadIdx.x] = std::min(smin[threadIdx.x], smin[threadIdx.x + d]);
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        base[0] = smin[0];
        grow[kMaxSlots] = 0;  // set if some record does not fit 32 bits
    }
}

constexpr uint32_t kFastMaxLive = 256;

__global__ __launch_bounds__(256) void sel_prep_kernel(
    const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
    const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
    const uint32_t* __restrict__ dense, uint32_t n_live, const int64_t* __restrict__ base,
    int64_t tbase, int64_t per, uint32_t qshift, int64_t slo, SelPack* __restrict__ rec,
    unsigned long long* __restrict__ grow)
{
    __shared__ unsigned long long sg[kFastMaxLive];
    const bool track = n_live <= kFastMaxLive;
    if (track)
        for (uint32_t k = threadIdx.x; k < n_live; k += blockDim.x)
            sg[k] = 0;
    __syncthreads();
    const int64_t b0 = base[0];
    unsigned long long bad = 0;
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t m1 = match[r], m2 = match[n + r];
        const int64_t len = offsets[r + 1] - offsets[r];
        const int64_t u1 = len - ((int64_t)m1 << bshift), u2 = len - ((int64_t)m2 << bshift);
        const bool eq = m1 == m2, aff1 = m1 > m2;
        const int64_t th = (slo - tbase - per * (aff1 ? u1 : u2) + 1) * ((int64_t)1 << qshift);
        int64_t thr = th - b0;  // relative loads are in [0, 2^31 - 1): clamp the bound
        thr = thr < -1 ? -1 : (thr > INT32_MAX ? INT32_MAX : thr);
        const uint32_t d1 = dense[cand[r]], d2 = dense[cand[n + r]];
        SelPack p;
        p.w = d1 | (d2 << 12) | ((eq ? 1u : 0u) << 24) | ((aff1 ? 1u : 0u) << 25);
        p.u1 = (uint32_t)u1;
        p.u2 = (uint32_t)u2;
        p.th = (int32_t)thr;
        rec[r] = p;
        const bool ok = u1 >= 0 && u2 >= 0 && u1 <= INT32_MAX && u2 <= INT32_MAX;
        bad |= ok ? 0ull : 1ull;
        if (track && ok) {
            const unsigned long long g = (unsigned long long)(u1 > u2 ? u1 : u2);
            atomicAdd(&sg[d1], g);
            if (d2 != d1)
                atomicAdd(&sg[d2], g);
        }
    }
    __syncthreads();
    if (track)
        for (uint32_t k = threadIdx.x; k < n_live; k += blockDim.x)
            if (sg[k])
                atomicAdd(&grow[k], sg[k]);
    if (bad)
        atomicOr(&grow[kMaxSlots], 1ull);
}

// Fast path iff n_live fits the register banks and every live load stays
// below base + 2^31 - 1 whatever the decisions.
__global__ __launch_bounds__(256) void sel_plan_kernel(const int64_t* __restrict__ loads,
                                                       const uint32_t* __restrict__ live_ids,
                                                       uint32_t n_live,
                                                       const int64_t* __restrict__ base,
                                                       const unsigned long long* __restrict__ grow,
                                                       uint32_t* __restrict__ plan)
{
    __shared__ int ok_all;
    if (threadIdx.x == 0)
        ok_all = n_live <= kFastMaxLive && grow[kMaxSlots] == 0;
    __syncthreads();
    for (uint32_t k = threadIdx.x; k < n_live && k < kFastMaxLive; k += blockDim.x) {
        const unsigned long long span = (unsigned long long)(loads[live_ids[k]] - base[0]);
        if (span >= (1ull << 30) || grow[k] >= (1ull << 30))
            atomicAnd(&ok_all, 0);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        plan[0] = ok_all ? 0 : 1;
        plan[1] = ok_all ? 1 : 0;
    }
}

template <int R>
__device__ __forceinline__ void fast_step(const SelPack& p, int32_t (&L)[R], int lane, int at,
                                          int32_t& rec1, int32_t& rec2)
{
    const uint32_t d1 = p.w & 0xFFF, d2 = (p.w >> 12) & 0xFFF;
    const uint32_t l1 = d1 & 63, l2 = d2 & 63, k1 = d1 >> 6, k2 = d2 >> 6;
    int32_t L1 = __builtin_amdgcn_readlane(L[0], l1);
    int32_t L2 = __builtin_amdgcn_readlane(L[0], l2);
#pragma unroll
    for (int k = 1; k < R; k++) {
        const int32_t a = __builtin_amdgcn_readlane(L[k], l1);
        const int32_t b = __builtin_amdgcn_readlane(L[k], l2);
        L1 = k1 == (uint32_t)k ? a : L1;
        L2 = k2 == (uint32_t)k ? b : L2;
    }
    // equal: L1 <= L2; c1 affine: L1 < th or L2 >= L1; c2 affine: L2 >= th and L1 < L2
    const uint32_t eq = (p.w >> 24) & 1, a1 = (p.w >> 25) & 1;
    const uint32_t le12 = L1 <= L2, lt12 = L1 < L2;
    const uint32_t lt1t = L1 < p.th, ge2t = L2 >= p.th;
    const uint32_t pick1 = (eq & le12) | ((eq ^ 1) & a1 & (lt1t | le12)) |
                           ((eq ^ 1) & (a1 ^ 1) & ge2t & lt12);
    const int32_t nv = pick1 ? L1 + (int32_t)p.u1 : L2 + (int32_t)p.u2;
    const uint32_t lc = pick1 ? l1 : l2, kc = pick1 ? k1 : k2;
    const bool mine = lane == (int)lc;
#pragma unroll
    for (int k = 0; k < R; k++)
        L[k] = (mine && kc == (uint32_t)k) ? nv : L[k];
    const bool here = lane == at;
    rec1 = here ? L1 : rec1;
    rec2 = here ? L2 : rec2;
}

constexpr int kFastUnroll = 8;  // record padding past n (prefetch never reads beyond n)

// Requests of a 64-request window that share no candidate commute: neither
// can read an instance the other may write.  So each window runs in
// dependency levels: lane j waits only for the earlier lanes of its window
// whose candidates overlap its own (a mask built from per-instance lane
// bitmaps), and every step runs all lanes whose such predecessors are done,
// in parallel, on loads kept in LDS.  The result equals request-order
// processing; the lowest unfinished lane is always ready, so every step
// makes progress.
template <int R>
__global__ __launch_bounds__(kWave) void select_fast_kernel(
    const SelPack* __restrict__ rec, uint64_t n, const uint32_t* __restrict__ live_ids,
    uint32_t n_live, int64_t* __restrict__ loads, const uint32_t* __restrict__ plan,
    const int64_t* __restrict__ base, int2* __restrict__ lpre)
{
    if (!plan[1])
        return;
    __shared__ int32_t L[kFastMaxLive];
    __shared__ unsigned long long M[kFastMaxLive];
    const int lane = lane_id();
    const uint64_t bit = 1ull << lane, lt = bit - 1;
    const int64_t b0 = base[0];
    for (uint32_t d = lane; d < kFastMaxLive; d += kWave) {
        L[d] = d < n_live ? (int32_t)(loads[live_ids[d]] - b0) : 0;
        M[d] = 0;
    }
    __syncthreads();
    SelPack mine = rec[lane < n ? lane : 0];
    for (uint64_t r0 = 0; r0 < n; r0 += kWave) {
        const uint64_t ni = r0 + kWave + lane;
        const SelPack nxt = rec[ni < n ? ni : 0];
        const bool valid = r0 + lane < n;
        const uint32_t d1 = mine.w & 0xFFF, d2 = (mine.w >> 12) & 0xFFF;
        if (valid) {
            atomicOr(&M[d1], bit);
            atomicOr(&M[d2], bit);
        }
        __syncthreads();
        const uint64_t wait = valid ? ((M[d1] | M[d2]) & lt) : 0;
        __syncthreads();
        if (valid) {
            M[d1] = 0;
            M[d2] = 0;
        }
        const uint32_t eq = (mine.w >> 24) & 1, a1 = (mine.w >> 25) & 1;
        uint64_t done = ~ballot(valid);
        int32_t L1v = 0, L2v = 0;
        while (done != ~0ull) {
            const bool ready = !(done & bit) && (wait & ~done) == 0;
            if (ready) {
                const int32_t L1 = L[d1], L2 = L[d2];
                // equal: L1 <= L2; c1 affine: L1 < th or L2 >= L1;
                // c2 affine: L2 >= th and L1 < L2
                const uint32_t le12 = L1 <= L2, lt12 = L1 < L2;
                const uint32_t lt1t = L1 < mine.th, ge2t = L2 >= mine.th;
                const uint32_t pick1 = (eq & le12) | ((eq ^ 1) & a1 & (lt1t | le12)) |
                                       ((eq ^ 1) & (a1 ^ 1) & ge2t & lt12);
                L[pick1 ? d1 : d2] = pick1 ? L1 + (int32_t)mine.u1 : L2 + (int32_t)mine.u2;
                L1v = L1;
                L2v = L2;
            }
            done |= ballot(ready);
        }
        if (valid)
            lpre[r0 + lane] = make_int2(L1v, L2v);
        __syncthreads();
        mine = nxt;
    }
    for (uint32_t d = lane; d < n_live && d < kFastMaxLive; d += kWave)
        loads[live_ids[d]] = b0 + L[d];
}

__global__ void sel_out_kernel(const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
                               const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
                               const int2* __restrict__ lpre, const int64_t* __restrict__ base,
                               const uint32_t* __restrict__ plan, uint8_t* __restrict__ flags,
                               uint32_t* __restrict__ chosen, int64_t* __restrict__ ttft,
                               int64_t tbase, int64_t per, uint32_t qshift, int64_t slo)
{
    if (!plan[1])
        return;
    const int64_t b0 = base[0];
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        SelRec s = load_rec(offsets, n, r, true, bshift, cand, match, tbase, per, qshift, slo);
        const int2 lp = lpre[r];
        store_out(s, r, b0 + lp.x, b0 + lp.y, flags, chosen, ttft, tbase, per, qshift, slo);
    }
}

template <int B>
void launch_hash(const HashArgs& a, uint32_t grid, hipStream_t s)
{
    hash_kernel<B><<<grid, kRouteThreads, 0, s>>>(a);
}

template <int R>
void launch_select(dm_ctx* c, const int64_t* offsets, uint64_t n, uint32_t bshift,
                   const dm_route_out* out, int64_t* loads, const uint32_t* plan)
{
    const dm_config& k = c->cfg;
    select_kernel<R><<<1, kWave, 0, c->stream>>>(offsets, n, bshift, out->cand, out->match,
                                                 out->flags, out->chosen, out->ttft_us, loads,
                                                 k.max_slots, k.ttft_base_us, k.ttft_per_token_us,
                                                 c->shift_div, k.slo_us, plan);
}

template <int R>
void launch_fast(dm_ctx* c, const SelPack* rec, uint64_t n, int64_t* loads, const uint32_t* plan,
                 const int64_t* base, int2* lpre)
{
    select_fast_kernel<R><<<1, kWave, 0, c->stream>>>(rec, n, c->d_live_ids, c->n_live, loads,
                                                      plan, base, lpre);
}

uint32_t grid_for(uint64_t n, int threads, uint32_t cap)
{
    uint64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    return (uint32_t)(g > cap ? cap : g);
}

}  // namespace

hipError_t route(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                 int64_t* loads, const dm_route_out* out)
{
    hipError_t e = hipSuccess;
    hipStream_t st = c->stream;
    if (c->timing && (e = hipEventRecord(c->ev[0], st)) != hipSuccess)
        return e;
    uint64_t* bstart = static_cast<uint64_t*>(scratch_get(c, 0, (n + 1) * sizeof(uint64_t), &e));
    if (!bstart)
        return e;
    if ((e = block_starts(c, offsets, n, bstart)) != hipSuccess)
        return e;
    uint64_t* hkeys = out->block_keys;
    if (!hkeys) {
        // block keys go to context scratch sized by the batch's full-block count
        uint64_t total = 0;
        if ((e = hipMemcpyAsync(&total, bstart + n, sizeof(uint64_t), hipMemcpyDeviceToHost, st)) !=
                hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess)
            return e;
        hkeys = static_cast<uint64_t*>(scratch_get(c, kKeySlot, (total + 1) * sizeof(uint64_t), &e));
        if (!hkeys)
            return e;
    }
    if (c->timing && (e = hipEventRecord(c->ev[1], st)) != hipSuccess)
        return e;
    HashArgs ha{tokens, offsets, n, c->d_hp, c->cfg.key_blocks, bstart, hkeys, out->key,
                c->d_status};
    const uint32_t hgrid = grid_for(n, kRouteThreads / kWave, 1u << 20);
    switch (c->cfg.block_size) {
        case 4: launch_hash<4>(ha, hgrid, st); break;
        case 8: launch_hash<8>(ha, hgrid, st); break;
        case 16: launch_hash<16>(ha, hgrid, st); break;
        case 32: launch_hash<32>(ha, hgrid, st); break;
        case 64: launch_hash<64>(ha, hgrid, st); break;
        default: return hipErrorInvalidValue;
    }
    if (c->timing && (e = hipEventRecord(c->ev[2], st)) != hipSuccess)
        return e;
    lookup_kernel<<<grid_for(n, 256, 8192), 256, 0, st>>>(
        n, out->key, view(c->ring[c->cur][0]), view(c->ring[c->cur][1]), c->d_next_live, c->n_live,
        out->cand, out->flags);
    // probe waves: request ranges balanced by full blocks
    const uint64_t pw = std::min<uint64_t>(n, kProbeWaves);
    const uint32_t pgrid = (uint32_t)((pw + kRouteThreads / kWave - 1) / (kRouteThreads / kWave));
    const uint32_t W = pgrid * (kRouteThreads / kWave);
    uint32_t* first =
        static_cast<uint32_t*>(scratch_get(c, kSplitSlot, (W + 1) * sizeof(uint32_t), &e));
    if (!first)
        return e;
    fill_first_kernel<<<grid_for(W + 1, 256, 1024), 256, 0, st>>>(first, W, (uint32_t)n);
    wave_split_kernel<<<grid_for(n + 1, 256, 8192), 256, 0, st>>>(bstart, n, W, first);
    ProbeArgs pa{hkeys, bstart, n, out->cand, c->d_tables, c->cfg.index_log2_slots, out->match,
                 first};
    probe_kernel<<<pgrid, kRouteThreads, 0, st>>>(pa);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (c->timing && (e = hipEventRecord(c->ev[3], st)) != hipSuccess)
        return e;
    uint32_t bshift = 0;
    while ((1u << bshift) < c->cfg.block_size)
        bshift++;
    const uint32_t S = c->cfg.max_slots;
    const dm_config& k = c->cfg;
    // selection work arrays: records, pre-update loads, base/plan words
    const uint64_t nrec = n + 2 * kFastUnroll;  // padding read by the loop's prefetch
    const size_t tail_bytes = 256 + (kMaxSlots + 1) * sizeof(unsigned long long);
    uint8_t* sw = static_cast<uint8_t*>(scratch_get(
        c, kSelSlot, nrec * sizeof(SelPack) + n * sizeof(int2) + tail_bytes + 256, &e));
    if (!sw)
        return e;
    SelPack* rec = reinterpret_cast<SelPack*>(sw);
    int2* lpre = reinterpret_cast<int2*>(sw + nrec * sizeof(SelPack));
    uint8_t* tail = sw + ((nrec * sizeof(SelPack) + n * sizeof(int2) + 255) & ~size_t(255));
    int64_t* base = reinterpret_cast<int64_t*>(tail);
    uint32_t* plan = reinterpret_cast<uint32_t*>(tail + 128);
    unsigned long long* grow = reinterpret_cast<unsigned long long*>(tail + 256);
    const uint32_t NL = c->n_live;
    sel_base_kernel<<<1, 256, 0, st>>>(loads, c->d_live_ids, NL, base, grow);
    sel_prep_kernel<<<grid_for(n, 256, 4096), 256, 0, st>>>(
        offsets, n, bshift, out->cand, out->match, c->d_dense, NL, base, k.ttft_base_us,
        k.ttft_per_token_us, c->shift_div, k.slo_us, rec, grow);
    sel_plan_kernel<<<1, 256, 0, st>>>(loads, c->d_live_ids, NL, base, grow, plan);
    if (NL <= 64)
        launch_fast<1>(c, rec, n, loads, plan, base, lpre);
    else if (NL <= 128)
        launch_fast<2>(c, rec, n, loads, plan, base, lpre);
    else if (NL <= 192)
        launch_fast<3>(c, rec, n, loads, plan, base, lpre);
    else if (NL <= kFastMaxLive)
        launch_fast<4>(c, rec, n, loads, plan, base, lpre);
    sel_out_kernel<<<grid_for(n, 256, 8192), 256, 0, st>>>(
        offsets, n, bshift, out->cand, out->match, lpre, base, plan, out->flags, out->chosen,
        out->ttft_us, k.ttft_base_us, k.ttft_per_token_us, c->shift_div, k.slo_us);
    if (S <= 64)
        launch_select<1>(c, offsets, n, bshift, out, loads, plan);
    else if (S <= 128)
        launch_select<2>(c, offsets, n, bshift, out, loads, plan);
    else if (S <= 192)
        launch_select<3>(c, offsets, n, bshift, out, loads, plan);
    else if (S <= 256)
        launch_select<4>(c, offsets, n, bshift, out, loads, plan);
    else
        select_lds_kernel<<<1, kWave, 0, st>>>(offsets, n, bshift, out->cand, out->match,
                                               out->flags, out->chosen, out->ttft_us, loads, S,
                                               k.ttft_base_us, k.ttft_per_token_us, c->shift_div,
                                               k.slo_us, plan);
    e = hipGetLastError();
    if (e == hipSuccess && c->timing)
        e = hipEventRecord(c->ev[4], st);
    return e;
}

}  // namespace dm
