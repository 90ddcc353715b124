// SLO-aware candidate selection in request order (Sec. 3.2).
//
// Every request takes its cache-affine candidate unless that candidate's
// TTFT misses the SLO and the other one is less loaded (equal matches: the
// less loaded, first candidate on ties); the chosen instance's load grows by
// the request's uncached tokens before the next request is decided.  The
// batch result is therefore defined by processing the requests one by one.
// The single-criterion rules of the ablation study (Sec. 4.3) run on the same
// machinery: cache affinity is the SLO-aware rule with an unbounded TTFT
// budget, least load is the equal-match rule for every request (both take
// the fast path), and minimum TTFT compares the two estimates (serial path).
//
// Fast path (at most 256 live instances, uncached counts within 32 bits,
// live loads within 2^62 of the smallest; checked on the device), on 32-bit
// absolute loads when every load stays below 2^31, else on 64-bit loads
// relative to the smallest:
//   sel_prep_kernel   one thread per request packs a 16-byte record: the
//                     affine candidate a and the other o (dense indices),
//                     their uncached tokens, and th such that the rule reads
//                     "take a iff L_a <= max(th, L_o)" (clamped to 32 bits;
//                     the 64-bit walk recomputes it exactly);
//   sel_level_kernel  one wave per block of requests (1024, or 2048 in
//                     batches of at least 512 Ki requests): the dependency
//                     level of every request inside its block (runs of up
//                     to three same-pair requests sharing a level), and the
//                     packing of whole levels into windows of two sets of
//                     64 lanes (one set for the window's even depths, one
//                     for its odd ones);
//   sel_scan_kernel,  the windows' places, the walk records of every lane
//   sel_fill_kernel   of both sets of every window and each request's slot;
//   select_fast_kernel one wave walks the windows in order and, inside a
//                     window, the levels in order: requests of one level
//                     share no instance, so they run together on loads kept
//                     in LDS, and each sees exactly the loads that the
//                     request-order walk would show it;
//   sel_out_kernel    chosen instance, TTFT and flags of every request from
//                     its recorded pre-update loads, in parallel.
// Slow path: the same rule, one request at a time, on 64-bit loads in
// registers (at most 256 slots) or in LDS.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kSelSlot = kSlotSelect;  // selection work arrays

// Shared by every selection kernel: the rule given the two candidates'
// pre-update loads.  kind bit0 = compare the loads (equal match, or the
// least-load rule), bit1 = c1 is the cache-affine candidate, bit2 = compare
// the TTFT estimates, bit3 = keep the cache-affine candidate whatever its
// TTFT; th = the affine candidate's load below which its TTFT meets the SLO,
// or for bit2 per * (u2 - u1), so that t1 <= t2 reads
// floor(L1 / 2^q) - floor(L2 / 2^q) <= th.
__device__ __forceinline__ bool pick_first(uint32_t kind, int64_t L1, int64_t L2, int64_t th,
                                           uint32_t qshift)
{
    if (kind & 4)
        return (L1 >> qshift) - (L2 >> qshift) <= th;
    if (kind & 1)
        return L1 <= L2;
    if (kind & 8)
        return (kind & 2) != 0;
    if (kind & 2)
        return L1 < th || !(L2 < L1);
    return !(L2 < th || !(L1 < L2));
}

// Per-lane request record for the serial loop and the output epilogue.
struct SelRec {
    uint32_t c1, c2, kind;
    bool eq, aff1;  // equal match; c1 has more cached blocks
    bool a2;        // the fast path's records take c2 as their "a" instance
    int64_t u1, u2, th;
};

__device__ __forceinline__ SelRec load_rec(const int64_t* offsets, uint64_t n, uint64_t r, bool ok,
                                           uint32_t bshift, const uint32_t* cand,
                                           const uint32_t* match, int64_t base, int64_t per,
                                           uint32_t qshift, int64_t slo, uint32_t policy)
{
    SelRec s;
    s.c1 = ok ? cand[r] : 0;
    s.c2 = ok ? cand[n + r] : 0;
    const uint32_t m1 = ok ? match[r] : 0, m2 = ok ? match[n + r] : 0;
    const int64_t len = ok ? offsets[r + 1] - offsets[r] : 0;
    s.u1 = len - ((int64_t)m1 << bshift);
    s.u2 = len - ((int64_t)m2 << bshift);
    s.eq = m1 == m2;
    s.aff1 = m1 > m2;
    // T_a <= slo  <=>  floor(L_a / 2^q) <= slo - base - per*u_a  <=>  L_a < th
    s.th = (slo - base - per * (s.aff1 ? s.u1 : s.u2) + 1) * ((int64_t)1 << qshift);
    s.kind = (s.eq ? 1u : 0u) | (s.aff1 ? 2u : 0u);
    s.a2 = !s.eq && !s.aff1;
    if (policy == DM_POLICY_CACHE_AFFINITY) {
        s.kind |= 8u;
    } else if (policy == DM_POLICY_LEAST_LOADED) {
        s.kind = 1u;
        s.a2 = false;
    } else if (policy == DM_POLICY_MIN_TTFT) {
        s.kind = 4u;
        s.th = per * (s.u2 - s.u1);
        s.a2 = false;
    }
    return s;
}

__device__ __forceinline__ void store_out(const SelRec& s, uint64_t r, int64_t L1, int64_t L2,
                                          uint8_t* flags, uint32_t* chosen, int64_t* ttft,
                                          int64_t base, int64_t per, uint32_t qshift, int64_t slo)
{
    const bool pick1 = pick_first(s.kind, L1, L2, s.th, qshift);
    const int64_t t1 = base + per * s.u1 + (L1 >> qshift);
    const int64_t t2 = base + per * s.u2 + (L2 >> qshift);
    uint32_t f = flags[r];
    if (t1 > slo && t2 > slo)
        f |= 2;
    if (s.eq)
        f |= 4;
    else if (pick1 != s.aff1)
        f |= 1;
    chosen[r] = pick1 ? s.c1 : s.c2;
    ttft[r] = pick1 ? t1 : t2;
    flags[r] = (uint8_t)f;
}

// Serial selection, loads in R register banks of one wave.
template <int R>
__global__ __launch_bounds__(kWave) void select_kernel(
    const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
    const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
    uint8_t* __restrict__ flags, uint32_t* __restrict__ chosen, int64_t* __restrict__ ttft,
    int64_t* __restrict__ loads, uint32_t S, int64_t base, int64_t per, uint32_t qshift, int64_t slo,
    uint32_t policy, const uint32_t* __restrict__ plan)
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
        const SelRec s = load_rec(offsets, n, r, ok, bshift, cand, match, base, per, qshift, slo,
                                  policy);
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
            const bool pick1 = pick_first(K, L1, L2, TH, qshift);
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
    uint32_t policy, const uint32_t* __restrict__ plan)
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
        const SelRec s = load_rec(offsets, n, r, ok, bshift, cand, match, base, per, qshift, slo,
                                  policy);
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
            const bool pick1 = pick_first(K, L1, L2, TH, qshift);
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
// Fast path.
// ---------------------------------------------------------------------------

// A request whose latest earlier request of its block on both of its
// instances is one request with the same pair and cache-affine instance
// joins that request's run while the run holds fewer than kRunMax requests:
// all take the same level, each replays the decisions of the run's earlier
// members (uncached tokens and thresholds copied into its record) before
// its own, and only the run's last member writes the pair's loads.
// Replaying zero increments changes nothing.
constexpr uint32_t kRunMax = 3;

// Per-request record of the packing kernel.
struct SelPack {
    uint32_t w;   // a | o << 8 (dense indices)
    uint32_t ua;  // uncached tokens on a
    uint32_t uo;  // uncached tokens on o
    int32_t th;   // take a iff L_a <= max(th, L_o), relative loads
};

// Per-lane record of one lane set of a window, in the form the window's
// depth steps consume:
// the LDS byte offsets (within the load array, 4-byte slots) of L_a and
// L_o, where the request writes them (its spare slot unless it is the last
// member of its run), rel = its depth in the window (0-based) + the
// window's entry step e, and the window's control word e | (passes - 1) << 4.
// Lanes past a set's requests and the padding windows are inert: every
// offset is the lane's spare slot and rel matches no step.
struct WalkRec {
    uint32_t a4, o4, wa, wo;
    uint32_t rel, ctl;
    uint32_t ua, uo;
    int32_t th;
    uint32_t pua, puo;    // the run's first member: its uncached tokens on a and o
    int32_t pth;          // and its threshold (zeros for a run's first member)
    uint32_t pua2, puo2;  // the run's second member, for its third (else zeros)
    int32_t pth2;
    uint32_t pad;
};
constexpr uint32_t kInertRel = 0xFFFFFFFFu;

// plan[0] = 1 for the serial path; plan[1] = 1 for the windowed path, whose
// loads are 64-bit when plan[2] = 1.
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
    }
    smin[threadIdx.x] = mn;
    __syncthreads();
    for (int d = 128; d > 0; d >>= 1) {
        if (threadIdx.x < d)
            smin[threadIdx.x] = std::min(smin[threadIdx.x], smin[threadIdx.x + d]);
        __syncthreads();
    }
    if (threadIdx.x == 0)
        base[0] = smin[0];
}

constexpr uint32_t kFastMaxLive = 256;
constexpr int kPrefetch = 6;  // record windows in flight ahead of the walk
// Lane sets of a window: every lane holds one request for the window's steps
// of even number and one for its steps of odd number.
constexpr uint32_t kSets = 2;

// grow[0..n_live) and the bad-record word grow[kMaxSlots] start at zero.
__global__ void sel_zero_kernel(unsigned long long* __restrict__ grow, uint32_t n_live)
{
    for (uint32_t k = threadIdx.x; k < n_live && k < kMaxSlots; k += blockDim.x)
        grow[k] = 0;
    if (threadIdx.x == 0)
        grow[kMaxSlots] = 0;
}

__global__ __launch_bounds__(256) void sel_prep_kernel(
    const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
    const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
    const uint32_t* __restrict__ dense, uint32_t n_live, int64_t tbase, int64_t per,
    uint32_t qshift, int64_t slo, uint32_t policy, SelPack* __restrict__ rec,
    unsigned long long* __restrict__ grow)
{
    __shared__ unsigned long long sg[kFastMaxLive];
    const bool track = n_live <= kFastMaxLive;
    if (track)
        for (uint32_t k = threadIdx.x; k < n_live; k += blockDim.x)
            sg[k] = 0;
    __syncthreads();
    unsigned long long bad = 0;
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t m1 = match[r], m2 = match[n + r];
        const int64_t len = offsets[r + 1] - offsets[r];
        const int64_t u1 = len - ((int64_t)m1 << bshift), u2 = len - ((int64_t)m2 << bshift);
        // least load: every request as an equal match, c1 as "a"
        const bool eq = m1 == m2 || policy == DM_POLICY_LEAST_LOADED;
        const bool aff2 = m2 > m1 && policy != DM_POLICY_LEAST_LOADED;
        const uint32_t d1 = dense[cand[r]], d2 = dense[cand[n + r]];
        // T_a <= slo  <=>  floor(L_a / 2^q) <= slo - tbase - per*u_a  <=>
        // L_a < (slo - tbase - per*u_a + 1) 2^q, i.e. "take a iff L_a <=
        // max(th, L_o)" with th one less.  The 32-bit walk uses absolute loads
        // in [0, 2^31 - 1), so th is clamped to that range; equal matches:
        // take c1 iff L1 <= L2, th = -2^31; cache affinity: always a,
        // th = 2^31 - 1.
        int32_t th = INT32_MIN;
        if (!eq && policy == DM_POLICY_CACHE_AFFINITY) {
            th = INT32_MAX;
        } else if (!eq) {
            const int64_t t = (slo - tbase - per * (aff2 ? u2 : u1) + 1) * ((int64_t)1 << qshift) - 1;
            th = (int32_t)(t < -1 ? -1 : (t > INT32_MAX ? INT32_MAX : t));
        }
        SelPack p;
        p.w = aff2 ? ((d2 & 0xFF) | (d1 & 0xFF) << 8) : ((d1 & 0xFF) | (d2 & 0xFF) << 8);
        p.ua = (uint32_t)(aff2 ? u2 : u1);
        p.uo = (uint32_t)(aff2 ? u1 : u2);
        p.th = th;
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

// Windowed path iff at most 256 instances are live and every record's
// uncached counts fit 32 bits (plan[1]).  Its loads are absolute 32-bit
// values when every live load lies in [0, 2^30) and grows by less than 2^30
// whatever the decisions; otherwise (plan[2]) 64-bit values relative to the
// smallest live load, as long as they stay below it + 2^62.  Otherwise the
// serial path (plan[0]).
__global__ __launch_bounds__(256) void sel_plan_kernel(const int64_t* __restrict__ loads,
                                                       const uint32_t* __restrict__ live_ids,
                                                       uint32_t n_live,
                                                       const int64_t* __restrict__ base,
                                                       const unsigned long long* __restrict__ grow,
                                                       uint32_t policy,
                                                       uint32_t* __restrict__ plan)
{
    __shared__ int ok_all, narrow;
    if (threadIdx.x == 0) {
        // the minimum-TTFT rule has no windowed form: serial path
        ok_all = n_live <= kFastMaxLive && grow[kMaxSlots] == 0 && policy != DM_POLICY_MIN_TTFT;
        narrow = 1;
    }
    __syncthreads();
    for (uint32_t k = threadIdx.x; k < n_live && k < kFastMaxLive; k += blockDim.x) {
        // loads - base cannot wrap in unsigned arithmetic: base is the minimum
        const int64_t v = loads[live_ids[k]];
        const unsigned long long span = (unsigned long long)v - (unsigned long long)base[0];
        if (v < 0 || v >= (1ll << 30) || grow[k] >= (1ull << 30))
            atomicAnd(&narrow, 0);
        if (span >= (1ull << 62) || grow[k] >= (1ull << 62))
            atomicAnd(&ok_all, 0);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        plan[0] = ok_all ? 0 : 1;
        plan[1] = ok_all ? 1 : 0;
        plan[2] = ok_all && !narrow ? 1 : 0;
    }
}

// Walk windows from dependency levels.  Requests are grouped in blocks of
// LB requests (request order).  Inside a block, a request's level is 1 + the
// larger level of the latest earlier request of the block on either
// candidate (0 when none), except that a request that joins a run (see
// kRunMax) takes the run's level.
// Along every instance's requests the level strictly grows outside runs, so
// the requests (runs) of one level touch pairwise distinct instances, and
// any order of the levels' requests that keeps levels in order and the
// blocks in order gives every request exactly the loads of the one-by-one
// walk.  A level of more than 64 requests is cut, runs kept whole, into
// parts of at most 64, each part a depth of its own.  Windows take
// consecutive parts, one per depth, and hold two sets of 64 lanes: the
// depths alternate between the sets (steps of even and odd number), so a
// window holds up to 128 requests.  Packing the same parts into windows of
// one set of 64 lanes would close a window only when the next part does not
// fit, so any two consecutive such windows hold more than 64 requests and a
// block needs at most 2 * ceil(LB / 65) + 1 of them; the two-set packing
// needs no more.
//
// Larger blocks give fewer depth steps and windows (on the large batch,
// 78,742 steps in 9,832 windows with blocks of 2048 against 79,786 in
// 10,225 with 1024) but take the level kernel twice as long per block, which
// only a batch long enough to hide it behind its walk repays: batches of
// at least kLargeFrom requests use blocks of 2048, others blocks of 1024.
template <uint32_t LB>
struct LevelShape {
    static constexpr uint32_t block = LB;
    static constexpr uint32_t wincap = LB == 1024 ? 36u : 66u;  // windows per block
    static_assert(wincap >= 2 * ((LB + 64) / 65) + 1, "room for the windows of a block");
};
constexpr uint64_t kLargeFrom = 1u << 19;
// The batch limit follows the large layout; the small one only serves
// batches whose slots stay far inside 32 bits.
static_assert(LevelShape<2048>::block == kSelBlock &&
                  LevelShape<2048>::wincap == kSelWindowsPerBlock &&
                  kLargeFrom / 1024 * LevelShape<1024>::wincap * kSets * kWave < (1ull << 32),
              "dm_route_batch's batch limit assumes this layout");

// Block size and window capacity of a batch of n requests.
struct BlockShape {
    uint32_t block, wincap;
};
static BlockShape block_shape(uint64_t n)
{
    return n >= kLargeFrom ? BlockShape{LevelShape<2048>::block, LevelShape<2048>::wincap}
                           : BlockShape{LevelShape<1024>::block, LevelShape<1024>::wincap};
}

// One wave per block.  Writes, per request, info = depth in its window |
// position in its run << 6 | (not the run's last) << 8 | run's first member
// << 9 | run's second member << 20 (block-local indices); per block, its
// window count, each window's depth and the block-local request index in
// every lane of both sets of every window (0xFFFF for none).  The result is that of taking the
// requests one by one; the wave takes them 64 at a time, in order:
//   - the latest earlier request on each instance: within the chunk from
//     per-instance lane masks, before it from the latest request of the
//     earlier chunks on that instance;
//   - a request whose latest earlier request on both instances is one
//     request of the same pair and orientation is a run candidate; its
//     position in the run is (the predecessor's position + 1) mod kRunMax,
//     0 for any other request (settled along the chunk's candidate chains
//     with wave-wide votes);
//   - levels: the least fixed point of the level rule over the chunk
//     (earlier chunks' levels are final; relaxation from 1, wave-wide votes);
//   - then, with the runs' sizes final, each run reserves its lanes within
//     its level (LDS atomics: any order of a level's runs is valid);
//   - the levels are cut into parts (a lane per level), and the parts placed
//     into windows by one uniform greedy pass over their sizes.
// Every LDS access is by this one wave, so no barrier is needed.
template <uint32_t LB>
__global__ __launch_bounds__(kWave) void sel_level_kernel(
    const SelPack* __restrict__ prep, uint64_t n, uint32_t* __restrict__ info,
    uint16_t* __restrict__ slotmap, uint8_t* __restrict__ wdepth, uint32_t* __restrict__ wcount,
    uint32_t* __restrict__ status)
{
    constexpr uint32_t kWinCap = LevelShape<LB>::wincap;
    __shared__ unsigned long long cm[kFastMaxLive];  // lanes of the chunk on each instance
    __shared__ uint16_t last[kFastMaxLive];         // latest request of earlier chunks, + 1
    __shared__ uint16_t W[LB];              // a | o << 8
    __shared__ int16_t P[LB];               // latest earlier request on a
    __shared__ uint8_t psn[LB];             // position in the run
    __shared__ uint16_t hd[LB];             // the run's first member
    __shared__ uint16_t lv[LB];
    __shared__ uint8_t has1[LB], has2[LB];  // a run has a 2nd / 3rd member
    __shared__ __align__(16) uint16_t key[LB];  // a run's first member: level << 2 | size
    __shared__ uint16_t hrank[LB];    // lanes of earlier runs of the same level
    __shared__ uint32_t cnt[LB + 2];  // requests per level (so far), then
                                               // each level's first part
    __shared__ uint16_t lstart[LB + 1];
    __shared__ uint16_t sorted[LB];   // requests by level, runs in order
    __shared__ uint16_t pl_s0[LB];     // part: first index in sorted
    __shared__ uint8_t pl_win[LB], pl_base[LB];  // window, first lane in set
    __shared__ uint16_t wfirst[kWinCap];        // first part of each window
    __shared__ uint16_t smap[kWinCap * kSets * kWave];
    __shared__ uint8_t wdep[kWinCap];
    const uint32_t lane = (uint32_t)lane_id();
    const uint64_t r0 = (uint64_t)blockIdx.x * LB;
    const uint32_t nb = (uint32_t)std::min<uint64_t>(LB, n - r0);
    const unsigned long long below = (1ull << lane) - 1, above = ~below << 1;
    for (uint32_t k = lane; k < kFastMaxLive; k += kWave)
        last[k] = 0;
    for (uint32_t k = lane; k < LB + 2; k += kWave)
        cnt[k] = 0;
    for (uint32_t k = lane; k < kWinCap * kSets * kWave; k += kWave)
        smap[k] = 0xFFFF;
    {
        // all pair codes first: 32 loads in flight per lane, one wait
        uint32_t wv[LB / kWave];
#pragma unroll
        for (uint32_t k = 0; k < LB / kWave; k++) {
            const uint32_t t = k * kWave + lane;
            wv[k] = t < nb ? prep[r0 + t].w : 0u;
        }
#pragma unroll
        for (uint32_t k = 0; k < LB / kWave; k++)
            W[k * kWave + lane] = (uint16_t)(wv[k] & 0xFFFFu);
    }
    uint32_t lmax = 0;
    for (uint32_t c0 = 0; c0 < nb; c0 += kWave) {
        const uint32_t t = c0 + lane;
        const bool valid = t < nb;
        const uint32_t w = W[t], a = w & 0xFF, o = w >> 8;
        has1[t] = has2[t] = 0;
        for (uint32_t k = lane; k < kFastMaxLive; k += kWave)
            cm[k] = 0;
        if (valid) {
            atomicOr(&cm[a], 1ull << lane);
            if (o != a)
                atomicOr(&cm[o], 1ull << lane);
        }
        const unsigned long long ma = valid ? cm[a] : 0, mo = valid ? cm[o] : 0;
        auto latest = [&](unsigned long long m, uint32_t x) -> int {
            m &= below;
            return m ? (int)(c0 + 63 - __clzll(m)) : (int)last[x] - 1;
        };
        const int pa = valid ? latest(ma, a) : -1, po = valid ? latest(mo, o) : -1;
        P[t] = (int16_t)pa;
        // the last lane of the chunk on an instance records it for later chunks
        if (valid && !(ma & above))
            last[a] = (uint16_t)(t + 1);
        if (valid && o != a && !(mo & above))
            last[o] = (uint16_t)(t + 1);
        const bool cand = valid && pa >= 0 && pa == po && a != o && W[pa] == w;
        // positions: 0 off the candidate chains; a predecessor in an earlier
        // chunk is settled; one in this chunk settles in turn
        const bool inchunk = cand && (uint32_t)pa >= c0;
        uint32_t pos = cand && !inchunk ? (psn[pa] + 1u) % kRunMax : 0u;
        bool done = !inchunk;
        for (;;) {
            const int src = inchunk ? pa - (int)c0 : (int)lane;
            const uint32_t ppos = (uint32_t)__shfl((int)pos, src);
            const bool pdone = __shfl((int)done, src) != 0;
            const bool now = !done && pdone;
            if (now) {
                pos = (ppos + 1u) % kRunMax;
                done = true;
            }
            if (!__any(now))
                break;
        }
        psn[t] = (uint8_t)pos;
        uint32_t h = t;
        for (uint32_t k = 0; k < pos; k++)
            h = (uint32_t)P[h];
        hd[t] = (uint16_t)h;
        if (valid && pos == 1)
            has1[h] = 1;
        if (valid && pos == 2)
            has2[h] = 1;
        // levels of the chunk: the least fixed point, from 1 up; levels of
        // earlier chunks are final (read once), those of this chunk's
        // predecessors come from their lanes
        const bool ina = pa >= (int)c0, ino = po >= (int)c0;
        const uint32_t la0 = !ina && pa >= 0 ? lv[pa] : 0u, lo0 = !ino && po >= 0 ? lv[po] : 0u;
        const int sa = ina ? pa - (int)c0 : (int)lane, so = ino ? po - (int)c0 : (int)lane;
        uint32_t L = valid ? 1u : 0u;
        for (;;) {
            const uint32_t xa = (uint32_t)__shfl((int)L, sa), xo = (uint32_t)__shfl((int)L, so);
            const uint32_t va = ina ? xa : la0, vo = ino ? xo : lo0;
            const uint32_t nl = !valid ? 0u : pos > 0 ? va : 1u + std::max(va, vo);
            const bool ch = nl != L;
            L = nl;
            if (!__any(ch))
                break;
        }
        lv[t] = (uint16_t)L;
        lmax = std::max(lmax, L);
    }
    for (int d = 1; d < kWave; d <<= 1)
        lmax = std::max(lmax, (uint32_t)__shfl_xor((int)lmax, d));
    lmax = (uint32_t)__builtin_amdgcn_readfirstlane((int)lmax);  // uniform from here on
    // inclusive sum over the wave
    auto wave_incl = [&](uint32_t v) -> uint32_t {
        for (int d = 1; d < kWave; d <<= 1) {
            const uint32_t y = (uint32_t)__shfl_up((int)v, d);
            if ((int)lane >= d)
                v += y;
        }
        return v;
    };
    // the lanes of the runs within their levels, with the runs' sizes final:
    // each run's first member reserves the run's size in its level's count.
    // Requests of one level are independent, so any order of a level's runs
    // is valid; a run's members stay together, in run order.
    for (uint32_t t = lane; t < nb; t += kWave) {
        const bool head = psn[t] == 0;
        const uint32_t L = lv[t], rs = 1u + has1[t] + has2[t];
        key[t] = head ? (uint16_t)(L << 2 | rs) : (uint16_t)0;
        if (head)
            hrank[t] = (uint16_t)atomicAdd(&cnt[L], rs);
    }
    // each level's first index in sorted (a scan of the counts)
    for (uint32_t l0 = 1, start = 0; l0 <= lmax; l0 += kWave) {
        const uint32_t l = l0 + lane, c = l <= lmax ? cnt[l] : 0u, x = wave_incl(c);
        if (l <= lmax)
            lstart[l] = (uint16_t)(start + x - c);
        start += (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
    }
    for (uint32_t t = lane; t < nb; t += kWave)
        sorted[lstart[lv[t]] + hrank[hd[t]] + psn[t]] = (uint16_t)t;
    // Parts, one lane per level: a level of at most 64 requests is one part;
    // a larger one is cut run by run into parts of at most 64 (its requests
    // are independent, so its parts may take consecutive depths).  The parts
    // cover sorted in order, so part p holds [pl_s0[p], pl_s0[p + 1]); cnt[l]
    // becomes level l's first part (a scan of the part counts).
    auto cut = [&](uint32_t s0, uint32_t c, uint32_t first, bool write) -> uint32_t {
        uint32_t np = 1, part = 0;
        if (write)
            pl_s0[first] = (uint16_t)s0;
        for (uint32_t k = s0; k < s0 + c;) {
            const uint32_t sz = key[sorted[k]] & 3u;  // k is a run's first member
            if (part + sz > kWave) {
                if (write)
                    pl_s0[first + np] = (uint16_t)k;
                np++;
                part = 0;
            }
            part += sz;
            k += sz;
        }
        return np;
    };
    uint32_t npl = 0;
    for (uint32_t l0 = 1; l0 <= lmax; l0 += kWave) {
        const uint32_t l = l0 + lane;
        const bool has = l <= lmax;
        const uint32_t c = has ? cnt[l] : 0u, s0 = has ? lstart[l] : 0u;
        const uint32_t np = !has ? 0u : c <= kWave ? 1u : cut(s0, c, 0, false);
        const uint32_t x = wave_incl(np), first = npl + x - np;
        if (has) {
            cnt[l] = first;
            if (c <= kWave)
                pl_s0[first] = (uint16_t)s0;
            else
                (void)cut(s0, c, first, true);
        }
        npl += (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
    }
    if (lane == 0)
        cnt[lmax + 1] = npl;
    // Windows of consecutive parts, one depth each: a window of depth D is
    // entered at step e = -D mod 16, so depth t runs on step e + t and takes
    // the lane set of that step's parity, (t + D) & 1.  S0 and S1 sum the
    // parts at an even and an odd distance from the window's last depth;
    // appending a part moves every other part one further, so the window
    // grows while c + S1 <= 64 and the depth stays below 65.  A window that
    // fits holds every window inside it, so closing at the first misfit
    // gives the fewest windows; any window that fits one set of 64 lanes
    // fits the two, so the bound of kWinCap holds.  Parts of one set are
    // those of one depth parity, so a part's first lane is the sum of the
    // earlier parts of its depth parity in the window.  The wave takes the
    // parts 64 at a time, their sizes in lanes; the decisions are uniform.
    uint32_t win = 0, D = 0, S0 = 0, S1 = 0, be = 0, bo = 0;
    for (uint32_t p0 = 0; p0 < npl; p0 += kWave) {
        const uint32_t p = p0 + lane;
        const uint32_t cl = p < npl ? (p + 1 < npl ? (uint32_t)pl_s0[p + 1] : nb) - pl_s0[p] : 0u;
        uint32_t wl = 0, bl = 0;
        const uint32_t m = npl - p0 < (uint32_t)kWave ? npl - p0 : (uint32_t)kWave;
        for (uint32_t i = 0; i < m; i++) {
            const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)cl, (int)i);
            if (D > 0 && (D == kWave || c + S1 > kWave)) {
                if (win < kWinCap) {
                    wdep[win] = (uint8_t)D;
                    wfirst[win] = (uint16_t)(p0 + i - D);
                }
                win++;
                D = S0 = S1 = be = bo = 0;
            }
            const uint32_t base = (D & 1u) ? bo : be;
            if (D & 1u)
                bo += c;
            else
                be += c;
            wl = lane == i ? win : wl;
            bl = lane == i ? base : bl;
            const uint32_t s0n = c + S1;
            S1 = S0;
            S0 = s0n;
            D++;
        }
        if (p < npl) {
            pl_win[p] = (uint8_t)wl;
            pl_base[p] = (uint8_t)bl;
        }
    }
    if (win < kWinCap) {
        wdep[win] = (uint8_t)D;
        wfirst[win] = (uint16_t)(npl - D);
    }
    const uint32_t nwin = win + 1;
    const bool okw = nwin <= kWinCap;
    if (!okw && lane == 0)  // cannot happen (see above); no window of this block is walked
        atomicOr(status, kErrInval);
    if (okw) {
        for (uint32_t t = lane; t < nb; t += kWave) {
            const uint32_t L = lv[t], pos = psn[t], h = hd[t], rs = 1u + has1[h] + has2[h];
            const uint32_t k = lstart[L] + hrank[h] + pos;  // index in sorted
            uint32_t p = cnt[L];
            while (p + 1 < cnt[L + 1] && pl_s0[p + 1] <= k)
                p++;
            const uint32_t w = pl_win[p], d = p - wfirst[w], set = (d + wdep[w]) & 1u;
            const uint32_t ln = pl_base[p] + (k - pl_s0[p]);
            smap[(w * kSets + set) * kWave + ln] = (uint16_t)t;
            const uint32_t m1 = pos == 2 ? (uint32_t)P[t] : 0u;
            info[r0 + t] = d | pos << 6 | (pos + 1 < rs ? 1u << 8 : 0u) | h << 9 | m1 << 20;
        }
    }
    for (uint32_t k = lane; k < kWinCap * kSets * kWave; k += kWave)
        slotmap[(uint64_t)blockIdx.x * kWinCap * kSets * kWave + k] = smap[k];
    if (lane < kWinCap)
        wdepth[(uint64_t)blockIdx.x * kWinCap + lane] = okw && lane < nwin ? wdep[lane] : 0;
    if (lane == 0)
        wcount[blockIdx.x] = okw ? nwin : 0;
}

// Exclusive scan of the blocks' window counts (one workgroup); total[0] =
// all windows.
__global__ __launch_bounds__(1024) void sel_scan_kernel(const uint32_t* __restrict__ wcount,
                                                        uint64_t nblk, uint32_t* __restrict__ woff,
                                                        uint32_t* __restrict__ total)
{
    __shared__ uint32_t part[1024 / kWave];
    __shared__ uint32_t carry;
    const uint32_t t = threadIdx.x, lane = t & 63, wv = t >> 6;
    if (t == 0)
        carry = 0;
    __syncthreads();
    for (uint64_t c0 = 0; c0 < nblk; c0 += 1024) {
        const uint64_t b = c0 + t;
        const uint32_t v = b < nblk ? wcount[b] : 0;
        uint32_t x = v;  // inclusive scan within the wave
        for (int d = 1; d < kWave; d <<= 1) {
            const uint32_t y = (uint32_t)__shfl_up((int)x, d);
            if ((int)lane >= d)
                x += y;
        }
        if (lane == 63)
            part[wv] = x;
        __syncthreads();
        uint32_t before = carry;
        for (uint32_t k = 0; k < wv; k++)
            before += part[k];
        if (b < nblk)
            woff[b] = before + x - v;
        __syncthreads();
        if (t == 1023)
            carry = before + x;
        __syncthreads();
    }
    if (t == 0)
        total[0] = carry;
}

// One wave per lane set of every (block, window) of capacity, then of
// 2 * kPrefetch padding windows: the walk records of every lane (inert past
// the set's requests) and each request's slot.  The records of window w's
// set s start at (w * kSets + s) * 64.
__global__ __launch_bounds__(4 * kWave) void sel_fill_kernel(
    const SelPack* __restrict__ prep, uint64_t n, const uint32_t* __restrict__ info,
    const uint16_t* __restrict__ slotmap, const uint8_t* __restrict__ wdepth,
    const uint32_t* __restrict__ wcount, const uint32_t* __restrict__ woff,
    const uint32_t* __restrict__ total, uint64_t nblk, BlockShape bs, WalkRec* __restrict__ rec,
    uint32_t* __restrict__ slot_of)
{
    const uint32_t wincap = bs.wincap, bsize = bs.block;
    const int lane = lane_id();
    const uint64_t gw = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const uint64_t ws = gw / kSets;  // window of capacity
    const uint32_t set = (uint32_t)(gw % kSets);
    const uint32_t sp = 4u * (kFastMaxLive + lane);
    uint64_t win;
    uint32_t k = 0xFFFF, depth = 1;
    uint64_t blk = 0;
    if (ws < nblk * wincap) {
        blk = ws / wincap;
        const uint32_t lw = (uint32_t)(ws % wincap);
        if (lw >= wcount[blk])
            return;
        win = (uint64_t)woff[blk] + lw;
        k = slotmap[gw * kWave + lane];
        depth = wdepth[ws];
    } else if (ws < nblk * wincap + 2 * kPrefetch) {
        win = (uint64_t)total[0] + (ws - nblk * wincap);
    } else {
        return;
    }
    const uint32_t e = (0u - depth) & 15u, passes = (depth + 15u) >> 4;
    WalkRec q;
    q.ctl = e | (passes - 1) << 4;
    const uint64_t r = blk * bsize + k;
    if (k != 0xFFFF && r < n) {
        const SelPack me = prep[r];
        const uint32_t f = info[r], pos = (f >> 6) & 3;
        const bool not_last = (f >> 8) & 1;
        q.a4 = 4u * (me.w & 0xFF);
        q.o4 = 4u * ((me.w >> 8) & 0xFF);
        q.wa = not_last ? sp : q.a4;
        q.wo = not_last ? sp : q.o4;
        q.rel = (f & 63) + e;
        q.ua = me.ua;
        q.uo = me.uo;
        q.th = me.th;
        q.pua = q.puo = q.pua2 = q.puo2 = 0;
        q.pth = q.pth2 = 0;
        q.pad = 0;
        if (pos >= 1) {
            const SelPack m0 = prep[blk * bsize + ((f >> 9) & (bsize - 1))];
            q.pua = m0.ua;
            q.puo = m0.uo;
            q.pth = m0.th;
        }
        if (pos >= 2) {
            const SelPack m1 = prep[blk * bsize + ((f >> 20) & (bsize - 1))];
            q.pua2 = m1.ua;
            q.puo2 = m1.uo;
            q.pth2 = m1.th;
        }
        slot_of[r] = (uint32_t)((win * kSets + set) * kWave + lane);
    } else {
        q.a4 = q.o4 = q.wa = q.wo = sp;
        q.rel = kInertRel;
        q.ua = q.uo = q.pua = q.puo = q.pua2 = q.puo2 = q.pad = 0;
        q.th = q.pth = q.pth2 = 0;
    }
    rec[(win * kSets + set) * kWave + lane] = q;
}

// Walks the windows in order; see the file comment.  T is the load type:
// int32_t or int64_t relative loads.  rec holds 2 * kPrefetch inert padding
// windows past the last and lpre kPrefetch, so that the unrolled walk and
// its prefetch stay in bounds; lpre receives the pre-update loads (L_a, L_o)
// of every request relative to the base, as int32 pairs for the 32-bit walk
// and int64 pairs for the 64-bit one, at the request's slot (window w, set
// s, lane l: (w * kSets + s) * 64 + l).
// Byte address of a shared-memory element within the workgroup's LDS.
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(T* p)
{
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) T*)p;
}

// One depth step of the 32-bit walk, as asm text for DM_WALK_BLOCK: the
// lanes of set S whose rel equals the inline constant K are on this depth
// (steps of even number take set A, of odd number set B).  The loads of a
// step live in one register pair X = (L_a, L_o): v[240:241] on even steps,
// v[242:243] on odd ones, so that a decision adds both of its increments
// with one 64-bit add.  No carry crosses the halves for a lane on its
// depth: on this path every live load and its growth stay below 2^31.  (A
// lane off its depth may carry; its values only reach its spare slot.)
// Reads X (L_o first), replays the decisions of the run's earlier members
// (no change for zero increments) into X: the loads this request saw;
// captures the previous step's pair XP (lane mask MP) into the other set's
// (La, Lo); M receives this step's lane mask.  Then the lane's own decision
// into v[246:247], and both loads of the pair written back (the second
// instance first, so that a pair of one instance keeps the first's value)
// -- to the lane's write slots (wa, wo) when on the depth, else to its spare
// slot.  The reads of a depth precede its writes in the LDS queue, and the
// writes of one depth precede the reads of the next, so the waits count
// this step's reads only.  Every step has the same instructions with
// fixed-size encodings (operands are registers and inline constants), which
// the computed entry relies on; the assembler checks the sizes.
#define DM_STEP_TEXT(K, XA, XO, X, M, XAP, XOP, MP, S, P)                                      \
    ".Ldmw%=_" #K ":\n\t"                                                                      \
    "ds_read_b32 " XO ", %[o4" S "]\n\t"                                                       \
    "ds_read_b32 " XA ", %[a4" S "]\n\t"                                                       \
    "v_cmp_eq_u32_e64 %[" M "], " #K ", %[rel" S "]\n\t"                                      \
    "v_cndmask_b32_e64 %[La" P "], %[La" P "], " XAP ", %[" MP "]\n\t"                         \
    "v_cndmask_b32_e64 %[Lo" P "], %[Lo" P "], " XOP ", %[" MP "]\n\t"                         \
    "v_cndmask_b32_e64 %[da], %[sp], %[wa" S "], %[" M "]\n\t"                                 \
    "v_cndmask_b32_e64 %[dz], %[sp], %[wo" S "], %[" M "]\n\t"                                 \
    "s_waitcnt lgkmcnt(1)\n\t"                                                                 \
    "v_max_i32_e32 v244, %[pth" S "], " XO "\n\t"                                              \
    "s_waitcnt lgkmcnt(0)\n\t"                                                                 \
    "v_cmp_le_i32_e32 vcc, " XA ", v244\n\t"                                                   \
    "v_cndmask_b32_e64 v244, 0, %[pua" S "], vcc\n\t"                                          \
    "v_cndmask_b32_e64 v245, %[puo" S "], 0, vcc\n\t"                                          \
    "v_lshl_add_u64 " X ", " X ", 0, v[244:245]\n\t"                                           \
    "v_max_i32_e32 v244, %[pth2" S "], " XO "\n\t"                                             \
    "v_cmp_le_i32_e32 vcc, " XA ", v244\n\t"                                                   \
    "v_cndmask_b32_e64 v244, 0, %[pua2" S "], vcc\n\t"                                         \
    "v_cndmask_b32_e64 v245, %[puo2" S "], 0, vcc\n\t"                                         \
    "v_lshl_add_u64 " X ", " X ", 0, v[244:245]\n\t"                                           \
    "v_max_i32_e32 v246, %[th" S "], " XO "\n\t"                                               \
    "v_cmp_le_i32_e32 vcc, " XA ", v246\n\t"                                                   \
    "v_cndmask_b32_e64 v244, 0, %[ua" S "], vcc\n\t"                                           \
    "v_cndmask_b32_e64 v245, %[uo" S "], 0, vcc\n\t"                                           \
    "v_lshl_add_u64 v[246:247], " X ", 0, v[244:245]\n\t"                                      \
    "ds_write_b32 %[dz], v247\n\t"                                                             \
    "ds_write_b32 %[da], v246\n\t"

#define DM_STEP_PAIR(K0, K1)                                                                   \
    DM_STEP_TEXT(K0, "v240", "v241", "v[240:241]", "m0", "v242", "v243", "m1", "A", "B")       \
    DM_STEP_TEXT(K1, "v242", "v243", "v[242:243]", "m1", "v240", "v241", "m0", "B", "A")

#define DM_SIZE_CHECK(K0, K1)                                                                  \
    ".if (.Ldmw%=_" #K1 " - .Ldmw%=_" #K0 ") != (.Ldmw%=_1 - .Ldmw%=_0)\n\t"                   \
    ".error \"walk steps differ in size\"\n\t"                                                 \
    ".endif\n\t"

#define DM_SET_OPERANDS(S)                                                                     \
    [a4##S] "v"(a4##S), [o4##S] "v"(o4##S), [wa##S] "v"(wa##S), [wo##S] "v"(wo##S),            \
        [th##S] "v"(c##S.th), [ua##S] "v"(c##S.ua), [uo##S] "v"(c##S.uo),                      \
        [pth##S] "v"(c##S.pth), [pua##S] "v"(c##S.pua), [puo##S] "v"(c##S.puo),                \
        [pth2##S] "v"(c##S.pth2), [pua2##S] "v"(c##S.pua2), [puo2##S] "v"(c##S.puo2)

// All depths of one window of the 32-bit walk in one block of 16 steps
// (K = 0..15), entered at step e by a computed jump (the PC-relative
// sequence of a long branch) and run np1 + 1 times, where the window's
// control word (the same in every lane) is e | np1 << 4; lane l of set A
// (B) is on even (odd) step K of pass j when its rel - 16 j = K.  The
// control word is read inside the block, so that the compiler waits only
// for this window's records.  The first step captures whatever its register
// set held, which is harmless: every lane of the batch is captured again
// after its own depth, and inert lanes' results are never read.  After the
// last pass the last depth's reads (an odd step: set B) are captured into
// (LaB, LoB).  e < 16 and np1 < 4 by the masks, and the assembler checks
// that the 16 steps have one size.
#define DM_WALK_BLOCK()                                                                        \
    asm volatile("v_readfirstlane_b32 s99, %[ctl]\n\t"                                         \
                 "s_getpc_b64 s[96:97]\n"                                                      \
                 ".Ldmw%=_pc:\n\t"                                                             \
                 "s_and_b32 s98, s99, 15\n\t"                                                  \
                 "s_mul_i32 s98, s98, (.Ldmw%=_1 - .Ldmw%=_0)\n\t"                             \
                 "s_add_u32 s98, s98, (.Ldmw%=_0 - .Ldmw%=_pc)\n\t"                            \
                 "s_add_u32 s96, s96, s98\n\t"                                                 \
                 "s_addc_u32 s97, s97, 0\n\t"                                                  \
                 "s_bfe_u32 s99, s99, 0x20004\n\t"                                             \
                 "s_setpc_b64 s[96:97]\n"                                                      \
                 DM_STEP_PAIR(0, 1) DM_STEP_PAIR(2, 3) DM_STEP_PAIR(4, 5) DM_STEP_PAIR(6, 7)  \
                 DM_STEP_PAIR(8, 9) DM_STEP_PAIR(10, 11) DM_STEP_PAIR(12, 13)                 \
                 DM_STEP_PAIR(14, 15)                                                          \
                 ".Ldmw%=_16:\n\t"                                                             \
                 "v_add_u32_e32 %[relA], -16, %[relA]\n\t"                                     \
                 "v_add_u32_e32 %[relB], -16, %[relB]\n\t"                                     \
                 "s_sub_u32 s99, s99, 1\n\t"                                                   \
                 "s_cbranch_scc0 .Ldmw%=_0\n\t"                                                \
                 "v_cndmask_b32_e64 %[LaB], %[LaB], v242, %[m1]\n\t"                             \
                 "v_cndmask_b32_e64 %[LoB], %[LoB], v243, %[m1]\n\t"                             \
                 DM_SIZE_CHECK(1, 2) DM_SIZE_CHECK(2, 3) DM_SIZE_CHECK(3, 4)                   \
                 DM_SIZE_CHECK(4, 5) DM_SIZE_CHECK(5, 6) DM_SIZE_CHECK(6, 7)                   \
                 DM_SIZE_CHECK(7, 8) DM_SIZE_CHECK(8, 9) DM_SIZE_CHECK(9, 10)                  \
                 DM_SIZE_CHECK(10, 11) DM_SIZE_CHECK(11, 12) DM_SIZE_CHECK(12, 13)             \
                 DM_SIZE_CHECK(13, 14) DM_SIZE_CHECK(14, 15) DM_SIZE_CHECK(15, 16)             \
                 : [m0] "=&s"(m0), [m1] "=&s"(m1), [LaA] "+v"(LaA), [LoA] "+v"(LoA),          \
                   [LaB] "+v"(LaB), [LoB] "+v"(LoB), [da] "=&v"(da), [dz] "=&v"(dz),          \
                   [relA] "+v"(relA), [relB] "+v"(relB)                                        \
                 : DM_SET_OPERANDS(A), DM_SET_OPERANDS(B), [sp] "v"(sp4), [ctl] "v"(ctl)      \
                 : "s96", "s97", "s98", "s99", "v240", "v241", "v242", "v243", "v244", "v245",  \
                   "v246", "v247", "vcc", "scc", "memory")

template <typename T>
__device__ __forceinline__ void walk_windows(const WalkRec* __restrict__ rec,
                                             const uint32_t* __restrict__ nwin,
                                             const uint32_t* __restrict__ live_ids,
                                             uint32_t n_live, int64_t* __restrict__ loads,
                                             int64_t b0, longlong2* __restrict__ lpre,
                                             int64_t tbase, int64_t per, uint32_t qshift,
                                             int64_t slo, uint32_t policy, T* L)
{
    constexpr bool wide = sizeof(T) == 8;
    const int lane = lane_id();
    for (uint32_t d = lane; d < kFastMaxLive + kWave; d += kWave)
        L[d] = d < n_live ? (T)(loads[live_ids[d]] - b0) : (T)0;
    __syncthreads();
    const uint64_t nw = __builtin_amdgcn_readfirstlane(nwin[0]);
    // the records hold offsets within L in 4-byte slots; the LDS address of
    // L itself is a link-time constant (zero when it is the only array)
    const uint32_t lbase = lds_addr(reinterpret_cast<int32_t*>(L));
    const uint32_t sp4 = lbase + 4u * (kFastMaxLive + lane);
    int32_t LaA32 = 0, LoA32 = 0, LaB32 = 0, LoB32 = 0;
    // window w: set A's records cA, set B's cB (same control word)
    auto window = [&](WalkRec& cA, WalkRec& cB, uint64_t w) {
        if constexpr (wide) {
            // the packed bounds are clamped to 32 bits: recompute them
            // exactly, relative to the base (equal matches: -inf; cache
            // affinity: +inf)
            const bool keep_a = policy == DM_POLICY_CACHE_AFFINITY;
            auto exact = [&](int32_t packed, uint32_t u) -> T {
                return packed == INT32_MIN ? (T)INT64_MIN
                       : keep_a            ? (T)INT64_MAX
                                           : (T)((slo - tbase - per * (int64_t)u + 1) *
                                                     ((int64_t)1 << qshift) -
                                                 1 - b0);
            };
            // Every lane reads and writes at every depth, without branches on
            // lane data; a lane not on the current depth, and a run member
            // other than the last, write their own spare slot.
            const uint32_t ctl = __builtin_amdgcn_readfirstlane(cA.ctl), e = ctl & 15u;
            const uint32_t depth = 16u * (((ctl >> 4) & 3u) + 1u) - e;
            const uint32_t sp = kFastMaxLive + lane;
            T La[kSets] = {0, 0}, Lo[kSets] = {0, 0};
            auto step = [&](const WalkRec& c, uint32_t l, T& la, T& lo) {
                const T th = exact(c.th, c.ua), pth = exact(c.pth, c.pua);
                const T pth2 = exact(c.pth2, c.pua2);
                const T ua = (T)c.ua, uo = (T)c.uo, pua = (T)c.pua, puo = (T)c.puo;
                const T pua2 = (T)c.pua2, puo2 = (T)c.puo2;
                const uint32_t a = c.a4 >> 2, o = c.o4 >> 2, wa = c.wa >> 2, wo = c.wo >> 2;
                const bool act = c.rel - e == l;
                const T xa = L[a], xo = L[o];
                const bool p1 = xa <= std::max(pth, xo);
                const T x0 = xa + (p1 ? pua : (T)0), y0 = xo + (p1 ? (T)0 : puo);
                const bool p2 = x0 <= std::max(pth2, y0);
                const T x1 = x0 + (p2 ? pua2 : (T)0), y1 = y0 + (p2 ? (T)0 : puo2);
                const bool take_a = x1 <= std::max(th, y1);
                L[act ? wo : sp] = take_a ? y1 : y1 + uo;
                L[act ? wa : sp] = take_a ? x1 + ua : x1;
                la = act ? x1 : la;
                lo = act ? y1 : lo;
            };
            for (uint32_t l = 0; l < depth; l++) {
                if ((e + l) & 1u)
                    step(cB, l, La[1], Lo[1]);
                else
                    step(cA, l, La[0], Lo[0]);
            }
            lpre[(w * kSets) * kWave + lane] = make_longlong2(La[0], Lo[0]);
            lpre[(w * kSets + 1) * kWave + lane] = make_longlong2(La[1], Lo[1]);
        } else {
            // The same walk in hand-scheduled depth steps (DM_WALK_BLOCK): the
            // ALU work of a step that does not wait for its reads runs in the
            // shadow of the LDS round trip, and the window's depths run as one
            // straight block entered at the step that leaves exactly its
            // depth's steps (a pass of 16 more per further 16 depths).
            const uint32_t a4A = lbase + cA.a4, o4A = lbase + cA.o4;
            const uint32_t waA = lbase + cA.wa, woA = lbase + cA.wo;
            const uint32_t a4B = lbase + cB.a4, o4B = lbase + cB.o4;
            const uint32_t waB = lbase + cB.wa, woB = lbase + cB.wo;
            const uint32_t ctl = cA.ctl;
            uint32_t relA = cA.rel, relB = cB.rel;
            int32_t da, dz;
            uint64_t m0, m1;
            int32_t LaA = LaA32, LoA = LoA32, LaB = LaB32, LoB = LoB32;
            DM_WALK_BLOCK();
            (void)m0; (void)m1; (void)da; (void)dz;
            LaA32 = LaA;
            LoA32 = LoA;
            LaB32 = LaB;
            LoB32 = LoB;
            int2* lp = reinterpret_cast<int2*>(lpre);
            lp[(w * kSets) * kWave + lane] = make_int2(LaA, LoA);
            lp[(w * kSets + 1) * kWave + lane] = make_int2(LaB, LoB);
        }
    };
    // Records arrive kPrefetch windows ahead.  The loop is unrolled by
    // kPrefetch so that each slot is used where it was loaded (no register
    // moves, which would wait for every load in flight); windows past the
    // last (inert padded records and outputs) change nothing.  With an odd
    // unroll the compiler's wait at the loop head let only a few loads stay
    // in flight (vmcnt(5)), which cost 12-15% of the walk.
    static_assert(kPrefetch % 2 == 0, "keep the unroll even (see above)");
    auto at = [&](uint64_t w, uint32_t s) { return rec[(w * kSets + s) * kWave + lane]; };
    WalkRec qa[kPrefetch], qb[kPrefetch];
#pragma unroll
    for (int i = 0; i < kPrefetch; i++) {
        qa[i] = at(i, 0);
        qb[i] = at(i, 1);
    }
    // Let the first records land before the loop: the wait the compiler
    // places at the loop head must hold on entry as well as on the
    // back-edge, and with these loads in flight on entry it would wait for
    // every record in flight on each iteration.  (s_waitcnt vmcnt(0),
    // expcnt and lgkmcnt unconstrained, in the gfx9 encoding.)
    __builtin_amdgcn_s_waitcnt(0x0F70);
    for (uint64_t w = 0; w < nw; w += kPrefetch) {
#pragma unroll
        for (int i = 0; i < kPrefetch; i++) {
            window(qa[i], qb[i], w + i);
            qa[i] = at(w + kPrefetch + i, 0);
            qb[i] = at(w + kPrefetch + i, 1);
        }
    }
    __syncthreads();
    for (uint32_t d = lane; d < n_live && d < kFastMaxLive; d += kWave)
        loads[live_ids[d]] = b0 + (int64_t)L[d];
}

#undef DM_WALK_BLOCK
#undef DM_SET_OPERANDS
#undef DM_SIZE_CHECK
#undef DM_STEP_PAIR
#undef DM_STEP_TEXT

// One wave: 32-bit relative loads unless plan[2] asks for 64-bit ones.
__global__ __launch_bounds__(kWave) void select_fast_kernel(
    const WalkRec* __restrict__ rec, const uint32_t* __restrict__ nwin,
    const uint32_t* __restrict__ live_ids, uint32_t n_live, int64_t* __restrict__ loads,
    const uint32_t* __restrict__ plan,
    const int64_t* __restrict__ base, longlong2* __restrict__ lpre, int64_t tbase, int64_t per,
    uint32_t qshift, int64_t slo, uint32_t policy)
{
    // Claim the whole register file of this wave's SIMD (256 + 256
    // registers), so that no wave of another kernel shares its issue slots:
    // this single wave is the serial critical path of a batch, and with
    // pipelining the next batch's kernels run beside it.
    asm volatile("" ::: "v255", "a255");
    if (!plan[1])
        return;
    __shared__ int64_t L[kFastMaxLive + kWave];  // loads, then one spare slot per lane
    const int64_t b0 = plan[2] ? base[0] : 0;  // 32-bit walks use absolute loads
    if (plan[2])
        walk_windows<int64_t>(rec, nwin, live_ids, n_live, loads, b0, lpre, tbase, per, qshift, slo,
                              policy, L);
    else
        walk_windows<int32_t>(rec, nwin, live_ids, n_live, loads, b0, lpre, tbase, per, qshift, slo,
                              policy, reinterpret_cast<int32_t*>(L));
}

__global__ void sel_out_kernel(const int64_t* __restrict__ offsets, uint64_t n, uint32_t bshift,
                               const uint32_t* __restrict__ cand, const uint32_t* __restrict__ match,
                               const longlong2* __restrict__ lpre,
                               const uint32_t* __restrict__ slot_of, uint64_t nslots,
                               const int64_t* __restrict__ base,
                               const uint32_t* __restrict__ plan, uint8_t* __restrict__ flags,
                               uint32_t* __restrict__ chosen, int64_t* __restrict__ ttft,
                               int64_t tbase, int64_t per, uint32_t qshift, int64_t slo,
                               uint32_t policy)
{
    if (!plan[1])
        return;
    const bool wide = plan[2] != 0;
    const int64_t b0 = wide ? base[0] : 0;
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        SelRec s = load_rec(offsets, n, r, true, bshift, cand, match, tbase, per, qshift, slo,
                            policy);
        const uint32_t q = slot_of[r];
        if (q >= nslots)  // only when the packing failed, which the status reports
            continue;
        int64_t La, Lo;
        if (wide) {
            const longlong2 lp = lpre[q];
            La = lp.x;
            Lo = lp.y;
        } else {
            const int2 lp = reinterpret_cast<const int2*>(lpre)[q];
            La = lp.x;
            Lo = lp.y;
        }
        // the walk records (L_a, L_o); a is c2 when c2 has the longer match
        // (never under the least-load rule)
        const bool a_is_c2 = s.a2;
        store_out(s, r, b0 + (a_is_c2 ? Lo : La), b0 + (a_is_c2 ? La : Lo), flags, chosen, ttft,
                  tbase, per, qshift, slo);
    }
}

template <int R>
void launch_select(dm_ctx* c, hipStream_t st, const int64_t* offsets, uint64_t n, uint32_t bshift,
                   const dm_route_out* out, int64_t* loads, const uint32_t* plan)
{
    const dm_config& k = c->cfg;
    select_kernel<R><<<1, kWave, 0, st>>>(offsets, n, bshift, out->cand, out->match,
                                                 out->flags, out->chosen, out->ttft_us, loads,
                                                 k.max_slots, k.ttft_base_us, k.ttft_per_token_us,
                                                 c->shift_div, k.slo_us, c->policy, plan);
}


}  // namespace

// Work arrays of one batch in flight: packing records, the level kernel's
// outputs, walk records (room for every block's window capacity, then
// 2 * kPrefetch inert padding windows), pre-update loads (kPrefetch padding
// windows), each request's slot, base/plan words and growth bounds.  Two
// such sets live in the selection slot, one per batch parity.
struct SelBuf {
    SelPack* prep;
    WalkRec* rec;
    longlong2* lpre;
    uint32_t* info;
    uint32_t* slot_of;
    uint16_t* slotmap;
    uint8_t* wdepth;
    uint32_t* wcount;
    uint32_t* woff;
    uint32_t* total;
    int64_t* base;
    uint32_t* plan;
    unsigned long long* grow;
    BlockShape shape;  // requests per block, windows per block
    uint64_t nblk;   // request blocks
    uint64_t nslots; // walk slots that can hold a request
};

static size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

// Sizes of one set's arrays for a batch of n requests, in layout order.
static void sel_sizes(uint64_t n, size_t* sizes)
{
    const BlockShape bs = block_shape(n);
    const uint64_t nblk = (n + bs.block - 1) / bs.block;
    const uint64_t wcap = nblk * bs.wincap;
    const size_t z[] = {
        up256(n * sizeof(SelPack)),                                  // prep
        up256((wcap + 2 * kPrefetch) * kSets * kWave * sizeof(WalkRec)),  // rec
        up256((wcap + kPrefetch) * kSets * kWave * sizeof(longlong2)),    // lpre
        up256(n * sizeof(uint32_t)),                                 // info
        up256(n * sizeof(uint32_t)),                                 // slot_of
        up256(wcap * kSets * kWave * sizeof(uint16_t)),              // slotmap
        up256(wcap),                                                 // wdepth
        up256(nblk * sizeof(uint32_t)),                              // wcount
        up256(nblk * sizeof(uint32_t)),                              // woff
        256 + 256 + (kMaxSlots + 1) * sizeof(unsigned long long),   // total, base/plan, grow
    };
    for (int i = 0; i < 10; i++)
        sizes[i] = z[i];
}

uint64_t select_scratch_bytes(uint64_t n)
{
    size_t sizes[10], one = 0;
    sel_sizes(n, sizes);
    for (size_t z : sizes)
        one += z;
    return one;
}

static hipError_t sel_buffers(dm_ctx* c, uint64_t n, int par, SelBuf* b)
{
    hipError_t e = hipSuccess;
    b->shape = block_shape(n);
    b->nblk = (n + b->shape.block - 1) / b->shape.block;
    b->nslots = b->nblk * b->shape.wincap * kSets * kWave;
    size_t sizes[10];
    sel_sizes(n, sizes);
    const size_t one = select_scratch_bytes(n);
    uint8_t* sw = nullptr;
    if (c->arena.on) {
        // allocation-free call: unpipelined, one set
        sw = static_cast<uint8_t*>(scratch_get(c, kSelSlot, one, &e));
    } else {
        // The two sets sit sel_stride apart whatever this batch's size: a
        // smaller batch must not move its set into the other parity's, which
        // the batch before it may still be walking.  A larger batch widens
        // the stride only once every stream is idle.
        if (one > c->sel_stride) {
            if ((e = sync_streams(c)) != hipSuccess)
                return e;
            c->sel_stride = one;
        }
        sw = static_cast<uint8_t*>(scratch_get(c, kSelSlot, 2 * c->sel_stride, &e));
        if (sw)
            sw += par * c->sel_stride;
    }
    if (!sw)
        return e;
    uint8_t* at[10];
    for (int i = 0; i < 10; i++) {
        at[i] = sw;
        sw += sizes[i];
    }
    b->prep = reinterpret_cast<SelPack*>(at[0]);
    b->rec = reinterpret_cast<WalkRec*>(at[1]);
    b->lpre = reinterpret_cast<longlong2*>(at[2]);
    b->info = reinterpret_cast<uint32_t*>(at[3]);
    b->slot_of = reinterpret_cast<uint32_t*>(at[4]);
    b->slotmap = reinterpret_cast<uint16_t*>(at[5]);
    b->wdepth = at[6];
    b->wcount = reinterpret_cast<uint32_t*>(at[7]);
    b->woff = reinterpret_cast<uint32_t*>(at[8]);
    uint8_t* tail = at[9];
    b->total = reinterpret_cast<uint32_t*>(tail);
    b->base = reinterpret_cast<int64_t*>(tail + 256);
    b->plan = reinterpret_cast<uint32_t*>(tail + 256 + 128);
    b->grow = reinterpret_cast<unsigned long long*>(tail + 512);
    return hipSuccess;
}

static uint32_t block_shift(const dm_ctx* c)
{
    uint32_t bshift = 0;
    while ((1u << bshift) < c->cfg.block_size)
        bshift++;
    return bshift;
}

hipError_t select_prepare(dm_ctx* c, hipStream_t st, const int64_t* offsets, uint64_t n,
                          const dm_route_out* out, int par)
{
    SelBuf b;
    hipError_t e = sel_buffers(c, n, par, &b);
    if (e != hipSuccess)
        return e;
    const uint64_t fill_waves = (b.nblk * b.shape.wincap + 2 * kPrefetch) * kSets;
    if (b.nblk > 0x7FFFFFFFull || fill_waves > 0x7FFFFFFFull)
        return hipErrorInvalidValue;
    const uint32_t NL = c->n_live;
    sel_zero_kernel<<<1, 256, 0, st>>>(b.grow, NL);
    const dm_config& k = c->cfg;
    // few workgroups: each adds its per-instance growth sums to the global
    // ones with one atomic per instance, and those atomics meet on a few lines
    sel_prep_kernel<<<grid_for(n, 256, 512), 256, 0, st>>>(
        offsets, n, block_shift(c), out->cand, out->match, c->d_dense, NL, k.ttft_base_us,
        k.ttft_per_token_us, c->shift_div, k.slo_us, c->policy, b.prep, b.grow);
    if (b.nblk > 0) {
        if (b.shape.block == LevelShape<2048>::block)
            sel_level_kernel<2048><<<(uint32_t)b.nblk, kWave, 0, st>>>(
                b.prep, n, b.info, b.slotmap, b.wdepth, b.wcount, c->d_status);
        else
            sel_level_kernel<1024><<<(uint32_t)b.nblk, kWave, 0, st>>>(
                b.prep, n, b.info, b.slotmap, b.wdepth, b.wcount, c->d_status);
    }
    sel_scan_kernel<<<1, 1024, 0, st>>>(b.wcount, b.nblk, b.woff, b.total);
    sel_fill_kernel<<<(uint32_t)((fill_waves + 3) / 4), 4 * kWave, 0, st>>>(
        b.prep, n, b.info, b.slotmap, b.wdepth, b.wcount, b.woff, b.total, b.nblk, b.shape,
        b.rec, b.slot_of);
    return hipGetLastError();
}

hipError_t select_run(dm_ctx* c, hipStream_t ss, hipStream_t os, hipEvent_t sel_done,
                      const int64_t* offsets, uint64_t n, const dm_route_out* out,
                      int64_t* loads, int par)
{
    SelBuf b;
    hipError_t e = sel_buffers(c, n, par, &b);
    if (e != hipSuccess)
        return e;
    const dm_config& k = c->cfg;
    const uint32_t S = k.max_slots, NL = c->n_live, bshift = block_shift(c);
    sel_base_kernel<<<1, 256, 0, ss>>>(loads, c->d_live_ids, NL, b.base, b.grow);
    sel_plan_kernel<<<1, 256, 0, ss>>>(loads, c->d_live_ids, NL, b.base, b.grow, c->policy,
                                       b.plan);
    select_fast_kernel<<<1, kWave, 0, ss>>>(b.rec, b.total, c->d_live_ids, NL, loads, b.plan,
                                            b.base, b.lpre, k.ttft_base_us, k.ttft_per_token_us,
                                            c->shift_div, k.slo_us, c->policy);
    if (S <= 64)
        launch_select<1>(c, ss, offsets, n, bshift, out, loads, b.plan);
    else if (S <= 128)
        launch_select<2>(c, ss, offsets, n, bshift, out, loads, b.plan);
    else if (S <= 192)
        launch_select<3>(c, ss, offsets, n, bshift, out, loads, b.plan);
    else if (S <= 256)
        launch_select<4>(c, ss, offsets, n, bshift, out, loads, b.plan);
    else
        select_lds_kernel<<<1, kWave, 0, ss>>>(offsets, n, bshift, out->cand, out->match,
                                               out->flags, out->chosen, out->ttft_us, loads, S,
                                               k.ttft_base_us, k.ttft_per_token_us, c->shift_div,
                                               k.slo_us, c->policy, b.plan);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (os != ss) {
        if ((e = hipEventRecord(sel_done, ss)) != hipSuccess ||
            (e = hipStreamWaitEvent(os, sel_done, 0)) != hipSuccess)
            return e;
    }
    sel_out_kernel<<<grid_for(n, 256, 8192), 256, 0, os>>>(
        offsets, n, bshift, out->cand, out->match, b.lpre, b.slot_of, b.nslots, b.base, b.plan,
        out->flags, out->chosen, out->ttft_us, k.ttft_base_us, k.ttft_per_token_us, c->shift_div,
        k.slo_us, c->policy);
    return hipGetLastError();
}

hipError_t select_batch(dm_ctx* c, hipStream_t st, const int64_t* offsets, uint64_t n,
                        const dm_route_out* out, int64_t* loads)
{
    hipError_t e = select_prepare(c, st, offsets, n, out, 0);
    if (e == hipSuccess)
        e = select_run(c, st, st, nullptr, offsets, n, out, loads, 0);
    return e;
}

}  // namespace dm
