// dm_rebalance: one non-recursive, single-round hotspot migration pass
// (Sec. 3.3, Eq. of the migration benefit; Sec. A.1.2).
//
// A stalled instance (decode-bottleneck telemetry, Sec. A.7) has its
// interval D added to every TTFT estimated on it; the comparisons below use
// the equivalent per-instance bound "TTFT without D against SLO - D".
//
// Pass-start state in parallel:
//   queue scan    per instance: each record's TTFT behind the base work and
//                 the records ahead of it; load; max TTFT; decode delay;
//                 overloaded flag;
//   benefit       per record: B = TTFT here - TTFT on the alternative;
//                 eligible if B > 0, source overloaded, target not;
//   source ranks  overloaded instances by (load desc, id asc);
//   ordering      eligible records sorted by (source rank, B desc,
//                 queue position asc) with stable radix passes (compaction
//                 already leaves them in record order, which is queue order
//                 within a source), and a second order grouping each
//                 source's records by target, cut into (source, target)
//                 segments.
// Then the sources are committed one after another by one workgroup.  For a
// source, the sequential rule "stop once the queue meets the SLO; move a
// record iff its TTFT on the target with the target's current load is below
// the SLO" is evaluated exactly as:
//   (i)  acceptance ignoring the stop: a record's acceptance depends only on
//        its target's load, so the targets' segments are walked
//        independently, each wave taking a run of whole segments 64 records
//        at a time.  The first undecided record of a segment has an exact
//        target load; if it is accepted, the following records are accepted
//        up to the first that fails with all of them accepted, if rejected,
//        they are rejected up to the first that passes at the same load, and
//        that record takes the other decision.  Each round settles such a run
//        in every segment at once (prefix sums give the loads), so a chunk
//        needs as many rounds as its segments have decision changes -- the
//        sequential walk's result exactly;
//   (ii) the stop only truncates that acceptance sequence and removing
//        records never raises a queued TTFT, so the number k of accepted
//        records that move is the smallest k after which the queue meets the
//        SLO -- found by bisection; each probe is one pass over the queue,
//        held in registers (a contiguous run of records per thread) when it
//        fits, with one workgroup scan and one vote per probe;
//   (iii) the first k accepted records move; target loads grow, the source's
//        shrinks.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kQThreads = 256;
constexpr uint32_t kQSplit = 16;  // workgroups per queue in the queue scan
constexpr int kCommitThreads = 512;
constexpr int kCommitWaves = kCommitThreads / kWave;
constexpr int kWalkBatch = 16;   // records loaded ahead of a dependent pass
constexpr int kWalkChunks = 4;   // 64-record chunks of an acceptance walk loaded together
constexpr int kQueueRegs = 64;   // queue records per thread held in registers
constexpr int kCommitBatch = 16; // candidates whose loads are in flight together in the commit
// acceptance bits of up to 262,144 candidates per source live in LDS; a
// source with more uses the same layout in device memory
constexpr uint32_t kLdsBitWords = 8192;
constexpr uint32_t kNoKey = 0xFFFFFFFFu;
// Passes with at most this many overloaded sources run each source's commit
// phases as kernels over the whole GPU; more sources, one workgroup for all.
constexpr uint32_t kSpreadSources = 64;

struct TtftK {
    int64_t base, per;
    uint32_t shift;
    int64_t slo;
    __device__ int64_t operator()(int64_t unc, int64_t load) const
    {
        return base + per * unc + (load >> shift);
    }
};

template <int NT>
__device__ int64_t block_excl_scan_i64(int64_t v, int64_t* sh, int64_t& total)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t inc = wave_incl_sum_u64((uint64_t)v, lane);
    if (lane == 63)
        sh[w] = (int64_t)inc;
    __syncthreads();
    int64_t before = 0, tot = 0;
    for (int k = 0; k < NT / kWave; k++) {
        if (k < w)
            before += sh[k];
        tot += sh[k];
    }
    __syncthreads();
    total = tot;
    return before + (int64_t)inc - v;
}

template <int NT>
__device__ int64_t block_max_i64(int64_t v, int64_t* sh)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const uint64_t o = shfl_u64((uint64_t)v, lane ^ d);
        v = std::max(v, (int64_t)o);
    }
    if (lane == 0)
        sh[w] = v;
    __syncthreads();
    int64_t m = sh[0];
    for (int k = 1; k < NT / kWave; k++)
        m = std::max(m, sh[k]);
    __syncthreads();
    return m;
}

// Per-queue TTFTs, loads and the overloaded set, each queue cut into kQSplit
// slices of contiguous records so that every queue spreads over kQSplit
// workgroups: slice sums; then each slice's records behind the base work and
// the slices ahead of it (largest TTFT per slice); then per instance the load
// and whether its largest queued TTFT exceeds the SLO.
__device__ __forceinline__ bool queue_ok(const int64_t* qoff, uint32_t i, uint64_t Q)
{
    const int64_t lo = qoff[i], hi = qoff[i + 1];
    return lo >= 0 && hi >= lo && hi <= (int64_t)Q;
}

__device__ __forceinline__ void slice_of(const int64_t* qoff, uint32_t i, uint32_t p, int64_t& b0,
                                         int64_t& b1)
{
    const int64_t lo = qoff[i], n = qoff[i + 1] - lo;
    b0 = lo + (int64_t)((uint64_t)n * p / kQSplit);
    b1 = lo + (int64_t)((uint64_t)n * (p + 1) / kQSplit);
}

__global__ __launch_bounds__(kQThreads) void queue_sum_kernel(
    const int64_t* __restrict__ qoff, uint64_t Q, const uint32_t* __restrict__ unc_here,
    int64_t* __restrict__ slice_sum, uint32_t* __restrict__ status)
{
    __shared__ int64_t sh[kQThreads / kWave];
    const uint32_t i = blockIdx.x / kQSplit, p = blockIdx.x % kQSplit;
    if (!queue_ok(qoff, i, Q)) {
        if (threadIdx.x == 0) {
            atomicOr(status, kErrInval);
            slice_sum[blockIdx.x] = 0;
        }
        return;
    }
    int64_t b0, b1;
    slice_of(qoff, i, p, b0, b1);
    int64_t sum = 0;
    for (int64_t b = b0 + threadIdx.x * kWalkBatch; b < b1; b += kQThreads * kWalkBatch) {
        uint32_t ub[kWalkBatch];
#pragma unroll
        for (int r = 0; r < kWalkBatch; r++)
            ub[r] = b + r < b1 ? unc_here[b + r] : 0u;
#pragma unroll
        for (int r = 0; r < kWalkBatch; r++)
            sum += ub[r];
    }
    int64_t tot;
    (void)block_excl_scan_i64<kQThreads>(sum, sh, tot);
    if (threadIdx.x == 0)
        slice_sum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kQThreads) void queue_ttft_kernel(
    const int64_t* __restrict__ qoff, uint64_t Q, const uint32_t* __restrict__ unc_here,
    const uint32_t* __restrict__ alt, const int64_t* __restrict__ base_work,
    const int64_t* __restrict__ slice_sum, uint32_t S, TtftK tk, int64_t* __restrict__ T,
    uint32_t* __restrict__ owner, int64_t* __restrict__ slice_max, uint32_t* __restrict__ status)
{
    __shared__ int64_t sh[kQThreads / kWave];
    const uint32_t i = blockIdx.x / kQSplit, p = blockIdx.x % kQSplit;
    if (!queue_ok(qoff, i, Q)) {
        if (threadIdx.x == 0)
            slice_max[blockIdx.x] = INT64_MIN;
        return;
    }
    int64_t b0, b1;
    slice_of(qoff, i, p, b0, b1);
    int64_t run0 = base_work[i];
    for (uint32_t k = 0; k < p; k++)
        run0 += slice_sum[i * kQSplit + k];
    // contiguous runs of the slice per thread, placed by one workgroup scan
    const uint64_t n = (uint64_t)(b1 - b0), per = (n + kQThreads - 1) / kQThreads;
    const int64_t r0 = b0 + (int64_t)std::min<uint64_t>(n, threadIdx.x * per);
    const int64_t r1 = b0 + (int64_t)std::min<uint64_t>(n, (threadIdx.x + 1) * per);
    int64_t sum = 0;
    for (int64_t b = r0; b < r1; b += kWalkBatch) {
        uint32_t ub[kWalkBatch];
#pragma unroll
        for (int r = 0; r < kWalkBatch; r++)
            ub[r] = b + r < r1 ? unc_here[b + r] : 0u;
#pragma unroll
        for (int r = 0; r < kWalkBatch; r++)
            sum += ub[r];
    }
    int64_t tot;
    int64_t run = run0 + block_excl_scan_i64<kQThreads>(sum, sh, tot);
    int64_t mx = INT64_MIN;
    bool bad = false;
    for (int64_t b = r0; b < r1; b += kWalkBatch) {
        uint32_t ub[kWalkBatch], ab[kWalkBatch];
#pragma unroll
        for (int r = 0; r < kWalkBatch; r++) {
            const bool in = b + r < r1;
            ub[r] = in ? unc_here[b + r] : 0u;
            ab[r] = in ? alt[b + r] : 0u;
        }
#pragma unroll
        for (int r = 0; r < kWalkBatch; r++) {
            if (b + r < r1) {
                const int64_t t = tk((int64_t)ub[r], run);
                T[b + r] = t;
                owner[b + r] = i;
                mx = std::max(mx, t);
                bad |= ab[r] >= S;
                run += ub[r];
            }
        }
    }
    if (bad)
        atomicOr(status, kErrInval);
    mx = block_max_i64<kQThreads>(mx, sh);
    if (threadIdx.x == 0)
        slice_max[blockIdx.x] = mx;
}

// Decode delay D of a stalled instance (non-empty queue, prefill interval
// above the threshold), else 0; intervals outside [0, 2^40] are rejected.
__global__ void queue_over_kernel(const int64_t* __restrict__ qoff, uint64_t Q,
                                  const int64_t* __restrict__ base_work,
                                  const int64_t* __restrict__ slice_sum,
                                  const int64_t* __restrict__ slice_max, uint32_t S, int64_t slo,
                                  const int64_t* __restrict__ interval, int64_t thresh,
                                  int64_t* __restrict__ L0, uint8_t* __restrict__ over,
                                  int64_t* __restrict__ delay, int64_t* __restrict__ slo_of,
                                  uint32_t* __restrict__ status)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= S)
        return;
    int64_t L = base_work[i], mx = INT64_MIN;
    const bool ok = queue_ok(qoff, i, Q);
    if (ok)
        for (uint32_t k = 0; k < kQSplit; k++) {
            L += slice_sum[i * kQSplit + k];
            mx = std::max(mx, slice_max[i * kQSplit + k]);
        }
    const bool busy = ok && qoff[i + 1] > qoff[i];
    int64_t d = 0;
    if (interval) {
        const int64_t v = interval[i];
        if (v < 0 || v > (int64_t(1) << 40))
            atomicOr(status, kErrInval);
        else if (busy && v > thresh)
            d = v;
    }
    L0[i] = L;
    delay[i] = d;
    slo_of[i] = slo - d;
    over[i] = (busy && mx > slo - d) ? 1 : 0;
}

// Per record: benefit and eligibility; the largest eligible benefit goes to
// *maxb (it sizes the sort key).
__global__ __launch_bounds__(256) void benefit_kernel(
    uint64_t Q, const int64_t* __restrict__ T, const uint32_t* __restrict__ owner,
    const uint32_t* __restrict__ alt, const uint32_t* __restrict__ unc_alt,
    const int64_t* __restrict__ L0, const uint8_t* __restrict__ over,
    const int64_t* __restrict__ delay, uint32_t S, TtftK tk, int64_t* __restrict__ benefit,
    uint64_t* __restrict__ elig, uint64_t* __restrict__ maxb)
{
    __shared__ int64_t sh[256 / kWave];
    int64_t mx = 0;
    for (uint64_t q = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; q < Q;
         q += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t i = owner[q], j = alt[q];
        bool e = false;
        int64_t b = 0;
        if (i < S && j < S && over[i]) {
            b = (T[q] + delay[i]) - (tk((int64_t)unc_alt[q], L0[j]) + delay[j]);
            e = b > 0 && !over[j];
        }
        benefit[q] = b;
        elig[q] = e ? 1 : 0;
        if (e)
            mx = std::max(mx, b);
    }
    mx = block_max_i64<256>(mx, sh);
    if (threadIdx.x == 0 && mx > 0)
        atomicMax((unsigned long long*)maxb, (unsigned long long)mx);
}

// rank[i] of overloaded instance i among (load desc, id asc); src[rank] = i.
__global__ __launch_bounds__(256) void rank_kernel(const int64_t* __restrict__ L0,
                                                   const uint8_t* __restrict__ over, uint32_t S,
                                                   uint32_t* __restrict__ rank,
                                                   uint32_t* __restrict__ src,
                                                   uint32_t* __restrict__ nsrc)
{
    __shared__ int64_t sl[kMaxSlots];
    __shared__ uint8_t so[kMaxSlots];
    for (uint32_t k = threadIdx.x; k < S; k += blockDim.x) {
        sl[k] = L0[k];
        so[k] = over[k];
    }
    __syncthreads();
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= S || !so[i])
        return;
    uint32_t r = 0;
    for (uint32_t k = 0; k < S; k++)
        r += so[k] && (sl[k] > sl[i] || (sl[k] == sl[i] && k < i));
    rank[i] = r;
    src[r] = i;
    atomicAdd(nsrc, 1u);
}

__global__ void zero_u32_kernel(uint32_t* p, uint32_t n)
{
    for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x)
        p[k] = 0;
}

__global__ void fill_u32_kernel(uint32_t* p, uint64_t n, uint32_t v)
{
    for (uint64_t k = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; k < n;
         k += (uint64_t)gridDim.x * blockDim.x)
        p[k] = v;
}

// Eligible records in record order (queue order within each source).
__global__ void compact_kernel(uint64_t Q, const uint64_t* __restrict__ elig,
                               const uint64_t* __restrict__ pos, uint32_t* __restrict__ vals)
{
    for (uint64_t q = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; q < Q;
         q += (uint64_t)gridDim.x * blockDim.x)
        if (elig[q])
            vals[pos[q]] = (uint32_t)q;
}

// keys[t] = a key of the record (or candidate index) held in vals[t].
// kByRankBenefit: (source rank, benefit descending in its low `sh` bits) of
// record vals[t]; kByRankTarget: (source rank, target in `sh` bits) of
// candidate vals[t]; kByBenefitDesc / kBySourceRank: the two halves of the
// first, for benefits too wide to share a key with the rank.
enum KeyKind { kByRankBenefit, kByRankTarget, kByBenefitDesc, kBySourceRank };

__global__ void rekey_kernel(uint64_t C, int kind, uint32_t sh, const uint32_t* __restrict__ vals,
                             const uint32_t* __restrict__ cand_q, const int64_t* __restrict__ benefit,
                             const uint32_t* __restrict__ owner, const uint32_t* __restrict__ rank,
                             const uint32_t* __restrict__ alt, uint64_t* __restrict__ keys)
{
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < C;
         t += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t v = vals[t];
        uint64_t k = 0;
        switch (kind) {
            case kByRankBenefit:
                k = ((uint64_t)rank[owner[v]] << sh) |
                    (((1ull << sh) - 1) - (uint64_t)benefit[v]);
                break;
            case kByRankTarget: {
                const uint32_t q = cand_q[v];
                k = ((uint64_t)rank[owner[q]] << sh) | alt[q];
                break;
            }
            case kByBenefitDesc: k = ~(uint64_t)benefit[v]; break;
            case kBySourceRank: k = rank[owner[v]]; break;
        }
        keys[t] = k;
    }
}

inline int bit_length(uint64_t x)
{
    int n = 0;
    while (x) {
        n++;
        x >>= 1;
    }
    return n;
}

__global__ void iota_kernel(uint64_t C, uint32_t* __restrict__ v)
{
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < C;
         t += (uint64_t)gridDim.x * blockDim.x)
        v[t] = (uint32_t)t;
}

// start[r] = first candidate of source rank r (r = 0..nsrc).
__global__ void bounds_kernel(uint64_t C, const uint32_t* __restrict__ cand_q,
                              const uint32_t* __restrict__ owner, const uint32_t* __restrict__ rank,
                              const uint32_t* __restrict__ nsrc_p, uint32_t* __restrict__ start)
{
    const uint32_t nsrc = *nsrc_p;
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t <= C;
         t += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t lo = t == 0 ? 0 : rank[owner[cand_q[t - 1]]] + 1;
        const uint32_t hi = t == C ? nsrc : rank[owner[cand_q[t]]];
        for (uint32_t r = lo; r <= hi; r++)
            start[r] = (uint32_t)t;
    }
}

// Per grouped position u: target, its uncached tokens, candidate index.
__global__ void gather_groups_kernel(uint64_t C, const uint32_t* __restrict__ grp,
                                     const uint32_t* __restrict__ cand_q,
                                     const uint32_t* __restrict__ alt,
                                     const uint32_t* __restrict__ unc_alt,
                                     uint32_t* __restrict__ g_alt, uint32_t* __restrict__ g_unc)
{
    for (uint64_t u = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; u < C;
         u += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t q = cand_q[grp[u]];
        g_alt[u] = alt[q];
        g_unc[u] = unc_alt[q];
    }
}

// Per candidate t (candidate order): the record's fields a commit writes.
__global__ void gather_cand_kernel(uint64_t C, const uint32_t* __restrict__ cand_q,
                                   const uint64_t* __restrict__ rec_id,
                                   const uint32_t* __restrict__ alt,
                                   const uint32_t* __restrict__ unc_alt,
                                   const uint32_t* __restrict__ unc_here,
                                   const int64_t* __restrict__ benefit, uint64_t* __restrict__ c_rec,
                                   uint32_t* __restrict__ c_alt, uint32_t* __restrict__ c_ua,
                                   uint32_t* __restrict__ c_uh, int64_t* __restrict__ c_ben)
{
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < C;
         t += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t q = cand_q[t];
        c_rec[t] = rec_id[q];
        c_alt[t] = alt[q];
        c_ua[t] = unc_alt[q];
        c_uh[t] = unc_here[q];
        c_ben[t] = benefit[q];
    }
}

// head[u] = 1 where grouped position u starts a (source, target) segment.
__global__ void seg_head_kernel(uint64_t C, const uint32_t* __restrict__ grp,
                                const uint32_t* __restrict__ cand_q,
                                const uint32_t* __restrict__ owner,
                                const uint32_t* __restrict__ rank,
                                const uint32_t* __restrict__ g_alt, uint64_t* __restrict__ head)
{
    for (uint64_t u = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; u < C;
         u += (uint64_t)gridDim.x * blockDim.x) {
        bool h = u == 0 || g_alt[u] != g_alt[u - 1];
        if (!h)
            h = rank[owner[cand_q[grp[u]]]] != rank[owner[cand_q[grp[u - 1]]]];
        head[u] = h ? 1 : 0;
    }
}

// seg_pos[g] = first grouped position of segment g (seg_pos[nseg] = C);
// sseg[r] = first segment of source rank r (sseg[nsrc] = nseg).
__global__ void seg_pos_kernel(uint64_t C, uint32_t S, const uint64_t* __restrict__ head,
                               const uint64_t* __restrict__ sid, const uint64_t* __restrict__ nseg_p,
                               const uint32_t* __restrict__ start,
                               const uint32_t* __restrict__ nsrc_p, uint32_t* __restrict__ seg_pos,
                               uint32_t* __restrict__ sseg)
{
    const uint32_t nseg = C ? (uint32_t)*nseg_p : 0u, nsrc = *nsrc_p;
    const uint64_t end = C > S ? C : S;
    for (uint64_t u = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; u <= end;
         u += (uint64_t)gridDim.x * blockDim.x) {
        if (u == C)
            seg_pos[nseg] = (uint32_t)C;
        else if (u < C && head[u])
            seg_pos[sid[u]] = (uint32_t)u;
        if (u <= nsrc)
            sseg[u] = start[u] < C ? (uint32_t)sid[start[u]] : nseg;
    }
}

__global__ void copy_i64_kernel(const int64_t* __restrict__ a, int64_t* __restrict__ b, uint32_t n)
{
    for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x)
        b[k] = a[k];
}

struct CommitArgs {
    const int64_t* qoff;
    const uint64_t* rec_id;
    const uint32_t* unc_here;
    const uint32_t* alt;
    const uint32_t* unc_alt;
    const int64_t* base_work;
    const int64_t* benefit;
    const uint32_t* src;      // [nsrc] instance of each rank
    const uint32_t* nsrc;
    const uint32_t* start;    // [nsrc + 1]
    const uint32_t* sseg;     // [nsrc + 1] first segment of each rank
    const uint32_t* seg_pos;  // [nseg + 1] first grouped position of each segment
    const uint32_t* cand_q;   // [C] record of candidate t
    const uint64_t* c_rec;    // [C] rec_id, alt, unc_alt, unc_here, benefit of candidate t
    const uint32_t* c_alt;
    const uint32_t* c_ua;
    const uint32_t* c_uh;
    const int64_t* c_ben;
    const uint32_t* grp;      // [C] candidate order grouped by (rank, target)
    const uint32_t* g_alt;    // [C] target of grp[u]
    const uint32_t* g_unc;    // [C] unc_alt of grp[u]
    uint32_t* gbits;          // [C / 32 + 1] acceptance bits when LDS cannot hold them
    uint32_t* gwpre;          // [C / 32 + 1] accepted candidates before each bit word
    int64_t* tto;             // [C]
    uint32_t* arank;          // [C] acceptance rank of candidate t, kNoKey if not accepted
    uint32_t* kstar_of;       // [nsrc] accepted records that move, per source rank
    uint64_t* base_of;        // [nsrc] their first index in the migration list
    uint32_t* qkey;           // [Q]
    int64_t* loads;           // [S] in: pass-start loads; out: loads after the pass
    const int64_t* delay;     // [S] decode delay per instance (0 unless stalled)
    const int64_t* slo_of;    // [S] the SLO less each instance's decode delay
    uint32_t* wpre_src;       // [C / 32 + 2] per source: accepted candidates before each word
    uint32_t* acc_of;         // [nsrc] accepted candidates per source
    unsigned long long* run;  // [1] migrations so far (sources in rank order)
    uint32_t S;
    TtftK tk;
    uint64_t cap;
    uint64_t* out_rec;
    uint32_t* out_from;
    uint32_t* out_to;
    int64_t* out_benefit;
    int64_t* out_ttft;
    uint64_t* out_count;
    uint32_t* status;
};

// Whether a record of queue [lo, hi) whose key is >= k (one still queued
// after the first k accepted records left) exceeds the SLO behind the base
// work and the records still ahead of it.  Chunked form, for queues longer
// than the register form holds.
__device__ bool queue_violates_chunked(const CommitArgs& a, const TtftK& tk, int64_t lo, int64_t hi,
                                       int64_t w0, uint32_t k, int64_t* sh)
{
    int64_t run = w0;
    bool v = false;
    for (int64_t b = lo; b < hi; b += kCommitThreads) {
        const int64_t q = b + threadIdx.x;
        const bool keep = q < hi && a.qkey[q] >= k;
        const int64_t u = keep ? (int64_t)a.unc_here[q] : 0;
        int64_t tot;
        const int64_t ex = block_excl_scan_i64<kCommitThreads>(u, sh, tot);
        if (keep)
            v |= tk(u, run + ex) > tk.slo;
        run += tot;
    }
    return __syncthreads_or(v) != 0;
}

// The same test with the queue in registers: thread x holds a contiguous run
// of records (key 0 marks an empty register: k >= 1 never keeps it).
__device__ __forceinline__ bool regs_violate(uint32_t (&u)[kQueueRegs],
                                             const uint32_t (&key)[kQueueRegs], int64_t w0,
                                             uint32_t k, const TtftK& tk, int64_t* sh)
{
    int64_t sum = 0;
#pragma unroll
    for (int r = 0; r < kQueueRegs; r++) {
        // keep per-record products out of registers across probes
        asm volatile("" : "+v"(u[r]));
        sum += key[r] >= k ? (int64_t)u[r] : 0;
    }
    int64_t tot;
    int64_t run = w0 + block_excl_scan_i64<kCommitThreads>(sum, sh, tot);
    asm volatile("" : "+v"(k));  // recompute the keep masks rather than hold 32 of them
    bool v = false;
#pragma unroll
    for (int r = 0; r < kQueueRegs; r++) {
        const bool keep = key[r] >= k;
        v |= keep && tk((int64_t)u[r], run) > tk.slo;
        run += keep ? (int64_t)u[r] : 0;
    }
    return __syncthreads_or(v) != 0;
}

// Acceptance bits: one per candidate of the current source, in candidate
// order.  The pointer is generic (LDS or device memory); every access is an
// atomic performed where the word lives.
__device__ __forceinline__ uint32_t bits_word(const uint32_t* w)
{
    return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Orders every memory access before it, LDS and device memory, for the whole
// workgroup.
__device__ __forceinline__ void wg_sync()
{
    __threadfence();
    __syncthreads();
}

// Smallest k in [1, A] after which queue [qlo, qlo + Lq) meets the SLO (A if
// none), the queue held in registers.  Kept out of line: the probes get the
// whole register file, and the caller's state is saved once per source.
__device__ __noinline__ uint32_t regs_bisect(const uint32_t* __restrict__ unc_here,
                                             const uint32_t* __restrict__ qkey, int64_t qlo,
                                             uint64_t Lq, int64_t w0, uint32_t A, TtftK tk,
                                             int64_t* sh)
{
    const uint32_t tid = threadIdx.x;
    const uint64_t pq = (Lq + kCommitThreads - 1) / kCommitThreads;
    const int64_t b0 = qlo + (int64_t)std::min<uint64_t>(Lq, tid * pq);
    const int64_t b1 = qlo + (int64_t)std::min<uint64_t>(Lq, (tid + 1) * pq);
    uint32_t u[kQueueRegs], key[kQueueRegs];
    // 16-byte loads where the run is aligned: a quarter of the address
    // requests of scalar loads, whose lanes each touch another cache line
    const bool vec = (b0 & 3) == 0 && (reinterpret_cast<uintptr_t>(unc_here) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(qkey) & 15) == 0;
#pragma unroll
    for (int k = 0; k < kQueueRegs / 4; k++) {
        const int64_t q = b0 + 4 * k;
        if (vec && q + 3 < b1) {
            const uint4 x = *reinterpret_cast<const uint4*>(unc_here + q);
            const uint4 y = *reinterpret_cast<const uint4*>(qkey + q);
            u[4 * k] = x.x;
            u[4 * k + 1] = x.y;
            u[4 * k + 2] = x.z;
            u[4 * k + 3] = x.w;
            key[4 * k] = y.x;
            key[4 * k + 1] = y.y;
            key[4 * k + 2] = y.z;
            key[4 * k + 3] = y.w;
        } else {
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const bool in = q + r < b1;
                u[4 * k + r] = in ? unc_here[q + r] : 0u;
                key[4 * k + r] = in ? qkey[q + r] : 0u;
            }
        }
    }
    uint32_t lo = 1, hi = A;
    if (regs_violate(u, key, w0, hi, tk, sh))
        return hi;
    while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (!regs_violate(u, key, w0, mid, tk, sh))
            hi = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

// Acceptance walk over grouped positions [P0, P1): whole (source, target)
// segments of the current source, by one wave (every lane active).  Sets the
// acceptance bit of each accepted candidate (bit t - cs) and stores every
// record's TTFT on its target at its turn.
__device__ __forceinline__ void walk_run(const CommitArgs& a, uint32_t* s_bits, uint32_t* g_bits,
                                         bool in_lds, const int64_t* s_L, const int64_t* s_slo,
                                         uint32_t cs, uint32_t P0, uint32_t P1)
{
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const uint64_t below = (1ull << lane) - 1;  // lanes under this one
    uint32_t carry_j = kNoKey;  // target of the segment open at the last chunk's end
    int64_t carry_L = 0;        // its load after the records walked so far
    uint32_t cu[kWalkChunks], ct[kWalkChunks], cj[kWalkChunks];
#pragma unroll
    for (int g = 0; g < kWalkChunks; g++) {
        const uint64_t v = (uint64_t)P0 + g * kWave + lane;
        const bool in = v < P1;
        cu[g] = in ? a.g_unc[v] : 0u;
        ct[g] = in ? a.grp[v] : 0u;
        cj[g] = in ? a.g_alt[v] : kNoKey;
    }
    for (uint64_t p = P0; p < P1; p += kWave * kWalkChunks) {
        uint32_t nu[kWalkChunks], nt[kWalkChunks], nj[kWalkChunks];
#pragma unroll
        for (int g = 0; g < kWalkChunks; g++) {
            const uint64_t v = p + (uint64_t)(kWalkChunks + g) * kWave + lane;
            const bool in = v < P1;
            nu[g] = in ? a.g_unc[v] : 0u;
            nt[g] = in ? a.grp[v] : 0u;
            nj[g] = in ? a.g_alt[v] : kNoKey;
        }
#pragma unroll
        for (int g = 0; g < kWalkChunks; g++) {
            const uint64_t pc = p + (uint64_t)g * kWave;
            if (pc >= P1)
                break;
            const bool valid = pc + lane < P1;
            const uint32_t u = cu[g], t = ct[g], j = cj[g];
            // the SLO less the target's decode delay; a run's records share
            // their target, so a record's bound is also its run start's
            const int64_t slo_j = valid ? s_slo[j] : a.tk.slo;
            uint32_t jprev = __shfl_up(j, 1);
            if (lane == 0)
                jprev = carry_j;
            const uint64_t H = __ballot(valid && j != jprev);
            const uint64_t self = 1ull << lane;
            const uint64_t hm = H & (below | self), nm = H & ~(below | self);
            const int seglo = hm ? 63 - __clzll(hm) : 0;  // my segment's lanes in this chunk
            const int seghi = nm ? __ffsll((long long)nm) - 2 : 63;
            const uint64_t segbits = (seghi == 63 ? ~0ull : (2ull << seghi) - 1) & ~((1ull << seglo) - 1);
            const uint64_t excl = wave_incl_sum_u64(u, lane) - u;
            // exact target load at the first unsettled record of a segment
            int64_t Lx = 0;
            if (valid && lane == seglo)
                Lx = (H & self) ? s_L[j] : carry_L;
            uint64_t U = __ballot(valid);  // unsettled records
            bool ok = false;
            int64_t Lt = 0;
            if ((H & ~1ull) == 0) {
                // one segment in this chunk: the same rounds with the first
                // undecided record and the run's end uniform, read by readlane
                int64_t Lf = (int64_t)readlane_u64((uint64_t)Lx, 0);
                while (U) {
                    const int f = __ffsll((long long)U) - 1;
                    const uint32_t uf = __builtin_amdgcn_readlane(u, f);
                    const uint64_t exf = readlane_u64(excl, f);
                    const bool pf = a.tk((int64_t)uf, Lf) < slo_j;
                    const int64_t Lv = pf ? Lf + (int64_t)(excl - exf) : Lf;
                    const bool pv = a.tk((int64_t)u, Lv) < slo_j;
                    const bool inU = (U >> lane) & 1;
                    const uint64_t sm = __ballot(inU && pv != pf);
                    const int st = sm ? __ffsll((long long)sm) - 1 : kWave;
                    if (inU && (int)lane <= st) {
                        ok = (int)lane < st ? pf : !pf;
                        Lt = Lv;
                    }
                    if (st == kWave)
                        break;
                    // the run's last record takes the other decision
                    Lf = (int64_t)readlane_u64((uint64_t)Lv, st) +
                         (pf ? 0 : (int64_t)__builtin_amdgcn_readlane(u, st));
                    U &= ~((2ull << st) - 1);
                }
                U = 0;
            }
            while (U) {
                // per segment: its first unsettled record f decides a run
                // (f accepted: records accepted until one fails; f rejected:
                // records rejected until one passes at f's load), and the
                // record ending the run takes the other decision
                const uint64_t fm = U & segbits;
                const int f = fm ? __ffsll((long long)fm) - 1 : (int)lane;
                const int64_t Lf = (int64_t)shfl_u64((uint64_t)Lx, f);
                const uint32_t uf = __shfl(u, f);
                const uint64_t exf = shfl_u64(excl, f);
                const bool pf = a.tk((int64_t)uf, Lf) < slo_j;
                const int64_t Lv = pf ? Lf + (int64_t)(excl - exf) : Lf;
                const bool pv = a.tk((int64_t)u, Lv) < slo_j;
                const bool inU = (U >> lane) & 1;
                const uint64_t sm = __ballot(inU && pv != pf) & segbits;
                const int st = sm ? __ffsll((long long)sm) - 1 : kWave;
                const bool settle = inU && (int)lane <= st;
                const bool d = (int)lane < st ? pf : !pf;
                const int64_t nxt = Lv + (d ? (int64_t)u : 0);
                const uint32_t plo = __shfl_up((uint32_t)nxt, 1);
                const uint32_t phi = __shfl_up((uint32_t)((uint64_t)nxt >> 32), 1);
                if (settle) {
                    ok = d;
                    Lt = Lv;
                } else if (inU && (int)lane == st + 1) {
                    Lx = (int64_t)(((uint64_t)phi << 32) | plo);
                }
                U &= ~__ballot(settle);
            }
            if (valid) {
                a.tto[t] = a.tk((int64_t)u, Lt) + (a.tk.slo - slo_j);
                if (ok) {
                    const uint32_t x = t - cs;
                    if (in_lds)
                        atomicOr(&s_bits[x >> 5], 1u << (x & 31));
                    else
                        atomicOr(&g_bits[x >> 5], 1u << (x & 31));
                }
            }
            const int last = (int)std::min<uint64_t>(kWave - 1, P1 - 1 - pc);
            carry_L = (int64_t)readlane_u64((uint64_t)(Lt + (ok ? (int64_t)u : 0)), last);
            carry_j = __builtin_amdgcn_readlane(j, last);
        }
#pragma unroll
        for (int g = 0; g < kWalkChunks; g++) {
            cu[g] = nu[g];
            ct[g] = nt[g];
            cj[g] = nj[g];
        }
    }
}

__global__ __launch_bounds__(kCommitThreads) void commit_kernel(CommitArgs a)
{
    __shared__ int64_t sh[kCommitThreads / kWave];
    __shared__ int64_t s_L[kMaxSlots];         // live loads of every instance
    __shared__ int64_t s_slo[kMaxSlots];       // SLO less each instance's decode delay
    __shared__ uint32_t s_bits[kLdsBitWords];
    __shared__ uint32_t s_wpre[kLdsBitWords];
    __shared__ uint64_t s_count;
    const uint32_t nsrc = *a.nsrc, S = a.S;
    const uint32_t tid = threadIdx.x;
    for (uint32_t j = tid; j < S; j += kCommitThreads) {
        s_L[j] = a.loads[j];
        s_slo[j] = a.tk.slo - a.delay[j];
    }
    if (tid == 0)
        s_count = 0;
    __syncthreads();
    for (uint32_t s = 0; s < nsrc; s++) {
        const uint32_t i = a.src[s];
        const uint32_t cs = a.start[s], ce = a.start[s + 1], nc = ce - cs;
        const uint32_t nw = (uint32_t)(((uint64_t)nc + 31) / 32);
        const bool in_lds = nw <= kLdsBitWords;
        uint32_t* bits = in_lds ? s_bits : a.gbits;
        uint32_t* wpre = in_lds ? s_wpre : a.gwpre;
        const int64_t qlo = a.qoff[i], qhi = a.qoff[i + 1];
        for (uint32_t w = tid; w < nw; w += kCommitThreads)
            __hip_atomic_store(&bits[w], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int64_t q = qlo + tid; q < qhi; q += kCommitThreads)
            a.qkey[q] = kNoKey;
        wg_sync();
        // (i) acceptance: each wave walks a run of whole segments
        {
            const uint32_t wv = tid / kWave, G0 = a.sseg[s], ng = a.sseg[s + 1] - G0;
            const uint32_t ga = G0 + (uint32_t)((uint64_t)ng * wv / kCommitWaves);
            const uint32_t gb = G0 + (uint32_t)((uint64_t)ng * (wv + 1) / kCommitWaves);
            if (ga < gb)
                walk_run(a, s_bits, a.gbits, in_lds, s_L, s_slo, cs, a.seg_pos[ga], a.seg_pos[gb]);
        }
        wg_sync();
        // (ii) acceptance ranks in candidate order: accepted candidates
        // before each bit word (a contiguous run of words per thread)
        const uint64_t pw = ((uint64_t)nw + kCommitThreads - 1) / kCommitThreads;
        const uint32_t w0 = (uint32_t)std::min<uint64_t>(nw, tid * pw);
        const uint32_t w1 = (uint32_t)std::min<uint64_t>(nw, (tid + 1) * pw);
        int64_t cnt = 0;
        for (uint32_t w = w0; w < w1; w++)
            cnt += __popc(in_lds ? s_bits[w] : bits_word(&bits[w]));
        int64_t A;
        uint32_t run = (uint32_t)block_excl_scan_i64<kCommitThreads>(cnt, sh, A);
        for (uint32_t w = w0; w < w1; w++) {
            if (in_lds)
                s_wpre[w] = run;
            else
                __hip_atomic_store(&wpre[w], run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            run += __popc(in_lds ? s_bits[w] : bits_word(&bits[w]));
        }
        wg_sync();
        // queue records of accepted candidates get their rank as key
        for (uint32_t b = cs + tid; b < ce; b += kCommitThreads * kWalkBatch) {
            uint32_t qb[kWalkBatch];
#pragma unroll
            for (int r = 0; r < kWalkBatch; r++) {
                const uint64_t t = b + (uint64_t)r * kCommitThreads;
                qb[r] = t < ce ? a.cand_q[t] : 0u;
            }
#pragma unroll
            for (int r = 0; r < kWalkBatch; r++) {
                const uint64_t t = b + (uint64_t)r * kCommitThreads;
                if (t < ce) {
                    const uint32_t x = (uint32_t)(t - cs), w = x >> 5, m = 1u << (x & 31);
                    const uint32_t word = in_lds ? s_bits[w] : bits_word(&bits[w]);
                    uint32_t rk = kNoKey;
                    if (word & m) {
                        rk = (in_lds ? s_wpre[w] : bits_word(&wpre[w])) + __popc(word & (m - 1));
                        a.qkey[qb[r]] = rk;
                    }
                    a.arank[t] = rk;
                }
            }
        }
        wg_sync();
        // smallest k in [1, A] after which the queue meets the SLO (A if none)
        uint32_t kstar = 0;
        if (A > 0) {
            const int64_t w0q = a.base_work[i];
            TtftK tks = a.tk;  // the source's queue against the SLO less its decode delay
            tks.slo = s_slo[i];
            const uint64_t Lq = (uint64_t)(qhi - qlo);
            uint32_t lo = 1, hi = (uint32_t)A;  // answer in [lo, hi]
            if (Lq <= (uint64_t)kCommitThreads * kQueueRegs) {
                lo = regs_bisect(a.unc_here, a.qkey, qlo, Lq, w0q, hi, tks, sh);
            } else {
                if (queue_violates_chunked(a, tks, qlo, qhi, w0q, hi, sh)) {
                    lo = hi;
                } else {
                    while (lo < hi) {
                        const uint32_t mid = lo + (hi - lo) / 2;
                        if (!queue_violates_chunked(a, tks, qlo, qhi, w0q, mid, sh))
                            hi = mid;
                        else
                            lo = mid + 1;
                    }
                }
            }
            kstar = lo;
        }
        // (iii) the first kstar accepted records move: target loads grow and
        // the source's shrinks, in LDS; emit_kernel writes the migrations
        const uint64_t base = s_count;
        if (tid == 0) {
            a.kstar_of[s] = kstar;
            a.base_of[s] = base;
        }
        int64_t dsrc = 0;
        for (uint32_t b = cs + tid; b < ce; b += kCommitThreads * kCommitBatch) {
            uint32_t rk[kCommitBatch], to[kCommitBatch], ua[kCommitBatch], uh[kCommitBatch];
#pragma unroll
            for (int r = 0; r < kCommitBatch; r++) {
                const uint64_t t = b + (uint64_t)r * kCommitThreads;
                const bool in = t < ce;
                rk[r] = in ? a.arank[t] : kNoKey;
                to[r] = in ? a.c_alt[t] : 0u;
                ua[r] = in ? a.c_ua[t] : 0u;
                uh[r] = in ? a.c_uh[t] : 0u;
            }
#pragma unroll
            for (int r = 0; r < kCommitBatch; r++) {
                if (rk[r] < kstar) {
                    atomicAdd((unsigned long long*)&s_L[to[r]], (unsigned long long)ua[r]);
                    dsrc += uh[r];
                }
            }
        }
        if (dsrc)
            atomicAdd((unsigned long long*)&s_L[i], (unsigned long long)(-dsrc));
        __syncthreads();
        if (tid == 0)
            s_count = base + kstar;
        __syncthreads();
    }
    for (uint32_t j = tid; j < S; j += kCommitThreads)
        a.loads[j] = s_L[j];
    if (tid == 0) {
        *a.out_count = s_count;
        if (s_count > a.cap)
            atomicOr(a.status, kErrFull);
    }
}


// ---------------------------------------------------------------------------
// The same commit spread over the GPU, one source at a time (the host
// launches these in source-rank order), for passes with few sources: every
// phase that the single workgroup above runs for a source becomes a kernel
// over all compute units, except the prefix of acceptance bits and the stop
// point, which stay on one workgroup.  The acceptance bits are indexed by
// candidate (all zero at the start of the pass); loads live in loads_out.
// ---------------------------------------------------------------------------

// Walk of source s's segments, one wave per segment; the blocks also reset
// the source's queue keys.
__global__ __launch_bounds__(256) void src_walk_kernel(CommitArgs a, uint32_t s)
{
    if (s >= *a.nsrc)
        return;
    const uint32_t i = a.src[s];
    const int64_t qlo = a.qoff[i], qhi = a.qoff[i + 1];
    for (int64_t q = qlo + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < qhi;
         q += (int64_t)gridDim.x * blockDim.x)
        a.qkey[q] = kNoKey;
    const uint64_t wv = blockIdx.x * (uint64_t)(blockDim.x >> 6) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t nwv = (uint64_t)gridDim.x * (blockDim.x >> 6);
    const uint32_t G0 = a.sseg[s], G1 = a.sseg[s + 1];
    for (uint64_t g = G0 + wv; g < G1; g += nwv)
        walk_run(a, nullptr, a.gbits, false, a.loads, a.slo_of, 0, a.seg_pos[g],
                 a.seg_pos[g + 1]);
}

// Accepted candidates of source s before each of its bit words (bits of
// other sources masked off), and their total.
__global__ __launch_bounds__(kCommitThreads) void src_rank_kernel(CommitArgs a, uint32_t s)
{
    __shared__ int64_t sh[kCommitThreads / kWave];
    if (s >= *a.nsrc)
        return;
    const uint32_t cs = a.start[s], ce = a.start[s + 1];
    if (cs == ce) {
        if (threadIdx.x == 0)
            a.acc_of[s] = 0;
        return;
    }
    const uint32_t w0 = cs >> 5, w1 = ((ce - 1) >> 5) + 1, nw = w1 - w0;
    auto word = [&](uint32_t w) -> uint32_t {
        uint32_t v = a.gbits[w];
        if (w == w0)
            v &= ~0u << (cs & 31);
        if (w == w1 - 1 && (ce & 31))
            v &= (1u << (ce & 31)) - 1;
        return v;
    };
    const uint64_t per = ((uint64_t)nw + kCommitThreads - 1) / kCommitThreads;
    const uint32_t a0 = w0 + (uint32_t)std::min<uint64_t>(nw, threadIdx.x * per);
    const uint32_t a1 = w0 + (uint32_t)std::min<uint64_t>(nw, (threadIdx.x + 1) * per);
    int64_t cnt = 0;
    for (uint32_t w = a0; w < a1; w++)
        cnt += __popc(word(w));
    int64_t A;
    uint32_t run = (uint32_t)block_excl_scan_i64<kCommitThreads>(cnt, sh, A);
    for (uint32_t w = a0; w < a1; w++) {
        a.wpre_src[w] = run;
        run += __popc(word(w));
    }
    if (threadIdx.x == 0)
        a.acc_of[s] = (uint32_t)A;
}

// Acceptance rank of every candidate of source s (kNoKey if not accepted),
// and as the key of its queue record.
__global__ void src_mark_kernel(CommitArgs a, uint32_t s)
{
    if (s >= *a.nsrc)
        return;
    const uint32_t cs = a.start[s], ce = a.start[s + 1];
    for (uint64_t t = cs + blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < ce;
         t += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t w = (uint32_t)(t >> 5), m = 1u << (t & 31);
        uint32_t v = a.gbits[w];
        if (w == (cs >> 5))
            v &= ~0u << (cs & 31);
        uint32_t rk = kNoKey;
        if (v & m) {
            rk = a.wpre_src[w] + __popc(v & (m - 1));
            a.qkey[a.cand_q[t]] = rk;
        }
        a.arank[t] = rk;
    }
}

// Stop point of source s (smallest k after which its queue meets the SLO,
// all accepted if none) and its place in the migration list.
__global__ __launch_bounds__(kCommitThreads) void src_stop_kernel(CommitArgs a, uint32_t s)
{
    __shared__ int64_t sh[kCommitThreads / kWave];
    if (s >= *a.nsrc)
        return;
    const uint32_t i = a.src[s];
    const uint32_t A = a.acc_of[s];
    uint32_t kstar = 0;
    if (A > 0) {
        const int64_t qlo = a.qoff[i], qhi = a.qoff[i + 1];
        const int64_t w0q = a.base_work[i];
        const uint64_t Lq = (uint64_t)(qhi - qlo);
        TtftK tks = a.tk;
        tks.slo = a.slo_of[i];
        uint32_t lo = 1, hi = A;
        if (Lq <= (uint64_t)kCommitThreads * kQueueRegs) {
            lo = regs_bisect(a.unc_here, a.qkey, qlo, Lq, w0q, hi, tks, sh);
        } else if (queue_violates_chunked(a, tks, qlo, qhi, w0q, hi, sh)) {
            lo = hi;
        } else {
            while (lo < hi) {
                const uint32_t mid = lo + (hi - lo) / 2;
                if (!queue_violates_chunked(a, tks, qlo, qhi, w0q, mid, sh))
                    hi = mid;
                else
                    lo = mid + 1;
            }
        }
        kstar = lo;
    }
    if (threadIdx.x == 0) {
        const unsigned long long base = *a.run;
        a.kstar_of[s] = kstar;
        a.base_of[s] = base;
        *a.run = base + kstar;
    }
}

// The first k* accepted records of source s move: one wave per segment
// adds its moved records' uncached tokens to its target (segments of a
// source have distinct targets) and takes theirs on the source away.
__global__ __launch_bounds__(256) void src_commit_kernel(CommitArgs a, uint32_t s)
{
    if (s >= *a.nsrc)
        return;
    const uint32_t i = a.src[s], kstar = a.kstar_of[s];
    const uint64_t wv = blockIdx.x * (uint64_t)(blockDim.x >> 6) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t nwv = (uint64_t)gridDim.x * (blockDim.x >> 6);
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t G0 = a.sseg[s], G1 = a.sseg[s + 1];
    for (uint64_t g = G0 + wv; g < G1; g += nwv) {
        const uint32_t P0 = a.seg_pos[g], P1 = a.seg_pos[g + 1];
        uint64_t to = 0, from = 0;
        for (uint64_t v = P0 + lane; v < P1; v += kWave) {
            const uint32_t t = a.grp[v];
            if (a.arank[t] < kstar) {
                to += a.g_unc[v];
                from += a.c_uh[t];
            }
        }
        to = wave_incl_sum_u64(to, (int)lane);
        from = wave_incl_sum_u64(from, (int)lane);
        to = readlane_u64(to, kWave - 1);
        from = readlane_u64(from, kWave - 1);
        if (lane == 0 && P0 < P1) {
            const uint32_t j = a.g_alt[P0];
            a.loads[j] += (int64_t)to;
            if (from)
                atomicAdd((unsigned long long*)&a.loads[i], (unsigned long long)(-(int64_t)from));
        }
    }
}

__global__ void src_finish_kernel(CommitArgs a)
{
    const unsigned long long n = *a.run;
    *a.out_count = n;
    if (n > a.cap)
        atomicOr(a.status, kErrFull);
}

// Migration list: candidate t of source rank r moves iff its acceptance rank
// is below kstar_of[r]; it lands at base_of[r] + rank (rank order within a
// source, sources in rank order).
__global__ void emit_kernel(uint64_t C, const uint32_t* __restrict__ start,
                            const uint32_t* __restrict__ nsrc_p, const uint32_t* __restrict__ src,
                            const uint32_t* __restrict__ arank,
                            const uint32_t* __restrict__ kstar_of,
                            const uint64_t* __restrict__ base_of, const uint64_t* __restrict__ c_rec,
                            const uint32_t* __restrict__ c_alt, const int64_t* __restrict__ c_ben,
                            const int64_t* __restrict__ tto, uint64_t cap,
                            uint64_t* __restrict__ out_rec, uint32_t* __restrict__ out_from,
                            uint32_t* __restrict__ out_to, int64_t* __restrict__ out_benefit,
                            int64_t* __restrict__ out_ttft)
{
    const uint32_t nsrc = *nsrc_p;
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < C;
         t += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t rk = arank[t];
        if (rk == kNoKey)
            continue;
        // source rank: the last r with start[r] <= t
        uint32_t lo = 0, hi = nsrc;  // start[lo] <= t < start[hi]
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) / 2;
            if (start[mid] <= t)
                lo = mid;
            else
                hi = mid;
        }
        if (rk >= kstar_of[lo])
            continue;
        const uint64_t idx = base_of[lo] + rk;
        if (idx < cap) {
            out_rec[idx] = c_rec[t];
            out_from[idx] = src[lo];
            out_to[idx] = c_alt[t];
            out_benefit[idx] = c_ben[t];
            out_ttft[idx] = tto[t];
        }
    }
}

template <typename T>
T* carve(uint8_t*& p, uint64_t n)
{
    T* r = reinterpret_cast<T*>(p);
    p += ((n * sizeof(T) + 255) / 256) * 256;
    return r;
}

}  // namespace

hipError_t rebalance(dm_ctx* c, const dm_queues* q, int64_t* loads_out, const dm_migrations* out,
                     uint64_t cap, uint64_t Q)
{
    const uint32_t S = c->cfg.max_slots;
    const TtftK tk{c->cfg.ttft_base_us, c->cfg.ttft_per_token_us, c->shift_div, c->cfg.slo_us};
    hipStream_t st = c->stream;
    hipError_t e;
    // per-instance arrays
    // per instance slot: L0, delay, slo_of, base_of 8 B; over 1 B; rank,
    // src, start, sseg, kstar_of, acc_of 4 B; slice sums and maxima
    // 2 x 8 x kQSplit B -- 313 B, and 16 carves of at most 256 B padding
    uint8_t* pi = static_cast<uint8_t*>(
        scratch_get(c, kSlotSelect, 320 * ((uint64_t)S + 64) + 8192, &e));
    if (!pi)
        return e;
    int64_t* L0 = carve<int64_t>(pi, S);
    int64_t* delay = carve<int64_t>(pi, S);
    int64_t* slo_of = carve<int64_t>(pi, S);
    uint32_t* acc_of = carve<uint32_t>(pi, S);
    unsigned long long* run = carve<unsigned long long>(pi, 1);
    uint8_t* over = carve<uint8_t>(pi, S);
    uint32_t* rank = carve<uint32_t>(pi, S);
    uint32_t* src = carve<uint32_t>(pi, S);
    uint32_t* start = carve<uint32_t>(pi, S + 1);
    uint32_t* sseg = carve<uint32_t>(pi, S + 1);
    uint32_t* kstar_of = carve<uint32_t>(pi, S);
    uint64_t* base_of = carve<uint64_t>(pi, S);
    int64_t* slice_sum = carve<int64_t>(pi, (uint64_t)S * kQSplit);
    int64_t* slice_max = carve<int64_t>(pi, (uint64_t)S * kQSplit);
    uint32_t* nsrc = carve<uint32_t>(pi, 1);
    uint64_t* ctot = carve<uint64_t>(pi, 2);  // candidate count, largest eligible benefit
    // per-record arrays
    const uint64_t Qa = Q ? Q : 1;
    uint8_t* pr = static_cast<uint8_t*>(scratch_get(c, kSlotProbe, Qa * 48 + 8 * 256, &e));
    if (!pr)
        return e;
    int64_t* T = carve<int64_t>(pr, Qa);
    uint32_t* owner = carve<uint32_t>(pr, Qa);
    int64_t* benefit = carve<int64_t>(pr, Qa);
    uint64_t* elig = carve<uint64_t>(pr, Qa);
    uint64_t* pos = carve<uint64_t>(pr, Qa);
    uint32_t* qkey = carve<uint32_t>(pr, Qa);

    zero_u32_kernel<<<1, 64, 0, st>>>(nsrc, 1);
    zero_u32_kernel<<<1, 64, 0, st>>>(reinterpret_cast<uint32_t*>(ctot), 4);
    fill_u32_kernel<<<grid_for(Qa, 256), 256, 0, st>>>(owner, Qa, 0xFFFFFFFFu);
    queue_sum_kernel<<<S * kQSplit, kQThreads, 0, st>>>(q->qoff, Q, q->unc_here, slice_sum,
                                                        c->d_status);
    queue_ttft_kernel<<<S * kQSplit, kQThreads, 0, st>>>(q->qoff, Q, q->unc_here, q->alt,
                                                         q->base_work, slice_sum, S, tk, T, owner,
                                                         slice_max, c->d_status);
    queue_over_kernel<<<(S + 255) / 256, 256, 0, st>>>(q->qoff, Q, q->base_work, slice_sum,
                                                        slice_max, S, tk.slo, q->prefill_interval,
                                                        q->decode_threshold_us, L0, over, delay,
                                                        slo_of, c->d_status);
    if (Q)
        // grid-stride: 256 workgroups, one atomic maximum each
        benefit_kernel<<<grid_for(Q, 256, 256), 256, 0, st>>>(Q, T, owner, q->alt, q->unc_alt, L0,
                                                              over, delay, S, tk, benefit, elig,
                                                              ctot + 1);
    rank_kernel<<<(S + 255) / 256, 256, 0, st>>>(L0, over, S, rank, src, nsrc);
    uint64_t hw[2] = {0, 0};  // candidate count, largest eligible benefit
    uint32_t nsrc_h = 0;      // overloaded sources
    if (Q) {
        e = exclusive_scan_u64(c, elig, Q, pos, ctot);
        if (e != hipSuccess)
            return e;
        e = hipMemcpyAsync(hw, ctot, sizeof(hw), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess)
            e = hipMemcpyAsync(&nsrc_h, nsrc, sizeof(nsrc_h), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess)
            e = hipStreamSynchronize(st);
        if (e != hipSuccess)
            return e;
    }
    const uint64_t C = hw[0];
    // per-candidate arrays
    const uint64_t Ca = C ? C : 1;
    uint8_t* pc = static_cast<uint8_t*>(scratch_get(c, kSlotRebalance, Ca * 64 + 16 * 256, &e));
    // per candidate: keys, ktmp 8 B; vals, vtmp, grp, g_alt, g_unc, seg_pos,
    // c_ua, c_uh, arank 4 B; tto 8 B; three bit-word arrays 1/8 B -- 60.4 B
    // and 15 carves of at most 256 B padding each
    if (!pc)
        return e;
    uint64_t* keys = carve<uint64_t>(pc, Ca);
    uint64_t* ktmp = carve<uint64_t>(pc, Ca);
    uint32_t* vals = carve<uint32_t>(pc, Ca);
    uint32_t* vtmp = carve<uint32_t>(pc, Ca);
    uint32_t* grp = carve<uint32_t>(pc, Ca);
    uint32_t* g_alt = carve<uint32_t>(pc, Ca);
    uint32_t* g_unc = carve<uint32_t>(pc, Ca);
    uint32_t* gbits = carve<uint32_t>(pc, Ca / 32 + 1);
    uint32_t* gwpre = carve<uint32_t>(pc, Ca / 32 + 1);
    uint32_t* wpre_src = carve<uint32_t>(pc, Ca / 32 + 2);
    int64_t* tto = carve<int64_t>(pc, Ca);
    uint32_t* seg_pos = carve<uint32_t>(pc, Ca + 1);
    uint32_t* c_ua = carve<uint32_t>(pc, Ca);
    uint32_t* c_uh = carve<uint32_t>(pc, Ca);
    uint32_t* arank = carve<uint32_t>(pc, Ca);
    uint32_t* cand_q = vals;  // the candidate order lands in vals

    if (C) {
        const uint32_t gc = grid_for(C, 256);
        compact_kernel<<<grid_for(Q, 256), 256, 0, st>>>(Q, elig, pos, vals);
        // candidate order (source rank, benefit desc), stable over record order
        // so equal benefits keep queue order; grouped order (source rank,
        // target), stable over candidate order.  Keys take only the bits the
        // ranks, targets and largest benefit need.
        const int rb = std::max(1, bit_length(S - 1));
        const int nb = bit_length(hw[1]);
        if (rb + nb <= 64) {
            rekey_kernel<<<gc, 256, 0, st>>>(C, kByRankBenefit, (uint32_t)nb, vals, nullptr, benefit,
                                             owner, rank, q->alt, keys);
            e = radix_sort_kv(c, keys, vals, ktmp, vtmp, C, rb + nb);
            if (e != hipSuccess) return e;
        } else {
            rekey_kernel<<<gc, 256, 0, st>>>(C, kByBenefitDesc, 0, vals, nullptr, benefit, owner,
                                             rank, q->alt, keys);
            e = radix_sort_kv(c, keys, vals, ktmp, vtmp, C, 64);
            if (e != hipSuccess) return e;
            rekey_kernel<<<gc, 256, 0, st>>>(C, kBySourceRank, 0, vals, nullptr, benefit, owner,
                                             rank, q->alt, keys);
            e = radix_sort_kv(c, keys, vals, ktmp, vtmp, C, rb);
            if (e != hipSuccess) return e;
        }
        iota_kernel<<<gc, 256, 0, st>>>(C, grp);
        rekey_kernel<<<gc, 256, 0, st>>>(C, kByRankTarget, (uint32_t)rb, grp, cand_q, benefit,
                                         owner, rank, q->alt, ktmp);
        // sort (ktmp, grp) using (keys, vtmp) as work arrays: keys is free once cand_q is final
        e = radix_sort_kv(c, ktmp, grp, keys, vtmp, C, 2 * rb);
        if (e != hipSuccess) return e;
        gather_groups_kernel<<<gc, 256, 0, st>>>(C, grp, cand_q, q->alt, q->unc_alt, g_alt, g_unc);
    }
    bounds_kernel<<<grid_for(C + 1, 256), 256, 0, st>>>(C, cand_q, owner, rank, nsrc, start);
    // (source, target) segments of the grouped order; keys and ktmp are free
    uint64_t* head = ktmp;
    uint64_t* sid = keys;
    if (C) {
        seg_head_kernel<<<grid_for(C, 256), 256, 0, st>>>(C, grp, cand_q, owner, rank, g_alt, head);
        e = exclusive_scan_u64(c, head, C, sid, ctot);
        if (e != hipSuccess)
            return e;
    }
    seg_pos_kernel<<<grid_for(std::max<uint64_t>(C, S) + 1, 256), 256, 0, st>>>(
        C, S, head, sid, ctot, start, nsrc, seg_pos, sseg);
    // the commit's record fields in candidate order (head and sid are spent)
    uint64_t* c_rec = ktmp;
    int64_t* c_ben = reinterpret_cast<int64_t*>(keys);
    uint32_t* c_alt = vtmp;
    if (C)
        gather_cand_kernel<<<grid_for(C, 256), 256, 0, st>>>(C, cand_q, q->rec_id, q->alt,
                                                            q->unc_alt, q->unc_here, benefit,
                                                            c_rec, c_alt, c_ua, c_uh, c_ben);
    copy_i64_kernel<<<grid_for(S, 256), 256, 0, st>>>(L0, loads_out, S);
    CommitArgs a;
    a.qoff = q->qoff;
    a.rec_id = q->rec_id;
    a.unc_here = q->unc_here;
    a.alt = q->alt;
    a.unc_alt = q->unc_alt;
    a.base_work = q->base_work;
    a.benefit = benefit;
    a.src = src;
    a.nsrc = nsrc;
    a.start = start;
    a.sseg = sseg;
    a.seg_pos = seg_pos;
    a.cand_q = cand_q;
    a.c_rec = c_rec;
    a.c_alt = c_alt;
    a.c_ua = c_ua;
    a.c_uh = c_uh;
    a.c_ben = c_ben;
    a.grp = grp;
    a.g_alt = g_alt;
    a.g_unc = g_unc;
    a.gbits = gbits;
    a.gwpre = gwpre;
    a.tto = tto;
    a.arank = arank;
    a.kstar_of = kstar_of;
    a.base_of = base_of;
    a.qkey = qkey;
    a.loads = loads_out;
    a.delay = delay;
    a.slo_of = slo_of;
    a.wpre_src = wpre_src;
    a.acc_of = acc_of;
    a.run = run;
    a.S = S;
    a.tk = tk;
    a.cap = cap;
    a.out_rec = out->rec_id;
    a.out_from = out->from;
    a.out_to = out->to;
    a.out_benefit = out->benefit_us;
    a.out_ttft = out->ttft_to_us;
    a.out_count = out->count;
    a.status = c->d_status;
    if (nsrc_h <= kSpreadSources) {
        // few sources: each source's phases as kernels over the whole GPU
        zero_u32_kernel<<<1, 64, 0, st>>>(reinterpret_cast<uint32_t*>(run), 2);
        zero_u32_kernel<<<grid_for(Ca / 32 + 1, 256, 1024), 256, 0, st>>>(gbits,
                                                                       (uint32_t)(Ca / 32 + 1));
        const uint32_t gw = (uint32_t)std::min<uint64_t>((S + 3) / 4, 1024);
        const uint32_t gm = grid_for(C, 256, 512);
        for (uint32_t sr = 0; sr < nsrc_h; sr++) {
            src_walk_kernel<<<gw, 256, 0, st>>>(a, sr);
            src_rank_kernel<<<1, kCommitThreads, 0, st>>>(a, sr);
            src_mark_kernel<<<gm, 256, 0, st>>>(a, sr);
            src_stop_kernel<<<1, kCommitThreads, 0, st>>>(a, sr);
            src_commit_kernel<<<gw, 256, 0, st>>>(a, sr);
        }
        src_finish_kernel<<<1, 1, 0, st>>>(a);
    } else {
        commit_kernel<<<1, kCommitThreads, 0, st>>>(a);
    }
    if (C)
        emit_kernel<<<grid_for(C, 256), 256, 0, st>>>(
            C, start, nsrc, src, arank, kstar_of, base_of, c_rec, c_alt, c_ben, tto, cap,
            out->rec_id, out->from, out->to, out->benefit_us, out->ttft_to_us);
    return hipGetLastError();
}

}  // namespace dm
