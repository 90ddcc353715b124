// dm_rebalance: one non-recursive, single-round hotspot migration pass
// (Sec. 3.3, Eq. of the migration benefit; Sec. A.1.2).
//
// Pass-start state in parallel:
//   queue scan    per instance: each record's TTFT behind the base work and
//                 the records ahead of it; load; max TTFT; overloaded flag;
//   benefit       per record: B = TTFT here - TTFT on the alternative;
//                 eligible if B > 0, source overloaded, target not;
//   source ranks  overloaded instances by (load desc, id asc);
//   ordering      eligible records sorted by (source rank, B desc,
//                 queue position asc) with stable radix passes, and a second
//                 order grouping each source's records by target.
// Then the sources are committed one after another by one workgroup.  For a
// source, the sequential rule "stop once the queue meets the SLO; move a
// record iff its TTFT on the target with the target's current load is below
// the SLO" is evaluated exactly as:
//   (i)  acceptance ignoring the stop: a record's acceptance depends only on
//        its target's load, so each target's records are walked in order by
//        one thread, all targets at once;
//   (ii) the stop only truncates that acceptance sequence and removing
//        records never raises a queued TTFT, so the number k of accepted
//        records that move is the smallest k after which the queue meets the
//        SLO -- found by bisection over parallel queue evaluations;
//   (iii) the first k accepted records move; target loads grow, the source's
//        shrinks.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kQThreads = 256;
constexpr int kCommitThreads = 1024;
constexpr uint32_t kNoKey = 0xFFFFFFFFu;

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

// Per instance (one workgroup each): record TTFTs, load, max TTFT.
__global__ __launch_bounds__(kQThreads) void queue_kernel(
    const int64_t* __restrict__ qoff, uint64_t Q, const uint32_t* __restrict__ unc_here,
    const uint32_t* __restrict__ alt, const int64_t* __restrict__ base_work, uint32_t S, TtftK tk,
    int64_t* __restrict__ T, uint32_t* __restrict__ owner, int64_t* __restrict__ L0,
    uint8_t* __restrict__ over, uint32_t* __restrict__ status)
{
    __shared__ int64_t sh[kQThreads / kWave];
    const uint32_t i = blockIdx.x;
    const int64_t lo = qoff[i], hi = qoff[i + 1];
    if (lo < 0 || hi < lo || hi > (int64_t)Q) {
        if (threadIdx.x == 0) {
            atomicOr(status, kErrInval);
            L0[i] = base_work[i];
            over[i] = 0;
        }
        return;
    }
    int64_t run = base_work[i], mx = INT64_MIN;
    for (int64_t b = lo; b < hi; b += kQThreads) {
        const int64_t q = b + threadIdx.x;
        const bool ok = q < hi;
        const int64_t u = ok ? (int64_t)unc_here[q] : 0;
        int64_t tot;
        const int64_t ex = block_excl_scan_i64<kQThreads>(u, sh, tot);
        if (ok) {
            const int64_t t = tk(u, run + ex);
            T[q] = t;
            owner[q] = i;
            mx = std::max(mx, t);
            if (alt[q] >= S)
                atomicOr(status, kErrInval);
        }
        run += tot;
    }
    mx = block_max_i64<kQThreads>(mx, sh);
    if (threadIdx.x == 0) {
        L0[i] = run;
        over[i] = (hi > lo && mx > tk.slo) ? 1 : 0;
    }
}

__global__ void benefit_kernel(uint64_t Q, const int64_t* __restrict__ T,
                               const uint32_t* __restrict__ owner, const uint32_t* __restrict__ alt,
                               const uint32_t* __restrict__ unc_alt, const int64_t* __restrict__ L0,
                               const uint8_t* __restrict__ over, uint32_t S, TtftK tk,
                               int64_t* __restrict__ benefit, uint64_t* __restrict__ elig)
{
    for (uint64_t q = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; q < Q;
         q += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t i = owner[q], j = alt[q];
        bool e = false;
        int64_t b = 0;
        if (i < S && j < S && over[i]) {
            b = T[q] - tk((int64_t)unc_alt[q], L0[j]);
            e = b > 0 && !over[j];
        }
        benefit[q] = b;
        elig[q] = e ? 1 : 0;
    }
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

// Eligible records in queue order -> (key = queue position, value = record).
__global__ void compact_kernel(uint64_t Q, const uint64_t* __restrict__ elig,
                               const uint64_t* __restrict__ pos, const uint32_t* __restrict__ owner,
                               const int64_t* __restrict__ qoff, uint64_t* __restrict__ keys,
                               uint32_t* __restrict__ vals)
{
    for (uint64_t q = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; q < Q;
         q += (uint64_t)gridDim.x * blockDim.x)
        if (elig[q]) {
            keys[pos[q]] = (uint64_t)((int64_t)q - qoff[owner[q]]);
            vals[pos[q]] = (uint32_t)q;
        }
}

// keys[t] = a key of the record (or candidate index) held in vals[t].
enum KeyKind { kByBenefitDesc, kBySourceRank, kByTarget, kByRankOfCand };

__global__ void rekey_kernel(uint64_t C, int kind, const uint32_t* __restrict__ vals,
                             const uint32_t* __restrict__ cand_q, const int64_t* __restrict__ benefit,
                             const uint32_t* __restrict__ owner, const uint32_t* __restrict__ rank,
                             const uint32_t* __restrict__ alt, uint64_t* __restrict__ keys)
{
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < C;
         t += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t v = vals[t];
        uint64_t k = 0;
        switch (kind) {
            case kByBenefitDesc: k = ~(uint64_t)benefit[v]; break;
            case kBySourceRank: k = rank[owner[v]]; break;
            case kByTarget: k = alt[cand_q[v]]; break;
            case kByRankOfCand: k = rank[owner[cand_q[v]]]; break;
        }
        keys[t] = k;
    }
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
    const uint32_t* cand_q;   // [C] record of candidate t
    const uint32_t* grp;      // [C] candidate order grouped by (rank, target)
    const uint32_t* g_alt;    // [C] target of grp[u]
    const uint32_t* g_unc;    // [C] unc_alt of grp[u]
    uint8_t* acc;             // [C]
    uint32_t* arank;          // [C]
    int64_t* tto;             // [C]
    uint32_t* qkey;           // [Q]
    int64_t* loads;           // [S] live loads (starts as pass-start loads)
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

// Largest TTFT over the records of queue [lo, hi) whose key is >= k
// (the records still queued after the first k accepted ones left).
__device__ int64_t queue_max_after(const CommitArgs& a, int64_t lo, int64_t hi, int64_t w0,
                                   uint32_t k, int64_t* sh)
{
    int64_t run = w0, mx = INT64_MIN;
    for (int64_t b = lo; b < hi; b += kCommitThreads) {
        const int64_t q = b + threadIdx.x;
        const bool keep = q < hi && a.qkey[q] >= k;
        const int64_t u = keep ? (int64_t)a.unc_here[q] : 0;
        int64_t tot;
        const int64_t ex = block_excl_scan_i64<kCommitThreads>(u, sh, tot);
        if (keep)
            mx = std::max(mx, a.tk(u, run + ex));
        run += tot;
    }
    return block_max_i64<kCommitThreads>(mx, sh);
}

__global__ __launch_bounds__(kCommitThreads) void commit_kernel(CommitArgs a)
{
    __shared__ int64_t sh[kCommitThreads / kWave];
    __shared__ uint64_t s_count;
    const uint32_t nsrc = *a.nsrc;
    if (threadIdx.x == 0)
        s_count = 0;
    __syncthreads();
    for (uint32_t s = 0; s < nsrc; s++) {
        const uint32_t i = a.src[s];
        const uint32_t cs = a.start[s], ce = a.start[s + 1];
        const int64_t qlo = a.qoff[i], qhi = a.qoff[i + 1];
        // (i) acceptance, one thread per target segment
        for (uint32_t u = cs + threadIdx.x; u < ce; u += kCommitThreads) {
            if (u != cs && a.g_alt[u] == a.g_alt[u - 1])
                continue;
            const uint32_t j = a.g_alt[u];
            // loads are updated with atomics at L2: read them past the L1
            int64_t Lt = __hip_atomic_load(&a.loads[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (uint32_t v = u; v < ce && a.g_alt[v] == j; v++) {
                const int64_t tj = a.tk((int64_t)a.g_unc[v], Lt);
                const bool ok = tj < a.tk.slo;
                const uint32_t t = a.grp[v];
                a.acc[t] = ok;
                a.tto[t] = tj;
                if (ok)
                    Lt += a.g_unc[v];
            }
        }
        __syncthreads();
        // (ii) acceptance ranks in candidate order; mark queue records
        for (int64_t q = qlo + threadIdx.x; q < qhi; q += kCommitThreads)
            a.qkey[q] = kNoKey;
        int64_t A = 0;
        for (uint32_t b = cs; b < ce; b += kCommitThreads) {
            const uint32_t t = b + threadIdx.x;
            const int64_t v = (t < ce && a.acc[t]) ? 1 : 0;
            int64_t tot;
            const int64_t ex = block_excl_scan_i64<kCommitThreads>(v, sh, tot);
            if (t < ce)
                a.arank[t] = (uint32_t)(A + ex);
            A += tot;
        }
        __syncthreads();
        for (uint32_t t = cs + threadIdx.x; t < ce; t += kCommitThreads)
            if (a.acc[t])
                a.qkey[a.cand_q[t]] = a.arank[t];
        __syncthreads();
        uint32_t kstar = 0;
        if (A > 0) {
            const int64_t w0 = a.base_work[i];
            if (queue_max_after(a, qlo, qhi, w0, (uint32_t)A, sh) > a.tk.slo) {
                kstar = (uint32_t)A;
            } else {
                uint32_t lo = 1, hi = (uint32_t)A;  // answer in [lo, hi]
                while (lo < hi) {
                    const uint32_t mid = lo + (hi - lo) / 2;
                    if (queue_max_after(a, qlo, qhi, w0, mid, sh) <= a.tk.slo)
                        hi = mid;
                    else
                        lo = mid + 1;
                }
                kstar = lo;
            }
        }
        // (iii) commit the first kstar accepted records
        const uint64_t base = s_count;
        for (uint32_t t = cs + threadIdx.x; t < ce; t += kCommitThreads) {
            if (!a.acc[t] || a.arank[t] >= kstar)
                continue;
            const uint32_t q = a.cand_q[t];
            const uint64_t idx = base + a.arank[t];
            if (idx < a.cap) {
                a.out_rec[idx] = a.rec_id[q];
                a.out_from[idx] = i;
                a.out_to[idx] = a.alt[q];
                a.out_benefit[idx] = a.benefit[q];
                a.out_ttft[idx] = a.tto[t];
            }
            atomicAdd((unsigned long long*)&a.loads[a.alt[q]], (unsigned long long)a.unc_alt[q]);
            atomicAdd((unsigned long long*)&a.loads[i],
                      (unsigned long long)(-(int64_t)a.unc_here[q]));
        }
        __syncthreads();
        if (threadIdx.x == 0)
            s_count = base + kstar;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *a.out_count = s_count;
        if (s_count > a.cap)
            atomicOr(a.status, kErrFull);
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
    uint8_t* pi = static_cast<uint8_t*>(scratch_get(c, 3, 64 * (S + 64) + 4096, &e));
    if (!pi)
        return e;
    int64_t* L0 = carve<int64_t>(pi, S);
    uint8_t* over = carve<uint8_t>(pi, S);
    uint32_t* rank = carve<uint32_t>(pi, S);
    uint32_t* src = carve<uint32_t>(pi, S);
    uint32_t* start = carve<uint32_t>(pi, S + 1);
    uint32_t* nsrc = carve<uint32_t>(pi, 1);
    uint64_t* ctot = carve<uint64_t>(pi, 1);
    // per-record arrays
    const uint64_t Qa = Q ? Q : 1;
    uint8_t* pr = static_cast<uint8_t*>(scratch_get(c, 1, Qa * 48 + 8 * 256, &e));
    if (!pr)
        return e;
    int64_t* T = carve<int64_t>(pr, Qa);
    uint32_t* owner = carve<uint32_t>(pr, Qa);
    int64_t* benefit = carve<int64_t>(pr, Qa);
    uint64_t* elig = carve<uint64_t>(pr, Qa);
    uint64_t* pos = carve<uint64_t>(pr, Qa);
    uint32_t* qkey = carve<uint32_t>(pr, Qa);

    zero_u32_kernel<<<1, 64, 0, st>>>(nsrc, 1);
    fill_u32_kernel<<<grid_for(Qa, 256), 256, 0, st>>>(owner, Qa, 0xFFFFFFFFu);
    queue_kernel<<<S, kQThreads, 0, st>>>(q->qoff, Q, q->unc_here, q->alt, q->base_work, S, tk, T,
                                          owner, L0, over, c->d_status);
    if (Q)
        benefit_kernel<<<grid_for(Q, 256), 256, 0, st>>>(Q, T, owner, q->alt, q->unc_alt, L0, over,
                                                         S, tk, benefit, elig);
    rank_kernel<<<(S + 255) / 256, 256, 0, st>>>(L0, over, S, rank, src, nsrc);
    uint64_t C = 0;
    if (Q) {
        e = exclusive_scan_u64(c, elig, Q, pos, ctot);
        if (e != hipSuccess)
            return e;
        e = hipMemcpyAsync(&C, ctot, sizeof(uint64_t), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess)
            e = hipStreamSynchronize(st);
        if (e != hipSuccess)
            return e;
    }
    // per-candidate arrays
    const uint64_t Ca = C ? C : 1;
    uint8_t* pc = static_cast<uint8_t*>(scratch_get(c, 2, Ca * 64 + 16 * 256, &e));
    if (!pc)
        return e;
    uint64_t* keys = carve<uint64_t>(pc, Ca);
    uint64_t* ktmp = carve<uint64_t>(pc, Ca);
    uint32_t* vals = carve<uint32_t>(pc, Ca);
    uint32_t* vtmp = carve<uint32_t>(pc, Ca);
    uint32_t* grp = carve<uint32_t>(pc, Ca);
    uint32_t* g_alt = carve<uint32_t>(pc, Ca);
    uint32_t* g_unc = carve<uint32_t>(pc, Ca);
    uint8_t* acc = carve<uint8_t>(pc, Ca);
    uint32_t* arank = carve<uint32_t>(pc, Ca);
    int64_t* tto = carve<int64_t>(pc, Ca);
    uint32_t* cand_q = vals;  // the candidate order lands in vals

    if (C) {
        const uint32_t gc = grid_for(C, 256);
        compact_kernel<<<grid_for(Q, 256), 256, 0, st>>>(Q, elig, pos, owner, q->qoff, keys, vals);
        // order: queue position asc, then benefit desc, then source rank asc (stable passes)
        e = radix_sort_kv(c, keys, vals, ktmp, vtmp, C, 32);
        if (e != hipSuccess) return e;
        rekey_kernel<<<gc, 256, 0, st>>>(C, kByBenefitDesc, vals, nullptr, benefit, owner, rank,
                                         q->alt, keys);
        e = radix_sort_kv(c, keys, vals, ktmp, vtmp, C, 64);
        if (e != hipSuccess) return e;
        rekey_kernel<<<gc, 256, 0, st>>>(C, kBySourceRank, vals, nullptr, benefit, owner, rank,
                                         q->alt, keys);
        e = radix_sort_kv(c, keys, vals, ktmp, vtmp, C, 16);
        if (e != hipSuccess) return e;
        // grouping: candidate indices by (source rank, target), order kept
        iota_kernel<<<gc, 256, 0, st>>>(C, grp);
        rekey_kernel<<<gc, 256, 0, st>>>(C, kByTarget, grp, cand_q, benefit, owner, rank, q->alt,
                                         ktmp);
        // sort (ktmp, grp) using (keys, vtmp) as work arrays: keys is free once cand_q is final
        e = radix_sort_kv(c, ktmp, grp, keys, vtmp, C, 16);
        if (e != hipSuccess) return e;
        rekey_kernel<<<gc, 256, 0, st>>>(C, kByRankOfCand, grp, cand_q, benefit, owner, rank,
                                         q->alt, ktmp);
        e = radix_sort_kv(c, ktmp, grp, keys, vtmp, C, 16);
        if (e != hipSuccess) return e;
        gather_groups_kernel<<<gc, 256, 0, st>>>(C, grp, cand_q, q->alt, q->unc_alt, g_alt, g_unc);
    }
    bounds_kernel<<<grid_for(C + 1, 256), 256, 0, st>>>(C, cand_q, owner, rank, nsrc, start);
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
    a.cand_q = cand_q;
    a.grp = grp;
    a.g_alt = g_alt;
    a.g_unc = g_unc;
    a.acc = acc;
    a.arank = arank;
    a.tto = tto;
    a.qkey = qkey;
    a.loads = loads_out;
    a.tk = tk;
    a.cap = cap;
    a.out_rec = out->rec_id;
    a.out_from = out->from;
    a.out_to = out->to;
    a.out_benefit = out->benefit_us;
    a.out_ttft = out->ttft_to_us;
    a.out_count = out->count;
    a.status = c->d_status;
    commit_kernel<<<1, kCommitThreads, 0, st>>>(a);
    return hipGetLastError();
}

}  // namespace dm
