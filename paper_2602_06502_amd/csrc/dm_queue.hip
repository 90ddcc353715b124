// Queued requests on the device: the serving state the rebalancing pass
// reads (Sec. 3.3).  Per instance slot a FIFO of records (request id,
// uncached tokens on it, the other candidate, uncached tokens there) in CSR
// form, and base work ahead of each queue.  Each operation reads one CSR
// and writes another:
//   append   a routed batch joins the tails of its chosen instances' queues,
//            in request order;
//   migrate  a migration list, in order: each record leaves its source
//            queue (the rest keep their order) and joins its target's tail
//            with the pair's roles swapped;
//   drain    units of service per instance: base work first, then whole
//            records from the head; a partly served head keeps the rest.
// Every record finds its queue by bisection over the offsets; order within
// a destination queue comes from exclusive scans and stable radix sorts.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

template <typename T>
T* carve(uint8_t*& p, uint64_t n)
{
    T* r = reinterpret_cast<T*>(p);
    p += ((n * sizeof(T) + 255) / 256) * 256;
    return r;
}

size_t up256q(size_t x) { return (x + 255) & ~size_t(255); }

// Queue (instance slot) of record q: the last i with qoff[i] <= q.
__device__ __forceinline__ uint32_t owner_of(const int64_t* qoff, uint32_t S, int64_t q)
{
    uint32_t lo = 0, hi = S;  // qoff[lo] <= q < qoff[hi]
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (qoff[mid] <= q)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

__global__ void q_zero_kernel(unsigned long long* __restrict__ p, uint64_t n)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// Every queue's bounds in [0, Q] and in order (bad |= 4 otherwise), and,
// when given, service and base work not negative (bad |= 1).  Everything
// that locates a record through the offsets runs after this check.
__global__ void q_check_kernel(const int64_t* __restrict__ qoff, uint32_t S, int64_t Q,
                               const int64_t* __restrict__ base, const int64_t* __restrict__ units,
                               uint32_t* __restrict__ bad)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i <= S; i += gridDim.x * blockDim.x) {
        const int64_t lo = qoff[i];
        if ((i == 0 && lo != 0) || (i == S && lo != Q) ||
            (i < S && (lo < 0 || lo > qoff[i + 1] || lo > Q)))
            atomicOr(bad, 4u);
        if (i < S && units && (units[i] < 0 || base[i] < 0))
            atomicOr(bad, 1u);
    }
}

// Per-instance counts are gathered per workgroup in LDS (dynamic shared
// memory of k * S words) and added to the device counters once per
// workgroup: a few hot instances would otherwise take every atomic.
__device__ __forceinline__ void lds_zero(uint32_t* sh, uint32_t m)
{
    for (uint32_t j = threadIdx.x; j < m; j += blockDim.x)
        sh[j] = 0;
    __syncthreads();
}

__device__ __forceinline__ void lds_flush(const uint32_t* sh, uint32_t S,
                                          unsigned long long* __restrict__ cnt)
{
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < S; j += blockDim.x)
        if (sh[j])
            atomicAdd(&cnt[j], (unsigned long long)sh[j]);
}

// Histogram of instance ids (bad |= 1 for one past the slots).
__global__ void q_hist_kernel(const uint32_t* __restrict__ id, uint64_t n, uint32_t S,
                              unsigned long long* __restrict__ cnt, uint32_t* __restrict__ bad)
{
    extern __shared__ uint32_t sh[];
    lds_zero(sh, S);
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t c = id[i];
        if (c >= S)
            atomicOr(bad, 1u);
        else
            atomicAdd(&sh[c], 1u);
    }
    lds_flush(sh, S, cnt);
}

// qoff2[i] = qoff[i] + extra_before[i] (qoff2[S] too); base copied.
__global__ void q_offsets_kernel(const int64_t* __restrict__ qoff, const uint64_t* __restrict__ ex,
                                 const uint64_t* __restrict__ ex_total, uint32_t S,
                                 const int64_t* __restrict__ base, int64_t* __restrict__ qoff2,
                                 int64_t* __restrict__ base2)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i <= S; i += gridDim.x * blockDim.x) {
        qoff2[i] = qoff[i] + (int64_t)(i < S ? ex[i] : *ex_total);
        if (i < S && base2 != base)
            base2[i] = base[i];
    }
}

struct QIn {
    const int64_t* qoff;
    const uint64_t* rec;
    const uint32_t *here, *alt, *there;
};
struct QOut {
    int64_t* qoff;
    uint64_t* rec;
    uint32_t *here, *alt, *there;
};

// Old records shift by the new records ahead of their queue.
__global__ void q_shift_kernel(QIn a, uint32_t S, int64_t Q, const uint64_t* __restrict__ ex,
                               QOut b)
{
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < Q;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t i = owner_of(a.qoff, S, q);
        const int64_t d = q + (int64_t)ex[i];
        b.rec[d] = a.rec[q];
        b.here[d] = a.here[q];
        b.alt[d] = a.alt[q];
        b.there[d] = a.there[q];
    }
}

__global__ void q_fill_kernel(int64_t* __restrict__ p, uint64_t n, int64_t v)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void q_widen_kernel(const uint32_t* __restrict__ a, uint64_t n, uint64_t* __restrict__ b)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        b[i] = a[i];
}

__global__ void q_key_kernel(const uint32_t* __restrict__ id, uint64_t n,
                             uint64_t* __restrict__ key, uint32_t* __restrict__ val)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x) {
        key[i] = id[i];
        val[i] = (uint32_t)i;
    }
}

// Batch requests in (chosen, request) order: request r goes after its
// queue's old records, at its rank among the batch's requests there.
__global__ void q_append_new_kernel(const uint32_t* __restrict__ order, uint64_t n,
                                    const int64_t* __restrict__ qoff,
                                    const int64_t* __restrict__ qoff2,
                                    const uint64_t* __restrict__ ex, const int64_t* __restrict__ off,
                                    const uint32_t* __restrict__ cand,
                                    const uint32_t* __restrict__ match,
                                    const uint32_t* __restrict__ chosen, uint32_t bshift,
                                    uint64_t rec_base, QOut b)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < n;
         p += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t r = order[p];
        const uint32_t i = chosen[r];
        const int64_t len = off[r + 1] - off[r];
        const uint32_t c1 = cand[r], c2 = cand[n + r];
        const int64_t u1 = len - ((int64_t)match[r] << bshift);
        const int64_t u2 = len - ((int64_t)match[n + r] << bshift);
        const bool first = i == c1;
        const int64_t d = qoff2[i] + (qoff[i + 1] - qoff[i]) + (int64_t)(p - ex[i]);
        b.rec[d] = rec_base + r;
        b.here[d] = (uint32_t)(first ? u1 : u2);
        b.alt[d] = first ? c2 : c1;
        b.there[d] = (uint32_t)(first ? u2 : u1);
    }
}

// Migrated record ids in an open-addressing table (value = list index).
__global__ void q_mig_table_kernel(const uint64_t* __restrict__ mrec, uint64_t m,
                                   unsigned long long* __restrict__ tk, uint32_t* __restrict__ tv,
                                   uint32_t log2, uint32_t* __restrict__ bad)
{
    const uint64_t mask = (1ull << log2) - 1;
    for (uint64_t k = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; k < m;
         k += (uint64_t)gridDim.x * blockDim.x) {
        if (mrec[k] == ~0ull) {  // its key would be the empty mark
            atomicOr(bad, 2u);
            continue;
        }
        const unsigned long long key = mrec[k] + 1;  // 0 marks an empty slot
        uint64_t h = mix64(mrec[k]) & mask;
        for (uint64_t step = 0; step <= mask; step++, h = (h + 1) & mask) {
            const unsigned long long prev = atomicCAS(&tk[h], 0ull, key);
            if (prev == 0) {
                tv[h] = (uint32_t)k;
                break;
            }
            if (prev == key) {  // a record migrated twice in one list
                atomicOr(bad, 2u);
                break;
            }
        }
    }
}

// gone[q] = 1 for migrated records (found in their source queue); at[k] =
// the queue position of list entry k.
__global__ void q_mig_find_kernel(QIn a, uint32_t S, int64_t Q,
                                  const unsigned long long* __restrict__ tk,
                                  const uint32_t* __restrict__ tv, uint32_t log2,
                                  const uint32_t* __restrict__ msrc, uint64_t* __restrict__ gone,
                                  int64_t* __restrict__ at)
{
    const uint64_t mask = (1ull << log2) - 1;
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < Q;
         q += (int64_t)gridDim.x * blockDim.x) {
        const unsigned long long key = a.rec[q] + 1;
        uint64_t h = mix64(a.rec[q]) & mask;
        uint64_t g = 0;
        for (uint64_t step = 0; step <= mask; step++, h = (h + 1) & mask) {
            const unsigned long long v = tk[h];
            if (v == 0)
                break;
            if (v == key) {
                const uint32_t k = tv[h];
                if (msrc[k] == owner_of(a.qoff, S, q)) {
                    g = 1;
                    at[k] = q;
                }
                break;
            }
        }
        gone[q] = g;
    }
}

// Per instance: records removed (counted per source) and received.
__global__ void q_mig_count_kernel(const uint32_t* __restrict__ msrc,
                                   const uint32_t* __restrict__ mdst, uint64_t m, uint32_t S,
                                   const int64_t* __restrict__ at,
                                   unsigned long long* __restrict__ delta_out,
                                   unsigned long long* __restrict__ in_cnt,
                                   uint32_t* __restrict__ bad)
{
    extern __shared__ uint32_t sh[];  // [2 S]: removed, received
    lds_zero(sh, 2 * S);
    for (uint64_t k = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; k < m;
         k += (uint64_t)gridDim.x * blockDim.x) {
        if (msrc[k] >= S || mdst[k] >= S || at[k] < 0) {
            atomicOr(bad, 1u);
            continue;
        }
        atomicAdd(&sh[msrc[k]], 1u);
        atomicAdd(&sh[S + mdst[k]], 1u);
    }
    lds_flush(sh, S, delta_out);
    for (uint32_t j = threadIdx.x; j < S; j += blockDim.x)
        if (sh[S + j])
            atomicAdd(&in_cnt[j], (unsigned long long)sh[S + j]);
}

// New queue lengths of the migration: len - removed + received; ex[i] =
// their exclusive prefix is done by a scan afterwards.
__global__ void q_mig_len_kernel(const int64_t* __restrict__ qoff, uint32_t S,
                                 const unsigned long long* __restrict__ removed,
                                 const unsigned long long* __restrict__ in_cnt,
                                 uint64_t* __restrict__ len2)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < S; i += gridDim.x * blockDim.x)
        len2[i] = (uint64_t)(qoff[i + 1] - qoff[i]) - removed[i] + in_cnt[i];
}

__global__ void q_fin_offsets_kernel(const uint64_t* __restrict__ ex,
                                     const uint64_t* __restrict__ total, uint32_t S,
                                     int64_t* __restrict__ qoff2)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i <= S; i += gridDim.x * blockDim.x)
        qoff2[i] = (int64_t)(i < S ? ex[i] : *total);
}

// Records that stay: their queue's new start plus their rank among the
// queue's records that stay (gscan: exclusive scan of gone).
__global__ void q_mig_keep_kernel(QIn a, uint32_t S, int64_t Q, const uint64_t* __restrict__ gone,
                                  const uint64_t* __restrict__ gscan, QOut b)
{
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < Q;
         q += (int64_t)gridDim.x * blockDim.x) {
        if (gone[q])
            continue;
        const uint32_t i = owner_of(a.qoff, S, q);
        const int64_t lo = a.qoff[i];
        const int64_t rank = (q - lo) - (int64_t)(gscan[q] - gscan[lo]);
        const int64_t d = b.qoff[i] + rank;
        b.rec[d] = a.rec[q];
        b.here[d] = a.here[q];
        b.alt[d] = a.alt[q];
        b.there[d] = a.there[q];
    }
}

// Migrants in (target, list) order at their target's tail, roles swapped.
__global__ void q_mig_in_kernel(QIn a, const uint32_t* __restrict__ order, uint64_t m, uint32_t S,
                                const uint32_t* __restrict__ msrc,
                                const uint32_t* __restrict__ mdst, const int64_t* __restrict__ at,
                                const uint64_t* __restrict__ in_ex,
                                const unsigned long long* __restrict__ in_cnt, QOut b)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < m;
         p += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t k = order[p];
        const uint32_t j = mdst[k];
        const int64_t q = at[k];
        const int64_t d = b.qoff[j + 1] - (int64_t)in_cnt[j] + (int64_t)(p - in_ex[j]);
        b.rec[d] = a.rec[q];
        b.here[d] = a.there[q];
        b.alt[d] = msrc[k];
        b.there[d] = a.here[q];
    }
}

// Drain: per record, whether the service left after the base work covers it
// and every record ahead of it (hs: exclusive scan of uncached tokens).
__global__ void q_drain_kernel(QIn a, uint32_t S, int64_t Q, const int64_t* __restrict__ base,
                               const int64_t* __restrict__ units, const uint64_t* __restrict__ hs,
                               uint64_t* __restrict__ popped, unsigned long long* __restrict__ npop)
{
    extern __shared__ uint32_t sh[];
    lds_zero(sh, S);
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < Q;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t i = owner_of(a.qoff, S, q);
        const int64_t left = units[i] - std::min(base[i], units[i]);
        const uint64_t upto = hs[q] - hs[a.qoff[i]] + a.here[q];  // tokens through q
        const uint64_t p = upto <= (uint64_t)left ? 1 : 0;
        popped[q] = p;
        if (p)
            atomicAdd(&sh[i], 1u);
    }
    lds_flush(sh, S, npop);
}

__global__ void q_drain_len_kernel(const int64_t* __restrict__ qoff, uint32_t S,
                                   const unsigned long long* __restrict__ npop,
                                   const int64_t* __restrict__ base,
                                   const int64_t* __restrict__ units, uint64_t* __restrict__ len2,
                                   int64_t* __restrict__ base2)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < S; i += gridDim.x * blockDim.x) {
        len2[i] = (uint64_t)(qoff[i + 1] - qoff[i]) - npop[i];
        base2[i] = base[i] - std::min(base[i], std::max<int64_t>(units[i], 0));
    }
}

// Records that stay, in order; the new head keeps what its service left.
__global__ void q_drain_keep_kernel(QIn a, uint32_t S, int64_t Q, const int64_t* __restrict__ base,
                                    const int64_t* __restrict__ units,
                                    const uint64_t* __restrict__ hs,
                                    const uint64_t* __restrict__ popped,
                                    const unsigned long long* __restrict__ npop, QOut b)
{
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < Q;
         q += (int64_t)gridDim.x * blockDim.x) {
        if (popped[q])
            continue;
        const uint32_t i = owner_of(a.qoff, S, q);
        const int64_t head = a.qoff[i] + (int64_t)npop[i];
        const int64_t d = b.qoff[i] + (q - head);
        uint32_t h = a.here[q];
        if (q == head) {
            const int64_t left = units[i] - std::min(base[i], units[i]);
            h -= (uint32_t)(left - (int64_t)(hs[q] - hs[a.qoff[i]]));
        }
        b.rec[d] = a.rec[q];
        b.here[d] = h;
        b.alt[d] = a.alt[q];
        b.there[d] = a.there[q];
    }
}

// Re-probe, checks first: every queued record's id has a chain inside the
// key array that fits its prompt (bad |= 1 otherwise).
__global__ void q_reprobe_check_kernel(QIn a, uint32_t S, int64_t Q, uint64_t n_ids,
                                       const int64_t* __restrict__ coff, uint64_t n_keys,
                                       const int64_t* __restrict__ plen, uint32_t bshift,
                                       uint32_t* __restrict__ bad)
{
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < Q;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t r = a.rec[q];
        bool ok = r < n_ids && a.alt[q] < S;
        if (ok) {
            const int64_t lo = coff[r], hi = coff[r + 1], len = plen[r];
            ok = lo >= 0 && hi >= lo && (uint64_t)hi <= n_keys && len >= 0 &&
                 len < (1ll << 32) && ((hi - lo) << bshift) <= len;
        }
        if (!ok)
            atomicOr(bad, 1u);
    }
}

// Leading blocks of chain[0, nb) cached in one table: lane l probes block
// base + l, the first miss over the wave ends the scan.  Wave-uniform.
__device__ __forceinline__ int64_t q_cached_blocks(const uint64_t* tab, uint32_t ls,
                                                   const uint64_t* chain, int64_t nb, int lane)
{
    for (int64_t b0 = 0; b0 < nb; b0 += kWave) {
        const int64_t k = b0 + lane;
        const bool miss = k < nb && !table_has(tab, ls, canon_key(chain[k]));
        const uint64_t m = ballot(miss);
        if (m)
            return b0 + __builtin_ctzll(m);
    }
    return nb;
}

// One wave per record: its uncached tokens on its instance and on its
// alternative from the caches as they are now; the rest copied.
__global__ void __launch_bounds__(256) q_reprobe_kernel(
    QIn a, uint32_t S, int64_t Q, const int64_t* __restrict__ coff,
    const uint64_t* __restrict__ keys, const int64_t* __restrict__ plen,
    const uint64_t* __restrict__ tables, uint32_t ls, uint32_t bshift, QOut b)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t q = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave; q < Q;
         q += waves) {
        const uint32_t i = owner_of(a.qoff, S, q);
        const uint64_t r = a.rec[q];
        const uint32_t j = a.alt[q];
        const int64_t lo = coff[r], nb = coff[r + 1] - lo, len = plen[r];
        const int64_t mh = q_cached_blocks(tables + ((uint64_t)i << ls), ls, keys + lo, nb, lane);
        const int64_t ma = q_cached_blocks(tables + ((uint64_t)j << ls), ls, keys + lo, nb, lane);
        if (lane == 0) {
            b.rec[q] = r;
            b.alt[q] = j;
            b.here[q] = (uint32_t)(len - (mh << bshift));
            b.there[q] = (uint32_t)(len - (ma << bshift));
        }
    }
}

__global__ void q_copy_offsets_kernel(const int64_t* __restrict__ qoff,
                                      const int64_t* __restrict__ base, uint32_t S,
                                      int64_t* __restrict__ qoff2, int64_t* __restrict__ base2)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i <= S; i += gridDim.x * blockDim.x) {
        qoff2[i] = qoff[i];
        if (i < S)
            base2[i] = base[i];
    }
}

hipError_t q_quiesce(dm_ctx* c)
{
    hipError_t e = join_selection(c);
    if (e == hipSuccess)
        e = sync_streams(c);
    return e;
}

// Record count of a queue set (its qoff[S], read from the device).
hipError_t q_count(dm_ctx* c, const int64_t* qoff, int64_t* Q)
{
    int64_t v[2] = {0, 0};
    hipError_t e = hipMemcpy(&v[0], qoff, 8, hipMemcpyDeviceToHost);
    if (e == hipSuccess)
        e = hipMemcpy(&v[1], qoff + c->cfg.max_slots, 8, hipMemcpyDeviceToHost);
    if (e == hipSuccess && (v[0] != 0 || v[1] < 0 || v[1] >= (1ll << 32)))
        e = hipErrorInvalidValue;
    *Q = v[1];
    return e;
}

}  // namespace

dm_status queue_append(dm_ctx* c, const dm_queues* q, const int64_t* offsets, uint64_t n,
                       const dm_route_out* routed, uint64_t rec_base, const dm_queue_out* out)
{
    const uint32_t S = c->cfg.max_slots;
    hipError_t e = q_quiesce(c);
    int64_t Q = 0;
    if (e == hipSuccess && (e = q_count(c, q->qoff, &Q)) == hipErrorInvalidValue)
        return fail(c, DM_EINVAL, "dm_queue_append: qoff[0] must be 0, fewer than 2^32 records");
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_queue_append");
    if ((uint64_t)Q + n > out->cap)
        return fail(c, DM_EFULL, "dm_queue_append: the output holds fewer records than the result");
    hipStream_t st = c->stream;
    const uint64_t na = n ? n : 1;
    uint8_t* w = static_cast<uint8_t*>(
        scratch_get(c, kSlotMembers, 4 * up256q(8 * (uint64_t)S) + 2 * up256q(8 * na) +
                                         2 * up256q(4 * na) + 1024, &e));
    if (!w)
        return hip_fail(c, e, "dm_queue_append");
    unsigned long long* cnt = carve<unsigned long long>(w, S);
    uint64_t* ex = carve<uint64_t>(w, S);
    uint64_t* tot = carve<uint64_t>(w, 2);
    uint32_t* bad = reinterpret_cast<uint32_t*>(tot + 1);
    uint64_t* key = carve<uint64_t>(w, na);
    uint64_t* ktmp = carve<uint64_t>(w, na);
    uint32_t* order = carve<uint32_t>(w, na);
    uint32_t* vtmp = carve<uint32_t>(w, na);
    q_zero_kernel<<<grid_for(S, 256), 256, 0, st>>>(cnt, S);
    q_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<unsigned long long*>(tot), 2);
    q_check_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(q->qoff, S, Q, nullptr, nullptr, bad);
    if (n)
        q_hist_kernel<<<grid_for(n, 256, 1024), 256, 4 * S, st>>>(routed->chosen, n, S, cnt, bad);
    uint32_t badh = 0;
    if ((e = hipMemcpyAsync(&badh, bad, 4, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_append");
    if (badh & 4)
        return fail(c, DM_EINVAL, "dm_queue_append: queue offsets out of order or range");
    if (badh)
        return fail(c, DM_EINVAL, "dm_queue_append: a chosen instance is >= max_slots");
    if ((e = exclusive_scan_u64(c, reinterpret_cast<const uint64_t*>(cnt), S, ex, tot)) !=
        hipSuccess)
        return hip_fail(c, e, "dm_queue_append");
    q_offsets_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(q->qoff, ex, tot, S, q->base_work,
                                                           out->qoff, out->base_work);
    const QIn a{q->qoff, q->rec_id, q->unc_here, q->alt, q->unc_alt};
    const QOut b{out->qoff, out->rec_id, out->unc_here, out->alt, out->unc_alt};
    if (Q)
        q_shift_kernel<<<grid_for(Q, 256, 8192), 256, 0, st>>>(a, S, Q, ex, b);
    if (n) {
        q_key_kernel<<<grid_for(n, 256, 4096), 256, 0, st>>>(routed->chosen, n, key, order);
        if ((e = radix_sort_kv(c, key, order, ktmp, vtmp, n, 16)) != hipSuccess)
            return hip_fail(c, e, "dm_queue_append");
        uint32_t bshift = 0;
        while ((1u << bshift) < c->cfg.block_size)
            bshift++;
        q_append_new_kernel<<<grid_for(n, 256, 4096), 256, 0, st>>>(
            order, n, q->qoff, out->qoff, ex, offsets, routed->cand, routed->match, routed->chosen,
            bshift, rec_base, b);
    }
    if ((e = hipGetLastError()) != hipSuccess || (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_append");
    return DM_OK;
}

dm_status queue_migrate(dm_ctx* c, const dm_queues* q, const uint64_t* mrec,
                        const uint32_t* msrc, const uint32_t* mdst, uint64_t m,
                        const dm_queue_out* out)
{
    const uint32_t S = c->cfg.max_slots;
    hipError_t e = q_quiesce(c);
    int64_t Q = 0;
    if (e == hipSuccess && (e = q_count(c, q->qoff, &Q)) == hipErrorInvalidValue)
        return fail(c, DM_EINVAL, "dm_queue_migrate: qoff[0] must be 0, fewer than 2^32 records");
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_queue_migrate");
    if ((uint64_t)Q > out->cap)
        return fail(c, DM_EFULL, "dm_queue_migrate: the output holds fewer records than the result");
    if (m > (uint64_t)Q)
        return fail(c, DM_EINVAL, "dm_queue_migrate: more migrations than queued records");
    hipStream_t st = c->stream;
    uint32_t log2 = 4;
    while ((1ull << log2) < 2 * m)
        log2++;
    const uint64_t T = 1ull << log2, Qa = Q ? Q : 1, ma = m ? m : 1;
    uint8_t* w = static_cast<uint8_t*>(scratch_get(
        c, kSlotMembers,
        4 * up256q(8 * (uint64_t)S) + up256q(8 * T) + up256q(4 * T) + 2 * up256q(8 * Qa) +
            up256q(8 * ma) + 2 * up256q(8 * ma) + 2 * up256q(4 * ma) + up256q(8 * S) + 2048,
        &e));
    if (!w)
        return hip_fail(c, e, "dm_queue_migrate");
    unsigned long long* removed = carve<unsigned long long>(w, S);
    unsigned long long* in_cnt = carve<unsigned long long>(w, S);
    uint64_t* in_ex = carve<uint64_t>(w, S);
    uint64_t* len2 = carve<uint64_t>(w, S);
    uint64_t* ex = carve<uint64_t>(w, S);
    unsigned long long* tk = carve<unsigned long long>(w, T);
    uint32_t* tv = carve<uint32_t>(w, T);
    uint64_t* gone = carve<uint64_t>(w, Qa);
    uint64_t* gscan = carve<uint64_t>(w, Qa);
    int64_t* at = carve<int64_t>(w, ma);
    uint64_t* key = carve<uint64_t>(w, ma);
    uint64_t* ktmp = carve<uint64_t>(w, ma);
    uint32_t* order = carve<uint32_t>(w, ma);
    uint32_t* vtmp = carve<uint32_t>(w, ma);
    uint64_t* tot = carve<uint64_t>(w, 4);
    uint32_t* bad = reinterpret_cast<uint32_t*>(tot + 3);
    q_zero_kernel<<<grid_for(2 * (uint64_t)S, 256), 256, 0, st>>>(removed, S);
    q_zero_kernel<<<grid_for(S, 256), 256, 0, st>>>(in_cnt, S);
    q_zero_kernel<<<grid_for(T, 256), 256, 0, st>>>(tk, T);
    q_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<unsigned long long*>(tot), 4);
    // at[k] = -1 until found
    q_fill_kernel<<<grid_for(ma, 256), 256, 0, st>>>(at, ma, -1);
    q_check_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(q->qoff, S, Q, nullptr, nullptr, bad);
    if (m)
        q_mig_table_kernel<<<grid_for(m, 256, 1024), 256, 0, st>>>(mrec, m, tk, tv, log2, bad);
    const QIn a{q->qoff, q->rec_id, q->unc_here, q->alt, q->unc_alt};
    if (Q)
        q_mig_find_kernel<<<grid_for(Q, 256, 8192), 256, 0, st>>>(a, S, Q, tk, tv, log2, msrc,
                                                                gone, at);
    if (m)
        q_mig_count_kernel<<<grid_for(m, 256, 1024), 256, 8 * S, st>>>(msrc, mdst, m, S, at, removed,
                                                                  in_cnt, bad);
    uint32_t badh = 0;
    if ((e = hipMemcpyAsync(&badh, bad, 4, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_migrate");
    if (badh & 4)
        return fail(c, DM_EINVAL, "dm_queue_migrate: queue offsets out of order or range");
    if (badh)
        return fail(c, DM_EINVAL, "dm_queue_migrate: a migration names an instance >= max_slots, "
                                  "a record not queued on its source, a record twice, or the "
                                  "record id 2^64 - 1");
    q_mig_len_kernel<<<grid_for(S, 256), 256, 0, st>>>(q->qoff, S, removed, in_cnt, len2);
    if ((e = exclusive_scan_u64(c, len2, S, ex, tot)) != hipSuccess ||
        (e = exclusive_scan_u64(c, reinterpret_cast<const uint64_t*>(in_cnt), S, in_ex,
                                tot + 1)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_migrate");
    q_fin_offsets_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(ex, tot, S, out->qoff);
    if (out->base_work != q->base_work &&
        (e = hipMemcpyAsync(out->base_work, q->base_work, 8 * (size_t)S, hipMemcpyDeviceToDevice,
                            st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_migrate");
    const QOut b{out->qoff, out->rec_id, out->unc_here, out->alt, out->unc_alt};
    if (Q) {
        if ((e = exclusive_scan_u64(c, gone, Q, gscan, tot + 2)) != hipSuccess)
            return hip_fail(c, e, "dm_queue_migrate");
        q_mig_keep_kernel<<<grid_for(Q, 256, 8192), 256, 0, st>>>(a, S, Q, gone, gscan, b);
    }
    if (m) {
        q_key_kernel<<<grid_for(m, 256, 1024), 256, 0, st>>>(mdst, m, key, order);
        if ((e = radix_sort_kv(c, key, order, ktmp, vtmp, m, 16)) != hipSuccess)
            return hip_fail(c, e, "dm_queue_migrate");
        q_mig_in_kernel<<<grid_for(m, 256, 1024), 256, 0, st>>>(a, order, m, S, msrc, mdst, at,
                                                               in_ex, in_cnt, b);
    }
    if ((e = hipGetLastError()) != hipSuccess || (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_migrate");
    return DM_OK;
}

dm_status queue_drain(dm_ctx* c, const dm_queues* q, const int64_t* units,
                      const dm_queue_out* out)
{
    const uint32_t S = c->cfg.max_slots;
    hipError_t e = q_quiesce(c);
    int64_t Q = 0;
    if (e == hipSuccess && (e = q_count(c, q->qoff, &Q)) == hipErrorInvalidValue)
        return fail(c, DM_EINVAL, "dm_queue_drain: qoff[0] must be 0, fewer than 2^32 records");
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_queue_drain");
    if ((uint64_t)Q > out->cap)
        return fail(c, DM_EFULL, "dm_queue_drain: the output holds fewer records than the result");
    hipStream_t st = c->stream;
    const uint64_t Qa = Q ? Q : 1;
    uint8_t* w = static_cast<uint8_t*>(scratch_get(
        c, kSlotMembers, 4 * up256q(8 * (uint64_t)S) + 3 * up256q(8 * Qa) + 1024, &e));
    if (!w)
        return hip_fail(c, e, "dm_queue_drain");
    unsigned long long* npop = carve<unsigned long long>(w, S);
    uint64_t* len2 = carve<uint64_t>(w, S);
    uint64_t* ex = carve<uint64_t>(w, S);
    uint64_t* here64 = carve<uint64_t>(w, Qa);
    uint64_t* hs = carve<uint64_t>(w, Qa);
    uint64_t* popped = carve<uint64_t>(w, Qa);
    uint64_t* tot = carve<uint64_t>(w, 4);
    uint32_t* bad = reinterpret_cast<uint32_t*>(tot + 3);
    q_zero_kernel<<<grid_for(S, 256), 256, 0, st>>>(npop, S);
    q_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<unsigned long long*>(tot), 4);
    q_check_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(q->qoff, S, Q, q->base_work, units, bad);
    uint32_t badh = 0;
    if ((e = hipMemcpyAsync(&badh, bad, 4, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_drain");
    if (badh & 4)
        return fail(c, DM_EINVAL, "dm_queue_drain: queue offsets out of order or range");
    if (badh)
        return fail(c, DM_EINVAL, "dm_queue_drain: negative units or base work");
    const QIn a{q->qoff, q->rec_id, q->unc_here, q->alt, q->unc_alt};
    const QOut b{out->qoff, out->rec_id, out->unc_here, out->alt, out->unc_alt};
    if (Q) {
        // uncached tokens widened for the scan
        q_widen_kernel<<<grid_for(Q, 256, 8192), 256, 0, st>>>(q->unc_here, Q, here64);
        if ((e = exclusive_scan_u64(c, here64, Q, hs, tot)) != hipSuccess)
            return hip_fail(c, e, "dm_queue_drain");
        q_drain_kernel<<<grid_for(Q, 256, 1024), 256, 4 * S, st>>>(a, S, Q, q->base_work, units, hs,
                                                              popped, npop);
    }
    const int64_t* base_in = q->base_work;
    q_drain_len_kernel<<<grid_for(S, 256), 256, 0, st>>>(q->qoff, S, npop, base_in, units, len2,
                                                         out->base_work);
    if ((e = exclusive_scan_u64(c, len2, S, ex, tot + 1)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_drain");
    q_fin_offsets_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(ex, tot + 1, S, out->qoff);
    if (Q)
        q_drain_keep_kernel<<<grid_for(Q, 256, 8192), 256, 0, st>>>(a, S, Q, base_in, units, hs,
                                                                   popped, npop, b);
    if ((e = hipGetLastError()) != hipSuccess || (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_drain");
    return DM_OK;
}

dm_status queue_reprobe(dm_ctx* c, const dm_queues* q, const int64_t* coff, const uint64_t* keys,
                        uint64_t n_keys, const int64_t* plen, uint64_t n_ids,
                        const dm_queue_out* out)
{
    const uint32_t S = c->cfg.max_slots;
    hipError_t e = q_quiesce(c);
    int64_t Q = 0;
    if (e == hipSuccess && (e = q_count(c, q->qoff, &Q)) == hipErrorInvalidValue)
        return fail(c, DM_EINVAL, "dm_queue_reprobe: qoff[0] must be 0, fewer than 2^32 records");
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_queue_reprobe");
    if ((uint64_t)Q > out->cap)
        return fail(c, DM_EFULL, "dm_queue_reprobe: the output holds fewer records than the input");
    if (Q && (!coff || !plen || !aligned(coff) || !aligned(plen) || (n_keys && !keys) ||
              (keys && !aligned(keys))))
        return fail(c, DM_EINVAL, "dm_queue_reprobe: null or misaligned chain arrays");
    hipStream_t st = c->stream;
    uint32_t* bad = static_cast<uint32_t*>(scratch_get(c, kSlotMembers, 256, &e));
    if (!bad)
        return hip_fail(c, e, "dm_queue_reprobe");
    uint32_t bshift = 0;
    while ((1u << bshift) < c->cfg.block_size)
        bshift++;
    q_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<unsigned long long*>(bad), 1);
    q_check_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(q->qoff, S, Q, nullptr, nullptr, bad);
    const QIn a{q->qoff, q->rec_id, q->unc_here, q->alt, q->unc_alt};
    if (Q)
        q_reprobe_check_kernel<<<grid_for(Q, 256, 8192), 256, 0, st>>>(a, S, Q, n_ids, coff, n_keys,
                                                                       plen, bshift, bad);
    uint32_t badh = 0;
    if ((e = hipMemcpyAsync(&badh, bad, 4, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_reprobe");
    if (badh & 4)
        return fail(c, DM_EINVAL, "dm_queue_reprobe: queue offsets out of order or range");
    if (badh)
        return fail(c, DM_EINVAL, "dm_queue_reprobe: a record id without a chain, a chain outside "
                                  "the key array or longer than its prompt, a prompt outside "
                                  "[0, 2^32), or an alternative >= max_slots");
    q_copy_offsets_kernel<<<grid_for(S + 1, 256), 256, 0, st>>>(q->qoff, q->base_work, S,
                                                                out->qoff, out->base_work);
    const QOut b{out->qoff, out->rec_id, out->unc_here, out->alt, out->unc_alt};
    if (Q)
        q_reprobe_kernel<<<grid_for(Q, 4, 8192), 256, 0, st>>>(a, S, Q, coff, keys, plen,
                                                               c->d_tables, c->cfg.index_log2_slots,
                                                               bshift, b);
    if ((e = hipGetLastError()) != hipSuccess || (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_queue_reprobe");
    return DM_OK;
}

}  // namespace dm
