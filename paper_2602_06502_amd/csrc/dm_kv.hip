// KV save with least-recently-used eviction: the serving step after routing
// (the KV query and save of Sec. A.3.2), on the device.  A served request's
// full blocks are touched on its instance, deepest block first; each
// instance's cache is the cap most recently touched distinct keys, and the
// difference is applied to its index (erase, then insert).
//
// The record of saved keys is one flat array of (instance, key, time of the
// latest touch).  One save:
//   1. the record and the batch's touches are concatenated;
//   2. sorted by key, then stably by instance (LSD radix), so each
//      (instance, key) is one run; each run keeps its latest time and
//      whether the key was already cached;
//   3. the runs sorted by (instance, time); in each instance the first
//      count - cap (the least recent) are dropped;
//   4. dropped keys that were cached are erased, kept keys that were not are
//      inserted, instance by instance, through the index's own kernels; the
//      kept runs become the record.
#include <algorithm>
#include <vector>

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

size_t up256v(size_t x) { return (x + 255) & ~size_t(255); }

// The record's entries, then the batch's touches (one wave per request):
// block b of request r at time clock + start_r + (nfull_r - 1 - b).
__global__ void kv_fill_kernel(const uint64_t* __restrict__ rkey, const uint64_t* __restrict__ rt,
                               const uint32_t* __restrict__ rinst, uint64_t nrec, uint64_t n,
                               const uint64_t* __restrict__ bstart,
                               const uint64_t* __restrict__ block_keys,
                               const uint32_t* __restrict__ inst, uint64_t clock,
                               uint64_t* __restrict__ key, uint64_t* __restrict__ t,
                               uint32_t* __restrict__ ins, uint32_t* __restrict__ idx)
{
    const uint64_t tid = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x;
    const uint64_t nth = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = tid; i < nrec; i += nth) {
        key[i] = rkey[i];
        t[i] = rt[i];
        ins[i] = rinst[i];
        idx[i] = (uint32_t)i;
    }
    const uint64_t w = blockIdx.x * (uint64_t)(blockDim.x >> 6) +
                       __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t nw = (uint64_t)gridDim.x * (blockDim.x >> 6);
    const uint32_t lane = threadIdx.x & 63;
    for (uint64_t r = w; r < n; r += nw) {
        const uint64_t s = bstart[r], nf = bstart[r + 1] - s;
        const uint32_t c = inst[r];
        // entries in touch order (deepest block first), so that after the
        // stable sorts a run's last entry is its latest touch of this batch
        for (uint64_t b = lane; b < nf; b += kWave) {
            const uint64_t e = nrec + s + (nf - 1 - b);
            key[e] = block_keys[s + b];
            t[e] = clock + (e - nrec);
            ins[e] = c;
            idx[e] = (uint32_t)e;
        }
    }
}

// bad |= 2 if a request's instance is out of range.
__global__ void kv_check_kernel(const uint32_t* __restrict__ inst, uint64_t n, uint32_t S,
                                uint32_t* __restrict__ bad)
{
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x)
        if (inst[r] >= S)
            atomicOr(bad, 2u);
}

// Sort key of the second pass: the instance of each entry, in the key order.
__global__ void kv_inst_key_kernel(const uint32_t* __restrict__ order,
                                   const uint32_t* __restrict__ ins, uint64_t m,
                                   uint64_t* __restrict__ out)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x)
        out[i] = ins[order[i]];
}

// head[p] = 1 where sorted position p starts an (instance, key) run.
__global__ void kv_head_kernel(const uint32_t* __restrict__ order,
                               const uint64_t* __restrict__ key, const uint32_t* __restrict__ ins,
                               uint64_t m, uint64_t* __restrict__ head)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < m;
         p += (uint64_t)gridDim.x * blockDim.x) {
        bool h = p == 0;
        if (!h) {
            const uint32_t a = order[p], b = order[p - 1];
            h = key[a] != key[b] || ins[a] != ins[b];
        }
        head[p] = h ? 1 : 0;
    }
}

// Runs of equal (instance, key) in sorted order, their entries in input
// order (the sorts are stable): a record entry first if there is one, then
// the batch's touches by increasing time.  The head writes the run's key,
// instance, whether it was already cached and its first entry's time; the
// last entry's time is merged in by kv_runs_last_kernel.
__global__ void kv_runs_kernel(const uint32_t* __restrict__ order,
                               const uint64_t* __restrict__ key, const uint64_t* __restrict__ t,
                               const uint32_t* __restrict__ ins, uint64_t m, uint64_t nrec,
                               const uint64_t* __restrict__ head, const uint64_t* __restrict__ run,
                               uint64_t* __restrict__ ukey, uint64_t* __restrict__ ut,
                               uint32_t* __restrict__ uins, uint32_t* __restrict__ uold)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < m;
         p += (uint64_t)gridDim.x * blockDim.x) {
        if (!head[p])
            continue;
        const uint32_t a = order[p];
        const uint64_t u = run[p];
        ukey[u] = key[a];
        ut[u] = t[a];
        uins[u] = ins[a];
        uold[u] = a < nrec ? 1u : 0u;
    }
}

// The latest time of each run of more than one entry: the larger of its
// first entry's (a record entry may carry any earlier time) and its last's.
__global__ void kv_runs_last_kernel(const uint32_t* __restrict__ order,
                                    const uint64_t* __restrict__ t, uint64_t m,
                                    const uint64_t* __restrict__ head,
                                    const uint64_t* __restrict__ run, uint64_t* __restrict__ ut)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < m;
         p += (uint64_t)gridDim.x * blockDim.x) {
        if (head[p] || (p + 1 < m && !head[p + 1]))
            continue;
        const uint64_t u = run[p] - 1;
        const uint64_t x = t[order[p]];
        ut[u] = ut[u] > x ? ut[u] : x;
    }
}

// Runs per instance: the runs are in (instance, key) order, so each
// instance's runs are one range; its bounds are where the instance changes.
__global__ void kv_count_kernel(const uint32_t* __restrict__ uins, uint64_t u,
                                unsigned long long* __restrict__ first,
                                unsigned long long* __restrict__ end)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < u;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t c = uins[i];
        if (i == 0 || uins[i - 1] != c)
            first[c] = i;
        if (i + 1 == u || uins[i + 1] != c)
            end[c] = i + 1;
    }
}

// cnt[c] = end[c] - first[c] (both zero for an instance without runs).
__global__ void kv_count_fin_kernel(const unsigned long long* __restrict__ first,
                                    unsigned long long* __restrict__ end, uint32_t S)
{
    for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < S; c += gridDim.x * blockDim.x)
        end[c] -= first[c];
}

// Sort key of the third pass: instance above the time (times < 2^40).
__global__ void kv_time_key_kernel(const uint64_t* __restrict__ ut,
                                   const uint32_t* __restrict__ uins, uint64_t u,
                                   uint64_t* __restrict__ k, uint32_t* __restrict__ v)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < u;
         i += (uint64_t)gridDim.x * blockDim.x) {
        k[i] = ((uint64_t)uins[i] << 40) | ut[i];
        v[i] = (uint32_t)i;
    }
}

// For the runs in (instance, time) order: dropped (the first count - cap of
// its instance) or kept; flags for the erase, insert and record lists.
__global__ void kv_decide_kernel(const uint32_t* __restrict__ order2,
                                 const uint32_t* __restrict__ uins,
                                 const uint32_t* __restrict__ uold, uint64_t u,
                                 const unsigned long long* __restrict__ cnt,
                                 const uint64_t* __restrict__ ibase, uint64_t cap,
                                 uint64_t* __restrict__ f_erase, uint64_t* __restrict__ f_insert,
                                 uint64_t* __restrict__ f_keep)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < u;
         p += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t x = order2[p];
        const uint32_t c = uins[x];
        const uint64_t n_c = cnt[c];
        const uint64_t drop = cap && n_c > cap ? n_c - cap : 0;
        const bool kept = p - ibase[c] >= drop;
        f_erase[p] = (!kept && uold[x]) ? 1 : 0;
        f_insert[p] = (kept && !uold[x]) ? 1 : 0;
        f_keep[p] = kept ? 1 : 0;
    }
}

__global__ void kv_emit_kernel(const uint32_t* __restrict__ order2,
                               const uint64_t* __restrict__ ukey, const uint64_t* __restrict__ ut,
                               const uint32_t* __restrict__ uins, uint64_t u,
                               const uint64_t* __restrict__ f_erase,
                               const uint64_t* __restrict__ p_erase,
                               const uint64_t* __restrict__ f_insert,
                               const uint64_t* __restrict__ p_insert,
                               const uint64_t* __restrict__ f_keep,
                               const uint64_t* __restrict__ p_keep,
                               uint64_t* __restrict__ erase_keys,
                               uint64_t* __restrict__ insert_keys, uint64_t* __restrict__ rkey,
                               uint64_t* __restrict__ rt, uint32_t* __restrict__ rinst)
{
    for (uint64_t p = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; p < u;
         p += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t x = order2[p];
        if (f_erase[p])
            erase_keys[p_erase[p]] = ukey[x];
        if (f_insert[p])
            insert_keys[p_insert[p]] = ukey[x];
        if (f_keep[p]) {
            const uint64_t q = p_keep[p];
            rkey[q] = ukey[x];
            rt[q] = ut[x];
            rinst[q] = uins[x];
        }
    }
}

// Per instance: how many of the erase and insert lists' entries are its.
// Its runs are positions [ibase[c], ibase[c] + cnt[c]) of the (instance,
// time) order, so the counts are differences of the lists' exclusive scans
// (tot_e, tot_i: the scans' totals).
__global__ void kv_list_count_kernel(const unsigned long long* __restrict__ cnt,
                                     const uint64_t* __restrict__ ibase, uint32_t S, uint64_t u,
                                     const uint64_t* __restrict__ p_erase,
                                     const uint64_t* __restrict__ p_insert,
                                     const uint64_t* __restrict__ tot_e,
                                     const uint64_t* __restrict__ tot_i,
                                     unsigned long long* __restrict__ ce,
                                     unsigned long long* __restrict__ ci)
{
    for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < S; c += gridDim.x * blockDim.x) {
        if (!cnt[c]) {
            ce[c] = ci[c] = 0;
            continue;
        }
        const uint64_t lo = ibase[c], hi = lo + cnt[c];
        ce[c] = (hi < u ? p_erase[hi] : *tot_e) - p_erase[lo];
        ci[c] = (hi < u ? p_insert[hi] : *tot_i) - p_insert[lo];
    }
}

__global__ void kv_zero_kernel(unsigned long long* __restrict__ p, uint64_t n)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// Record entries of the given instances dropped (their indexes were emptied).
__global__ void kv_forget_kernel(const uint32_t* __restrict__ rinst, uint64_t n,
                                 const uint8_t* __restrict__ gone, uint64_t* __restrict__ keep)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        keep[i] = gone[rinst[i]] ? 0 : 1;
}

__global__ void kv_compact_kernel(const uint64_t* __restrict__ keep,
                                  const uint64_t* __restrict__ pos, uint64_t n,
                                  const uint64_t* __restrict__ k0, const uint64_t* __restrict__ t0,
                                  const uint32_t* __restrict__ i0, uint64_t* __restrict__ k1,
                                  uint64_t* __restrict__ t1, uint32_t* __restrict__ i1)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        if (keep[i]) {
            const uint64_t q = pos[i];
            k1[q] = k0[i];
            t1[q] = t0[i];
            i1[q] = i0[i];
        }
}

hipError_t quiesce_kv(dm_ctx* c)
{
    hipError_t e = join_selection(c);
    if (e == hipSuccess)
        e = sync_streams(c);
    return e;
}

// The record's arrays hold at least n entries (contents kept).
hipError_t kv_reserve(dm_ctx* c, uint64_t n)
{
    KvRecord& r = c->kv;
    if (n <= r.cap)
        return hipSuccess;
    const uint64_t cap = std::max<uint64_t>(n, 2 * r.cap);
    uint64_t *k = nullptr, *t = nullptr;
    uint32_t* i = nullptr;
    hipError_t e;
    if ((e = hipMalloc(&k, cap * 8)) != hipSuccess || (e = hipMalloc(&t, cap * 8)) != hipSuccess ||
        (e = hipMalloc(&i, cap * 4)) != hipSuccess) {
        (void)hipFree(k);
        (void)hipFree(t);
        (void)hipFree(i);
        return e;
    }
    if (r.n && ((e = hipMemcpy(k, r.key, r.n * 8, hipMemcpyDeviceToDevice)) != hipSuccess ||
                (e = hipMemcpy(t, r.t, r.n * 8, hipMemcpyDeviceToDevice)) != hipSuccess ||
                (e = hipMemcpy(i, r.inst, r.n * 4, hipMemcpyDeviceToDevice)) != hipSuccess))
        return e;
    (void)hipFree(r.key);
    (void)hipFree(r.t);
    (void)hipFree(r.inst);
    r.key = k;
    r.t = t;
    r.inst = i;
    r.cap = cap;
    return hipSuccess;
}

}  // namespace

void kv_free(dm_ctx* c)
{
    KvRecord& r = c->kv;
    (void)hipFree(r.key);
    (void)hipFree(r.t);
    (void)hipFree(r.inst);
    r = KvRecord{};
}

hipError_t kv_forget(dm_ctx* c, const uint8_t* d_gone)
{
    KvRecord& r = c->kv;
    if (r.n == 0)
        return hipSuccess;
    hipError_t e = hipSuccess;
    const uint64_t n = r.n;
    uint8_t* w = static_cast<uint8_t*>(
        scratch_get(c, kSlotMembers, 2 * up256v(8 * n) + 2 * up256v(8 * n) + up256v(4 * n) + 512, &e));
    if (!w)
        return e;
    uint64_t* keep = carve<uint64_t>(w, n);
    uint64_t* pos = carve<uint64_t>(w, n);
    uint64_t* k1 = carve<uint64_t>(w, n);
    uint64_t* t1 = carve<uint64_t>(w, n);
    uint32_t* i1 = carve<uint32_t>(w, n);
    uint64_t* total = carve<uint64_t>(w, 1);
    const uint32_t g = grid_for(n, 256, 4096);
    kv_forget_kernel<<<g, 256, 0, c->stream>>>(r.inst, n, d_gone, keep);
    if ((e = exclusive_scan_u64(c, keep, n, pos, total)) != hipSuccess)
        return e;
    kv_compact_kernel<<<g, 256, 0, c->stream>>>(keep, pos, n, r.key, r.t, r.inst, k1, t1, i1);
    uint64_t m = 0;
    if ((e = hipMemcpyAsync(&m, total, 8, hipMemcpyDeviceToHost, c->stream)) != hipSuccess ||
        (e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return e;
    if (m &&
        ((e = hipMemcpyAsync(r.key, k1, m * 8, hipMemcpyDeviceToDevice, c->stream)) != hipSuccess ||
         (e = hipMemcpyAsync(r.t, t1, m * 8, hipMemcpyDeviceToDevice, c->stream)) != hipSuccess ||
         (e = hipMemcpyAsync(r.inst, i1, m * 4, hipMemcpyDeviceToDevice, c->stream)) != hipSuccess))
        return e;
    if ((e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return e;
    r.n = m;
    return hipSuccess;
}

dm_status kv_save(dm_ctx* c, const int64_t* offsets, uint64_t n, const uint64_t* block_keys,
                  const uint32_t* inst, uint64_t clock, uint64_t cap, uint64_t* added,
                  uint64_t* removed)
{
    const uint32_t S = c->cfg.max_slots;
    hipError_t e = quiesce_kv(c);
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    hipStream_t st = c->stream;
    KvRecord& rec = c->kv;
    // block starts (offsets checked on the device) and the batch's block count
    uint64_t* bstart =
        static_cast<uint64_t*>(scratch_get(c, kSlotStarts, (n + 2) * sizeof(uint64_t), &e));
    if (!bstart)
        return hip_fail(c, e, "dm_kv_save");
    uint32_t* bad = reinterpret_cast<uint32_t*>(bstart + n + 1);
    kv_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<unsigned long long*>(bad), 1);
    if ((e = block_starts(c, offsets, n, 1ull << 62, bstart, bad)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    if (n)
        kv_check_kernel<<<grid_for(n, 256, 1024), 256, 0, st>>>(inst, n, S, bad);
    uint64_t E = 0;
    uint32_t badh = 0;
    if ((e = hipMemcpyAsync(&E, bstart + n, 8, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipMemcpyAsync(&badh, bad, 4, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    if (badh & 2)
        return fail(c, DM_EINVAL, "dm_kv_save: an instance id is >= max_slots");
    if (badh)
        return fail(c, DM_EINVAL, "dm_kv_save: offsets must be non-decreasing and non-negative");
    if (E && !block_keys)
        return fail(c, DM_EINVAL, "dm_kv_save: null block keys");
    if (clock + E >= (1ull << 40))
        return fail(c, DM_EINVAL, "dm_kv_save: touch times must stay below 2^40");
    const uint64_t M = rec.n + E;
    if (M >= (1ull << 32))
        return fail(c, DM_EINVAL, "dm_kv_save: more than 2^32 record entries");
    if (M == 0) {
        if (added) *added = 0;
        if (removed) *removed = 0;
        return DM_OK;
    }
    // work arrays: entries (key, t, inst, index), their sort temporaries,
    // run heads and ids, the runs, and the flags and positions of the lists
    const uint64_t A = up256v(8 * M), A4 = up256v(4 * M), Sa = up256v(8 * (uint64_t)S);
    uint8_t* w = static_cast<uint8_t*>(
        scratch_get(c, kSlotMembers, 16 * A + 8 * A4 + 4 * Sa + up256v(16 * ((uint64_t)S + 1)) + 4096,
                    &e));
    if (!w)
        return hip_fail(c, e, "dm_kv_save");
    uint64_t* key = carve<uint64_t>(w, M);
    uint64_t* t = carve<uint64_t>(w, M);
    uint32_t* ins = carve<uint32_t>(w, M);
    uint32_t* order = carve<uint32_t>(w, M);
    uint64_t* sk = carve<uint64_t>(w, M);
    uint64_t* sktmp = carve<uint64_t>(w, M);
    uint32_t* vtmp = carve<uint32_t>(w, M);
    uint64_t* head = carve<uint64_t>(w, M);
    uint64_t* run = carve<uint64_t>(w, M);
    uint64_t* ukey = carve<uint64_t>(w, M);
    uint64_t* ut = carve<uint64_t>(w, M);
    uint32_t* uins = carve<uint32_t>(w, M);
    uint32_t* uold = carve<uint32_t>(w, M);
    uint32_t* order2 = carve<uint32_t>(w, M);
    uint64_t* f_erase = carve<uint64_t>(w, M);
    uint64_t* f_insert = carve<uint64_t>(w, M);
    uint64_t* f_keep = carve<uint64_t>(w, M);
    uint64_t* p_erase = carve<uint64_t>(w, M);
    uint64_t* p_insert = carve<uint64_t>(w, M);
    uint64_t* p_keep = carve<uint64_t>(w, M);
    uint64_t* erase_keys = carve<uint64_t>(w, M);
    uint64_t* insert_keys = carve<uint64_t>(w, M);
    unsigned long long* cnt = carve<unsigned long long>(w, S);
    uint64_t* ibase = carve<uint64_t>(w, S);
    unsigned long long* ce = carve<unsigned long long>(w, S);
    unsigned long long* ci = carve<unsigned long long>(w, S);
    uint64_t* tot = carve<uint64_t>(w, 8);
    uint64_t* dseg = carve<uint64_t>(w, 2 * ((uint64_t)S + 1));
    const uint32_t g = grid_for(M, 256, 8192);
    kv_fill_kernel<<<grid_for(std::max(rec.n, n * 64), 256, 8192), 256, 0, st>>>(
        rec.key, rec.t, rec.inst, rec.n, n, bstart, block_keys, inst, clock, key, t, ins, order);
    // (instance, key) runs: by key, then stably by instance
    if ((e = hipMemcpyAsync(sk, key, M * 8, hipMemcpyDeviceToDevice, st)) != hipSuccess ||
        (e = radix_sort_kv(c, sk, order, sktmp, vtmp, M, 64)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    kv_inst_key_kernel<<<g, 256, 0, st>>>(order, ins, M, sk);
    if ((e = radix_sort_kv(c, sk, order, sktmp, vtmp, M, 16)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    kv_head_kernel<<<g, 256, 0, st>>>(order, key, ins, M, head);
    if ((e = exclusive_scan_u64(c, head, M, run, tot)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    kv_runs_kernel<<<g, 256, 0, st>>>(order, key, t, ins, M, rec.n, head, run, ukey, ut, uins,
                                      uold);
    kv_runs_last_kernel<<<g, 256, 0, st>>>(order, t, M, head, run, ut);
    uint64_t U = 0;
    if ((e = hipMemcpyAsync(&U, tot, 8, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    // per instance: run counts and their first place in (instance, time) order
    kv_zero_kernel<<<grid_for(S, 256), 256, 0, st>>>(cnt, S);
    kv_zero_kernel<<<grid_for(S, 256), 256, 0, st>>>(ce, S);
    kv_zero_kernel<<<grid_for(S, 256), 256, 0, st>>>(ci, S);
    const uint32_t gu = grid_for(U, 256, 8192);
    kv_count_kernel<<<gu, 256, 0, st>>>(uins, U, ce, cnt);
    kv_count_fin_kernel<<<grid_for(S, 256), 256, 0, st>>>(ce, cnt, S);
    if ((e = exclusive_scan_u64(c, reinterpret_cast<const uint64_t*>(cnt), S, ibase, tot + 1)) !=
        hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    kv_time_key_kernel<<<gu, 256, 0, st>>>(ut, uins, U, sk, order2);
    if ((e = radix_sort_kv(c, sk, order2, sktmp, vtmp, U, 56)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    kv_decide_kernel<<<gu, 256, 0, st>>>(order2, uins, uold, U, cnt, ibase, cap, f_erase, f_insert,
                                         f_keep);
    if ((e = exclusive_scan_u64(c, f_erase, U, p_erase, tot + 2)) != hipSuccess ||
        (e = exclusive_scan_u64(c, f_insert, U, p_insert, tot + 3)) != hipSuccess ||
        (e = exclusive_scan_u64(c, f_keep, U, p_keep, tot + 4)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    uint64_t totals[3] = {0, 0, 0};  // erased, inserted, kept
    if ((e = hipMemcpyAsync(totals, tot + 2, 24, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    // the record keeps what was there until the new one is written
    if ((e = kv_reserve(c, std::max(totals[2], rec.n))) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    kv_emit_kernel<<<gu, 256, 0, st>>>(order2, ukey, ut, uins, U, f_erase, p_erase, f_insert,
                                       p_insert, f_keep, p_keep, erase_keys, insert_keys, rec.key,
                                       rec.t, rec.inst);
    kv_list_count_kernel<<<grid_for(S, 256), 256, 0, st>>>(cnt, ibase, S, U, p_erase, p_insert,
                                                           tot + 2, tot + 3, ce, ci);
    std::vector<unsigned long long> hce(S), hci(S);
    if ((e = hipMemcpyAsync(hce.data(), ce, 8 * (size_t)S, hipMemcpyDeviceToHost, st)) !=
            hipSuccess ||
        (e = hipMemcpyAsync(hci.data(), ci, 8 * (size_t)S, hipMemcpyDeviceToHost, st)) !=
            hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    rec.n = totals[2];
    // the lists are in instance order: every erase, then every insert
    std::vector<uint64_t> seg(2 * ((size_t)S + 1), 0);
    for (uint32_t i = 0; i < S; i++) {
        seg[i + 1] = seg[i] + hce[i];
        seg[S + 1 + i + 1] = seg[S + 1 + i] + hci[i];
    }
    if ((e = hipMemcpyAsync(dseg, seg.data(), seg.size() * sizeof(uint64_t),
                            hipMemcpyHostToDevice, st)) != hipSuccess ||
        (e = index_erase_many(c, erase_keys, dseg, seg[S])) != hipSuccess ||
        (e = index_insert_many(c, insert_keys, dseg + S + 1, seg.data() + S + 1,
                               seg[2 * (size_t)S + 1])) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    if ((e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_kv_save");
    if (added) *added = totals[1];
    if (removed) *removed = totals[0];
    return DM_OK;
}

}  // namespace dm
