// Adaptive hash-key length (Sec. 3.2, "How long prefix is appropriate for
// the hash key?"; Sec. A.1.1): the prefix hotness tree's set-up, window
// close and export, and the window's record of each routed batch.  Routing
// reads the tree in ring_key_kernel and extend_kernel (dm_hash.hip).
//
// The tree is the set of its extended prefixes (canonical f1 key of each
// prefix's last block) in an open-addressing table of 8-slot buckets, probed
// like the instance indexes.  The window's record holds every prefix of
// depth >= K of every routed request (its f1 block keys from block K - 1
// on, appended after the batch's members pass).
//
// Closing a window applies the hot and cold rules until nothing changes.
// A prefix's count never exceeds its parent's, so with W routed requests
// and n live instances the result is the set of prefixes with count c
//   extended now:  c * n >= W      (not cold: rho >= 1/n)
//   a leaf now:    c * n >  2 W    (hot: rho > 2/n)
// (extended prefixes the window never saw, c = 0, are dropped): the record
// sorted in place (radix), each run of equal keys counted at its first
// entry, the kept ones compacted in key order into the next tree (built in
// the other table).
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

__global__ void kl_fill_kernel(uint64_t* __restrict__ p, uint64_t n, uint64_t v)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// Distinct canonical keys into an empty table with room to spare (at most
// half full): the first empty slot along the key's bucket sequence.
__global__ void kl_insert_kernel(uint64_t* __restrict__ tab, uint32_t ls,
                                 const uint64_t* __restrict__ keys, const uint64_t* __restrict__ n_p)
{
    const uint64_t n = *n_p;
    const uint32_t nbk = 1u << (ls - 3);
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t k = keys[i];
        uint32_t b = home32(k, ls);
        bool done = false;
        for (uint32_t step = 0; step < nbk && !done; step++, b = (b + 1) & (nbk - 1))
            for (uint32_t s = 0; s < kBucket && !done; s++) {
                const unsigned long long prev =
                    atomicCAS((unsigned long long*)(tab + (uint64_t)b * kBucket + s),
                              (unsigned long long)kEmpty, (unsigned long long)k);
                done = prev == kEmpty || prev == k;
            }
    }
}

// Window record of one batch: request r contributes its block keys from
// block K - 1 on (its prefixes of depth >= K), canonical, at the record's
// current end plus its offset among the batch's entries.
__global__ void kl_entries_kernel(const uint64_t* __restrict__ bstart, uint64_t n, uint64_t K,
                                  uint64_t* __restrict__ ent)
{
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t nfull = bstart[r + 1] - bstart[r];
        ent[r] = nfull >= K ? nfull - K + 1 : 0;
    }
}

__global__ void kl_append_kernel(uint64_t n, const uint64_t* __restrict__ bstart,
                                 const uint64_t* __restrict__ epos,
                                 const uint64_t* __restrict__ ent, uint64_t K,
                                 const uint64_t* __restrict__ hkeys, uint64_t* __restrict__ log,
                                 uint32_t* __restrict__ roots, uint64_t cap,
                                 const unsigned long long* __restrict__ log_n)
{
    const uint64_t base = *log_n;
    const uint64_t w = blockIdx.x * (uint64_t)(blockDim.x >> 6) +
                       __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t nw = (uint64_t)gridDim.x * (blockDim.x >> 6);
    const uint32_t lane = threadIdx.x & 63;
    for (uint64_t r = w; r < n; r += nw) {
        const uint64_t e = ent[r], at = base + epos[r];
        const uint64_t* src = hkeys + bstart[r] + (K - 1);
        for (uint64_t j = lane; j < e; j += kWave)
            if (at + j < cap)
                log[at + j] = canon_key(src[j]);
        // the request's first entry (its depth-K prefix) starts its run
        if (lane == 0 && e && at < cap)
            atomicOr(&roots[at >> 5], 1u << (at & 31));
    }
}

// Roots of the record: per 32-entry word its root count (for a scan).
__global__ void kl_root_count_kernel(const uint32_t* __restrict__ roots, uint64_t nw,
                                     uint64_t* __restrict__ cnt)
{
    for (uint64_t w = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; w < nw;
         w += (uint64_t)gridDim.x * blockDim.x)
        cnt[w] = __popc(roots[w]);
}

// Run (request) of record entry i: the roots at or before it, minus one.
__device__ __forceinline__ uint64_t kl_run_of(const uint32_t* roots, const uint64_t* wpre,
                                              uint64_t i)
{
    const uint32_t below = roots[i >> 5] & (0xFFFFFFFFu >> (31 - (i & 31)));  // bits <= i
    return wpre[i >> 5] + __popc(below) - 1;
}

// Each run's root key, in record order.
__global__ void kl_root_keys_kernel(const uint64_t* __restrict__ log, uint64_t m,
                                    const uint32_t* __restrict__ roots,
                                    const uint64_t* __restrict__ wpre, uint64_t* __restrict__ rk)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x)
        if ((roots[i >> 5] >> (i & 31)) & 1)
            rk[kl_run_of(roots, wpre, i)] = log[i];
}

// Over the sorted root keys: at the first of each run of equal keys, flag
// it when its count c (requests carrying that depth-K prefix) has
// c n >= W.  No prefix under a root without it can reach c n >= W.
__global__ void kl_hot_root_kernel(const uint64_t* __restrict__ keys, uint64_t m, uint64_t W,
                                   uint64_t n_live, uint64_t* __restrict__ flag)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t key = keys[i];
        uint64_t f = 0;
        if (i == 0 || keys[i - 1] != key) {
            uint64_t lo = i + 1, hi = m;
            while (lo < hi) {
                const uint64_t mid = lo + (hi - lo) / 2;
                if (keys[mid] == key)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            f = (lo - i) * n_live >= W ? 1 : 0;
        }
        flag[i] = f;
    }
}

// Is key among the h sorted hot roots?
__device__ __forceinline__ bool kl_is_hot(const uint64_t* hot, uint64_t h, uint64_t key)
{
    uint64_t lo = 0, hi = h;
    while (lo < hi) {
        const uint64_t mid = lo + (hi - lo) / 2;
        if (hot[mid] < key)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo < h && hot[lo] == key;
}

// keep[i] = 1 for record entries whose run has a hot root.
__global__ void kl_keep_kernel(uint64_t m, const uint32_t* __restrict__ roots,
                               const uint64_t* __restrict__ wpre, const uint64_t* __restrict__ rk,
                               const uint64_t* __restrict__ hot, const uint64_t* __restrict__ h_p,
                               uint64_t* __restrict__ keep)
{
    const uint64_t h = *h_p;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x)
        keep[i] = h && kl_is_hot(hot, h, rk[kl_run_of(roots, wpre, i)]) ? 1 : 0;
}

__global__ void kl_zero_u32_kernel(uint32_t* __restrict__ p, uint64_t n)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

__global__ void kl_advance_kernel(unsigned long long* __restrict__ log_n,
                                  const uint64_t* __restrict__ total, uint64_t cap,
                                  uint32_t* __restrict__ status)
{
    const unsigned long long v = *log_n + *total;
    *log_n = v;
    if (v > cap)
        atomicOr(status, kErrFull);
}

// flag[i] = 1 at the first entry of each run of equal sorted keys whose
// prefix the next tree holds: count c = run length (its end by bisection),
// extended now and c n >= W, or a leaf now and c n > 2 W.
__global__ void kl_decide_kernel(const uint64_t* __restrict__ keys, uint64_t m,
                                 const uint64_t* __restrict__ tab, uint32_t ls, uint64_t W,
                                 uint64_t n_live, uint64_t* __restrict__ flag)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t key = keys[i];
        uint64_t f = 0;
        if (i == 0 || keys[i - 1] != key) {
            uint64_t lo = i + 1, hi = m;  // first index past the run in [lo, hi]
            while (lo < hi) {
                const uint64_t mid = lo + (hi - lo) / 2;
                if (keys[mid] == key)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            const uint64_t cnt = lo - i;
            const bool ext = table_has(tab, ls, key);
            f = (ext ? cnt * n_live >= W : cnt * n_live > 2 * W) ? 1 : 0;
        }
        flag[i] = f;
    }
}

// Kept prefixes in key order, at most cap of them written.
__global__ void kl_compact_kernel(const uint64_t* __restrict__ keys,
                                  const uint64_t* __restrict__ flag,
                                  const uint64_t* __restrict__ pos, uint64_t m,
                                  uint64_t* __restrict__ out, uint64_t cap)
{
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x)
        if (flag[i] && pos[i] < cap)
            out[pos[i]] = keys[i];
}

template <typename T>
T* carve(uint8_t*& p, uint64_t n)
{
    T* r = reinterpret_cast<T*>(p);
    p += ((n * sizeof(T) + 255) / 256) * 256;
    return r;
}

// All work of the context finished (pipelined batches included).
hipError_t quiesce(dm_ctx* c)
{
    hipError_t e = join_selection(c);
    if (e == hipSuccess)
        e = sync_streams(c);
    return e;
}

void reset_window(dm_ctx* c)
{
    KeyLen& k = c->kl;
    k.win = 0;
    kl_fill_kernel<<<1, 64, 0, c->stream>>>(reinterpret_cast<uint64_t*>(k.log_n), 1, 0);
}

size_t up256k(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

void keylen_free(dm_ctx* c)
{
    KeyLen& k = c->kl;
    for (uint64_t* p : {k.tab[0], k.tab[1], k.list, k.log})
        if (p)
            (void)hipFree(p);
    if (k.roots)
        (void)hipFree(k.roots);
    if (k.log_n)
        (void)hipFree(k.log_n);
    k = KeyLen{};
}

uint64_t keylen_record_bytes(uint64_t n) { return 2 * up256k(8 * n) + 256; }

// (Malformed offsets leave every request with no full block in bstart, so
// such a batch records nothing.)
hipError_t keylen_record(dm_ctx* c, uint64_t n, const uint64_t* bstart, const uint64_t* hkeys,
                         uint64_t* work)
{
    const KeyLen& k = c->kl;
    uint64_t* ent = work;
    uint64_t* epos = work + up256k(8 * n) / 8;
    uint64_t* total = work + 2 * (up256k(8 * n) / 8);
    const uint64_t K = c->cfg.key_blocks;
    kl_entries_kernel<<<grid_for(n, 256, 8192), 256, 0, c->stream>>>(bstart, n, K, ent);
    hipError_t e = exclusive_scan_u64(c, ent, n, epos, total);
    if (e != hipSuccess)
        return e;
    kl_append_kernel<<<grid_for(n, 4, 16384), 256, 0, c->stream>>>(n, bstart, epos, ent, K, hkeys,
                                                                   k.log, k.roots, k.cap, k.log_n);
    kl_advance_kernel<<<1, 1, 0, c->stream>>>(k.log_n, total, k.cap, c->d_status);
    return hipGetLastError();
}

dm_status keylen_enable(dm_ctx* c, uint64_t max_nodes, uint64_t max_window_blocks)
{
    if (max_nodes > (1ull << 28))
        return fail(c, DM_EINVAL, "dm_keylen_enable: max_nodes must be <= 2^28");
    if (max_nodes && (max_window_blocks == 0 || max_window_blocks >= (1ull << 36)))
        return fail(c, DM_EINVAL, "dm_keylen_enable: max_window_blocks must be in [1, 2^36)");
    hipError_t e = quiesce(c);
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_keylen_enable");
    keylen_free(c);
    if (max_nodes == 0)
        return DM_OK;
    KeyLen k;
    k.max_nodes = max_nodes;
    k.cap = max_window_blocks;
    k.log2 = 6;
    while ((1ull << k.log2) < 2 * max_nodes)
        k.log2++;
    const uint64_t slots = 1ull << k.log2;
    if ((e = hipMalloc(&k.tab[0], slots * 8)) == hipSuccess &&
        (e = hipMalloc(&k.tab[1], slots * 8)) == hipSuccess &&
        (e = hipMalloc(&k.list, max_nodes * 8)) == hipSuccess &&
        (e = hipMalloc(&k.log, k.cap * 8)) == hipSuccess &&
        (e = hipMalloc(&k.roots, (k.cap / 32 + 1) * 4)) == hipSuccess)
        e = hipMalloc(&k.log_n, 8);
    c->kl = k;
    if (e != hipSuccess) {
        keylen_free(c);
        return fail(c, DM_ENOMEM, "dm_keylen_enable: device allocation failed");
    }
    c->kl.on = true;
    kl_fill_kernel<<<grid_for(slots, 256), 256, 0, c->stream>>>(c->kl.tab[0], slots, kEmpty);
    kl_zero_u32_kernel<<<grid_for(k.cap / 32 + 1, 256, 8192), 256, 0, c->stream>>>(
        c->kl.roots, k.cap / 32 + 1);
    reset_window(c);
    if ((e = hipGetLastError()) == hipSuccess)
        e = hipStreamSynchronize(c->stream);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_keylen_enable");
}

dm_status keylen_window(dm_ctx* c)
{
    KeyLen& k = c->kl;
    if (!k.on)
        return fail(c, DM_ESTATE, "dm_keylen_window: the hotness tree is off");
    if (c->n_live == 0)
        return fail(c, DM_ESTATE, "dm_keylen_window: rings not built");
    hipError_t e = quiesce(c);
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_keylen_window");
    unsigned long long M = 0;
    if ((e = hipMemcpy(&M, k.log_n, sizeof(M), hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(c, e, "dm_keylen_window");
    const uint64_t W = k.win;
    hipStream_t st = c->stream;
    if (M > k.cap) {
        reset_window(c);
        kl_zero_u32_kernel<<<grid_for(k.cap / 32 + 1, 256, 8192), 256, 0, st>>>(k.roots,
                                                                              k.cap / 32 + 1);
        if ((e = hipStreamSynchronize(st)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        return fail(c, DM_EFULL, "dm_keylen_window: the window held more prefixes than its "
                                 "record (tree unchanged)");
    }
    if (W == 0) {  // no traffic: no change
        reset_window(c);
        e = hipStreamSynchronize(st);
        return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_keylen_window");
    }
    const uint64_t Ma = M ? M : 1, outcap = k.max_nodes + 1, nw = (Ma + 31) / 32;
    uint8_t* w = static_cast<uint8_t*>(scratch_get(
        c, kSlotMembers, 3 * up256k(8 * Ma) + up256k(8 * outcap) + 2 * up256k(8 * nw) + 1024, &e));
    if (!w)
        return hip_fail(c, e, "dm_keylen_window");
    uint64_t* ktmp = carve<uint64_t>(w, Ma);
    uint64_t* flag = carve<uint64_t>(w, Ma);
    uint64_t* pos = carve<uint64_t>(w, Ma);
    uint64_t* out = carve<uint64_t>(w, outcap);
    uint64_t* wcnt = carve<uint64_t>(w, nw);
    uint64_t* wpre = carve<uint64_t>(w, nw);
    uint64_t* count = carve<uint64_t>(w, 4);
    kl_fill_kernel<<<1, 64, 0, st>>>(count, 4, 0);
    if (M) {
        // Only prefixes under a root (depth-K prefix) carried by at least
        // W / n requests can be kept (a prefix's count never exceeds its
        // root's): count the roots first, one per request, and sort only
        // the entries of requests with such a root.
        kl_root_count_kernel<<<grid_for(nw, 256, 8192), 256, 0, st>>>(k.roots, nw, wcnt);
        uint64_t R = 0;
        if ((e = exclusive_scan_u64(c, wcnt, nw, wpre, count + 1)) != hipSuccess ||
            (e = hipMemcpyAsync(&R, count + 1, 8, hipMemcpyDeviceToHost, st)) != hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        const uint64_t Ra = R ? R : 1;
        uint8_t* rw = static_cast<uint8_t*>(
            scratch_get(c, kSlotProbe, 6 * up256k(8 * Ra) + 256, &e));
        if (!rw)
            return hip_fail(c, e, "dm_keylen_window");
        uint64_t* rk = carve<uint64_t>(rw, Ra);     // each run's root, record order
        uint64_t* rs = carve<uint64_t>(rw, Ra);     // the same, sorted
        uint64_t* rtmp = carve<uint64_t>(rw, Ra);
        uint64_t* rflag = carve<uint64_t>(rw, Ra);
        uint64_t* rpos = carve<uint64_t>(rw, Ra);
        uint64_t* hot = carve<uint64_t>(rw, Ra);
        const uint32_t g = grid_for(M, 256, 8192), gr = grid_for(Ra, 256, 8192);
        kl_root_keys_kernel<<<g, 256, 0, st>>>(k.log, M, k.roots, wpre, rk);
        uint64_t Mk = 0;
        if ((e = hipMemcpyAsync(rs, rk, 8 * R, hipMemcpyDeviceToDevice, st)) != hipSuccess ||
            (e = radix_sort_kv(c, rs, nullptr, rtmp, nullptr, R, 64)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        kl_hot_root_kernel<<<gr, 256, 0, st>>>(rs, R, W, c->n_live, rflag);
        if ((e = exclusive_scan_u64(c, rflag, R, rpos, count + 2)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        kl_compact_kernel<<<gr, 256, 0, st>>>(rs, rflag, rpos, R, hot, Ra);
        kl_keep_kernel<<<g, 256, 0, st>>>(M, k.roots, wpre, rk, hot, count + 2, flag);
        if ((e = exclusive_scan_u64(c, flag, M, pos, count + 3)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        kl_compact_kernel<<<g, 256, 0, st>>>(k.log, flag, pos, M, ktmp, Ma);
        if ((e = hipMemcpyAsync(&Mk, count + 3, 8, hipMemcpyDeviceToHost, st)) != hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        if (Mk) {
            const uint32_t gk = grid_for(Mk, 256, 8192);
            if ((e = radix_sort_kv(c, ktmp, nullptr, pos, nullptr, Mk, 64)) != hipSuccess)
                return hip_fail(c, e, "dm_keylen_window");
            kl_decide_kernel<<<gk, 256, 0, st>>>(ktmp, Mk, k.tab[k.cur], k.log2, W, c->n_live,
                                                 flag);
            if ((e = exclusive_scan_u64(c, flag, Mk, pos, count)) != hipSuccess)
                return hip_fail(c, e, "dm_keylen_window");
            kl_compact_kernel<<<gk, 256, 0, st>>>(ktmp, flag, pos, Mk, out, outcap);
        }
        kl_zero_u32_kernel<<<grid_for(nw, 256, 8192), 256, 0, st>>>(k.roots, nw);
    }
    uint64_t n_next = 0;
    if ((e = hipGetLastError()) != hipSuccess ||
        (e = hipMemcpyAsync(&n_next, count, 8, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_keylen_window");
    reset_window(c);
    if (n_next > k.max_nodes) {
        if ((e = hipStreamSynchronize(st)) != hipSuccess)
            return hip_fail(c, e, "dm_keylen_window");
        return fail(c, DM_EFULL, "dm_keylen_window: the new tree would hold " +
                                     std::to_string(n_next) + " extended prefixes, more than " +
                                     std::to_string(k.max_nodes) + " (tree unchanged)");
    }
    const int nx = 1 - k.cur;
    const uint64_t slots = 1ull << k.log2;
    kl_fill_kernel<<<grid_for(slots, 256), 256, 0, st>>>(k.tab[nx], slots, kEmpty);
    kl_insert_kernel<<<grid_for(std::max<uint64_t>(n_next, 1), 256, 4096), 256, 0, st>>>(
        k.tab[nx], k.log2, out, count);
    if (n_next &&
        (e = hipMemcpyAsync(k.list, out, n_next * 8, hipMemcpyDeviceToDevice, st)) != hipSuccess)
        return hip_fail(c, e, "dm_keylen_window");
    if ((e = hipGetLastError()) != hipSuccess || (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "dm_keylen_window");
    k.cur = nx;
    k.n_ext = n_next;
    return DM_OK;
}

dm_status keylen_export(dm_ctx* c, uint64_t* keys_host, uint64_t cap, uint64_t* n_host)
{
    const KeyLen& k = c->kl;
    if (!k.on)
        return fail(c, DM_ESTATE, "dm_keylen_export: the hotness tree is off");
    hipError_t e = quiesce(c);
    const uint64_t m = std::min(cap, k.n_ext);
    if (e == hipSuccess && m)
        e = hipMemcpy(keys_host, k.list, m * 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_keylen_export");
    *n_host = k.n_ext;
    return DM_OK;
}

}  // namespace dm
