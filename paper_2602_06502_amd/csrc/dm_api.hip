// C ABI of the DualMap engine: argument checks, context state and the
// host-side orchestration of the kernels.  Every computation on the routing
// path runs in the kernels of the other files; this file only validates,
// allocates and launches.
#include <algorithm>
#include <cstring>
#include <string>

#include "dm_internal.h"

using namespace dm;

namespace dm {

dm_status fail(dm_ctx* c, dm_status s, const std::string& msg)
{
    if (c)
        c->err = msg;
    return s;
}

dm_status hip_fail(dm_ctx* c, hipError_t e, const char* what)
{
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
        return fail(c, DM_ENOMEM, std::string(what) + ": out of device memory");
    return fail(c, DM_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

hipError_t sync_streams(dm_ctx* c)
{
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess && c->home_stream != c->stream)
        e = hipStreamSynchronize(c->home_stream);
    for (hipStream_t s : {c->work_stream, c->sel_stream, c->out_stream})
        if (e == hipSuccess && s)
            e = hipStreamSynchronize(s);
    return e;
}

void* scratch_get(dm_ctx* c, int slot, size_t bytes, hipError_t* e)
{
    Scratch& s = c->scratch[slot];
    *e = hipSuccess;
    if (bytes == 0)
        bytes = 256;
    if (c->arena.on) {
        // allocation-free call: the region planned for this slot, or an error
        if (bytes <= c->arena.len[slot])
            return c->arena.base + c->arena.off[slot];
        *e = hipErrorOutOfMemory;
        return nullptr;
    }
    if (s.bytes >= bytes)
        return s.p;
    // Work already queued (on any of the context's streams) may still use
    // the old buffer.
    if ((*e = sync_streams(c)) != hipSuccess)
        return nullptr;
    size_t nb = std::max(bytes, s.bytes * 2);
    nb = (nb + 4095) & ~size_t(4095);
    if (s.p)
        (void)hipFree(s.p);
    s.p = nullptr;
    s.bytes = 0;
    *e = hipMalloc(&s.p, nb);
    if (*e != hipSuccess) {
        s.p = nullptr;
        return nullptr;
    }
    s.bytes = nb;
    return s.p;
}

hipError_t join_selection(dm_ctx* c)
{
    if (!c->pipelined || c->batches == 0)
        return hipSuccess;
    return hipStreamWaitEvent(c->stream, c->out_done[(c->batches - 1) & 1], 0);
}

// Host checks shared by both routing entry points (what = the caller's name).
dm_status route_args_check(dm_ctx* c, const int32_t* tokens, uint64_t n_tokens,
                           const int64_t* offsets, uint64_t n, int64_t* loads,
                           const dm_route_out* out, const char* what)
{
    if (c->n_live == 0)
        return fail(c, DM_ESTATE, std::string(what) + ": rings not built");
    if (n == 0)
        return DM_OK;
    if ((!tokens && n_tokens) || !offsets || !loads || !out || !out->key || !out->cand ||
        !out->match || !out->chosen || !out->ttft_us || !out->flags)
        return fail(c, DM_EINVAL, std::string(what) + ": null argument");
    if (!aligned(tokens) || !aligned(offsets) || !aligned(loads) || !aligned(out->key) ||
        !aligned(out->cand) || !aligned(out->match) || !aligned(out->chosen) ||
        !aligned(out->ttft_us) || (out->block_keys && !aligned(out->block_keys)) ||
        (out->key_len && !aligned(out->key_len)))
        return fail(c, DM_EINVAL, std::string(what) + ": misaligned pointer");

    // the selection's slot indices are 32-bit: 66 windows of two sets of 64
    // lanes per 2048 requests must stay below 2^32
    if (n > kMaxRouteBatch)
        return fail(c, DM_EINVAL, std::string(what) + ": batch too large (n <= 1,041,203,200)");
    if (n_tokens > (1ull << 62))
        return fail(c, DM_EINVAL, std::string(what) + ": token count too large");
    return DM_OK;
}

}  // namespace dm

namespace {

// Makes ctx's device current for the duration of a call.
struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess)
            prev = -1;
        if (prev != dev)
            ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard()
    {
        int now = -1;
        if (prev >= 0 && hipGetDevice(&now) == hipSuccess && now != prev)
            hipSetDevice(prev);
    }
};

bool is_pow2(uint64_t x) { return x && !(x & (x - 1)); }

uint32_t log2u(uint64_t x)
{
    uint32_t k = 0;
    while ((1ull << k) < x)
        k++;
    return k;
}

uint64_t sm_next(uint64_t& st)
{
    st += 0x9E3779B97F4A7C15ull;
    return mix64(st);
}

// Per-function hash parameters: B key words, odd multiplier P, chain start,
// then the modular inverse of P and the lane power tables.
void make_params(HashParams& hp, const dm_config& cfg)
{
    std::memset(&hp, 0, sizeof(hp));
    for (int s = 0; s < 2; s++) {
        uint64_t st = cfg.seed[s];
        hp.seed[s] = cfg.seed[s];
        for (uint32_t j = 0; j < cfg.block_size; j++)
            hp.kk[s][j] = (uint32_t)sm_next(st);
        const uint64_t P = sm_next(st) | 1ull;
        hp.P[s] = P;
        hp.H0[s] = sm_next(st);
        uint64_t x = P;  // Newton iteration for P^-1 mod 2^64 (3 -> 96 bits)
        for (int it = 0; it < 5; it++)
            x *= 2 - P * x;
        hp.Q[s] = x;
        uint64_t pp = 1, qq = 1;
        for (int l = 0; l < kWave; l++) {
            pp *= P;
            qq *= x;
            hp.ppow[s][l] = pp;
            hp.qpow[s][l] = qq;
        }
    }
}


hipError_t upload_live(dm_ctx* c)
{
    const uint32_t S = c->cfg.max_slots;
    std::vector<uint32_t> ids, nxt(S, 0), dense(S, 0);
    for (uint32_t i = 0; i < S; i++)
        if (c->live[i])
            ids.push_back(i);
    for (size_t k = 0; k < ids.size(); k++) {
        nxt[ids[k]] = ids[(k + 1) % ids.size()];
        dense[ids[k]] = (uint32_t)k;
    }
    ids.resize(S, 0);
    hipError_t e = hipMemcpyAsync(c->d_live_ids, ids.data(), S * sizeof(uint32_t),
                                  hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->d_next_live, nxt.data(), S * sizeof(uint32_t),
                           hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->d_dense, dense.data(), S * sizeof(uint32_t), hipMemcpyHostToDevice,
                           c->stream);
    if (e == hipSuccess)
        e = hipStreamSynchronize(c->stream);  // host vectors go out of scope
    return e;
}

void free_ring(dm::Ring& r)
{
    (void)hipFree(r.pos);
    (void)hipFree(r.id);
    (void)hipFree(r.dir);
    r = dm::Ring{};
}

}  // namespace

extern "C" {

dm_status dm_create(const dm_config* cfg, void* hip_stream, dm_ctx** out)
{
    if (!cfg || !out)
        return DM_EINVAL;
    const dm_config& k = *cfg;
    if (!is_pow2(k.block_size) || k.block_size < 4 || k.block_size > 64 || k.key_blocks < 1 ||
        k.key_blocks > 64 || k.vnodes < 1 || k.vnodes > (1u << 20) || k.max_slots < 1 ||
        k.max_slots > kMaxSlots || k.index_log2_slots < 4 || k.index_log2_slots > 30 ||
        k.reserved != 0 || k.queue_div < 1 || !is_pow2((uint64_t)k.queue_div))
        return DM_EINVAL;
    dm_ctx* c = new (std::nothrow) dm_ctx();
    if (!c)
        return DM_ENOMEM;
    c->cfg = k;
    c->stream = static_cast<hipStream_t>(hip_stream);
    c->home_stream = c->stream;
    c->shift_div = log2u((uint64_t)k.queue_div);
    c->live.assign(k.max_slots, 0);
    make_params(c->hp, k);
    hipError_t e = hipGetDevice(&c->device);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device);
    const size_t S = k.max_slots;
    const size_t table_slots = S << k.index_log2_slots;
    if (e == hipSuccess) e = hipMalloc(&c->d_hp, sizeof(HashParams));
    if (e == hipSuccess) e = hipMalloc(&c->d_next_live, S * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(&c->d_live_ids, S * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(&c->d_dense, S * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(&c->d_flag_add, S);
    if (e == hipSuccess) e = hipMalloc(&c->d_flag_rm, S);
    if (e == hipSuccess) e = hipMalloc(&c->d_tables, table_slots * sizeof(uint64_t));
    if (e == hipSuccess) e = hipMalloc(&c->d_counts, 2 * S * sizeof(uint64_t));
    if (e == hipSuccess) e = hipMalloc(&c->d_status, sizeof(uint32_t));
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->d_hp, &c->hp, sizeof(HashParams), hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess)
        e = hipMemsetAsync(c->d_tables, 0, table_slots * sizeof(uint64_t), c->stream);
    if (e == hipSuccess) e = hipMemsetAsync(c->d_counts, 0, 2 * S * sizeof(uint64_t), c->stream);
    if (e == hipSuccess) e = hipMemsetAsync(c->d_status, 0, sizeof(uint32_t), c->stream);
    if (e == hipSuccess) e = hipMemsetAsync(c->d_next_live, 0, S * sizeof(uint32_t), c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    // the static work area of allocation-free routing on this device; if it
    // cannot be found, that entry point reports DM_EDEVICE and nothing else
    // is affected
    if (e == hipSuccess && noalloc_attach(c) != hipSuccess)
        (void)hipGetLastError();
    if (e != hipSuccess) {
        dm_status s = (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) ? DM_ENOMEM
                                                                                   : DM_EDEVICE;
        dm_destroy(c);
        return s;
    }
    *out = c;
    return DM_OK;
}

void dm_destroy(dm_ctx* c)
{
    if (!c)
        return;
    DeviceGuard g(c->device);
    (void)hipStreamSynchronize(c->stream);
    for (hipStream_t s : {c->work_stream, c->sel_stream, c->out_stream})
        if (s)
            (void)hipStreamSynchronize(s);
    for (auto& b : c->ring)
        for (auto& r : b)
            free_ring(r);
    for (auto& s : c->scratch)
        (void)hipFree(s.p);
    keylen_free(c);
    kv_free(c);
    for (auto& ev : c->tev)
        if (ev)
            (void)hipEventDestroy(ev);
    for (hipEvent_t ev : {c->in_ready, c->prep_done, c->sel_done, c->out_done[0], c->out_done[1]})
        if (ev)
            (void)hipEventDestroy(ev);
    for (hipStream_t s : {c->work_stream, c->sel_stream, c->out_stream})
        if (s)
            (void)hipStreamDestroy(s);
    (void)hipFree(c->d_hp);
    (void)hipFree(c->d_next_live);
    (void)hipFree(c->d_live_ids);
    (void)hipFree(c->d_dense);
    (void)hipFree(c->d_flag_add);
    (void)hipFree(c->d_flag_rm);
    (void)hipFree(c->d_tables);
    (void)hipFree(c->d_counts);
    (void)hipFree(c->d_status);
    delete c;
}

dm_status dm_build_rings(dm_ctx* c, const uint32_t* ids, uint32_t n)
{
    if (!c)
        return DM_EINVAL;
    if (!ids || n == 0)
        return fail(c, DM_EINVAL, "dm_build_rings: need at least one instance id");
    std::vector<uint8_t> seen(c->cfg.max_slots, 0);
    for (uint32_t i = 0; i < n; i++) {
        if (ids[i] >= c->cfg.max_slots)
            return fail(c, DM_EINVAL, "dm_build_rings: id out of range");
        if (seen[ids[i]])
            return fail(c, DM_EINVAL, "dm_build_rings: duplicate id");
        seen[ids[i]] = 1;
    }
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_build_rings");
    c->live = seen;
    c->n_live = n;
    hipError_t e = upload_live(c);
    for (int s = 0; s < 2 && e == hipSuccess; s++)
        e = ring_build(c, c->ring[c->cur][s], s, c->d_live_ids, n);
    if (e != hipSuccess) {
        c->n_live = 0;
        return hip_fail(c, e, "dm_build_rings");
    }
    return DM_OK;
}

dm_status dm_ring_export(dm_ctx* c, int s, uint64_t* pos, uint32_t* id, uint64_t cap,
                         uint64_t* len)
{
    if (!c || s < 0 || s > 1 || !len)
        return fail(c, DM_EINVAL, "dm_ring_export: bad arguments");
    const Ring& r = c->ring[c->cur][s];
    *len = c->n_live ? r.len : 0;
    if (!pos && !id)
        return DM_OK;
    if (cap < *len)
        return fail(c, DM_EINVAL, "dm_ring_export: output too small");
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_ring_export");
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess && pos && *len)
        e = hipMemcpy(pos, r.pos, *len * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e == hipSuccess && id && *len)
        e = hipMemcpy(id, r.id, *len * sizeof(uint32_t), hipMemcpyDeviceToHost);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_ring_export");
}

dm_status dm_index_insert(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n)
{
    if (!c)
        return DM_EINVAL;
    if (id >= c->cfg.max_slots || (n && (!keys || !aligned(keys))))
        return fail(c, DM_EINVAL, "dm_index_insert: bad id or key pointer");
    if (n == 0)
        return DM_OK;
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_index_insert");
    hipError_t e = index_insert(c, id, keys, n);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_index_insert");
}

dm_status dm_index_erase(dm_ctx* c, uint32_t id, const uint64_t* keys, uint64_t n)
{
    if (!c)
        return DM_EINVAL;
    if (id >= c->cfg.max_slots || (n && (!keys || !aligned(keys))))
        return fail(c, DM_EINVAL, "dm_index_erase: bad id or key pointer");
    if (n == 0)
        return DM_OK;
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_index_erase");
    hipError_t e = index_erase(c, id, keys, n);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_index_erase");
}

dm_status dm_index_clear(dm_ctx* c, uint32_t id)
{
    if (!c)
        return DM_EINVAL;
    if (id >= c->cfg.max_slots)
        return fail(c, DM_EINVAL, "dm_index_clear: bad id");
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_index_clear");
    hipError_t e = index_clear(c, id);
    if (e == hipSuccess && c->kv.n) {
        // the saved-key record of the emptied cache goes with it
        std::vector<uint8_t> gone(c->cfg.max_slots, 0);
        gone[id] = 1;
        if ((e = hipMemcpy(c->d_flag_add, gone.data(), gone.size(), hipMemcpyHostToDevice)) ==
            hipSuccess)
            e = kv_forget(c, c->d_flag_add);
    }
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_index_clear");
}

// Host checks shared by the queue operations.
static dm_status queue_args(dm_ctx* c, const dm_queues* q, const dm_queue_out* out,
                            const char* what)
{
    if (!q || !out || !q->qoff || !q->base_work || !out->qoff || !out->base_work)
        return fail(c, DM_EINVAL, std::string(what) + ": null argument");
    if (out->cap && (!out->rec_id || !out->unc_here || !out->alt || !out->unc_alt))
        return fail(c, DM_EINVAL, std::string(what) + ": null output array");
    if (!aligned(q->qoff) || !aligned(q->base_work) || !aligned(out->qoff) ||
        !aligned(out->base_work) || !aligned(q->rec_id) || !aligned(out->rec_id))
        return fail(c, DM_EINVAL, std::string(what) + ": misaligned pointer");
    const void* in_p[] = {q->qoff, q->rec_id, q->unc_here, q->alt, q->unc_alt, q->base_work};
    const void* out_p[] = {out->qoff, out->rec_id, out->unc_here, out->alt, out->unc_alt,
                           out->base_work};
    for (const void* a : in_p)
        for (const void* b : out_p)
            if (a && a == b)
                return fail(c, DM_EINVAL, std::string(what) + ": output aliases the input");
    return DM_OK;
}

dm_status dm_queue_append(dm_ctx* c, const dm_queues* q, const int64_t* offsets, uint64_t n,
                          const dm_route_out* routed, uint64_t rec_base, const dm_queue_out* out)
{
    if (!c)
        return DM_EINVAL;
    if (dm_status s = queue_args(c, q, out, "dm_queue_append"); s != DM_OK)
        return s;
    if (n && (!offsets || !routed || !routed->cand || !routed->match || !routed->chosen))
        return fail(c, DM_EINVAL, "dm_queue_append: null batch argument");
    if (n >= (1ull << 32))
        return fail(c, DM_EINVAL, "dm_queue_append: batch too large");
    DeviceGuard g(c->device);
    return queue_append(c, q, offsets, n, routed, rec_base, out);
}

dm_status dm_queue_migrate(dm_ctx* c, const dm_queues* q, const uint64_t* rec_id,
                           const uint32_t* from, const uint32_t* to, uint64_t m,
                           const dm_queue_out* out)
{
    if (!c)
        return DM_EINVAL;
    if (dm_status s = queue_args(c, q, out, "dm_queue_migrate"); s != DM_OK)
        return s;
    if (m && (!rec_id || !from || !to))
        return fail(c, DM_EINVAL, "dm_queue_migrate: null migration array");
    DeviceGuard g(c->device);
    return queue_migrate(c, q, rec_id, from, to, m, out);
}

dm_status dm_queue_drain(dm_ctx* c, const dm_queues* q, const int64_t* units,
                         const dm_queue_out* out)
{
    if (!c)
        return DM_EINVAL;
    if (dm_status s = queue_args(c, q, out, "dm_queue_drain"); s != DM_OK)
        return s;
    if (!units || !aligned(units))
        return fail(c, DM_EINVAL, "dm_queue_drain: null or misaligned units");
    DeviceGuard g(c->device);
    return queue_drain(c, q, units, out);
}

dm_status dm_queue_reprobe(dm_ctx* c, const dm_queues* q, const int64_t* chain_off,
                           const uint64_t* chain_keys, uint64_t n_keys, const int64_t* prompt_len,
                           uint64_t n_ids, const dm_queue_out* out)
{
    if (!c)
        return DM_EINVAL;
    if (dm_status s = queue_args(c, q, out, "dm_queue_reprobe"); s != DM_OK)
        return s;
    if (!q->alt && out->cap)
        return fail(c, DM_EINVAL, "dm_queue_reprobe: null alt array");
    DeviceGuard g(c->device);
    return queue_reprobe(c, q, chain_off, chain_keys, n_keys, prompt_len, n_ids, out);
}

dm_status dm_kv_save(dm_ctx* c, const int64_t* offsets, uint64_t n, const uint64_t* block_keys,
                     const uint32_t* inst, uint64_t clock, uint64_t cap, uint64_t* added_host,
                     uint64_t* removed_host)
{
    if (!c)
        return DM_EINVAL;
    if (c->n_live == 0)
        return fail(c, DM_ESTATE, "dm_kv_save: rings not built");
    if (n && (!offsets || !inst))
        return fail(c, DM_EINVAL, "dm_kv_save: null argument");
    if (!aligned(offsets) || !aligned(block_keys) || !aligned(inst))
        return fail(c, DM_EINVAL, "dm_kv_save: misaligned pointer");
    if (cap > (1ull << (c->cfg.index_log2_slots - 1)))
        return fail(c, DM_EINVAL, "dm_kv_save: cap past the index's load limit");
    if (n >= (1ull << 32))
        return fail(c, DM_EINVAL, "dm_kv_save: batch too large");
    DeviceGuard g(c->device);
    return kv_save(c, offsets, n, block_keys, inst, clock, cap, added_host, removed_host);
}

dm_status dm_index_size(dm_ctx* c, uint32_t id, uint64_t* n_host)
{
    if (!c)
        return DM_EINVAL;
    if (id >= c->cfg.max_slots || !n_host)
        return fail(c, DM_EINVAL, "dm_index_size: bad arguments");
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_index_size");
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess)
        e = hipMemcpy(n_host, c->d_counts + id, sizeof(uint64_t), hipMemcpyDeviceToHost);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_index_size");
}

dm_status dm_route_batch(dm_ctx* c, const int32_t* tokens, uint64_t n_tokens,
                         const int64_t* offsets, uint64_t n, int64_t* loads,
                         const dm_route_out* out)
{
    if (!c)
        return DM_EINVAL;
    if (dm_status st = route_args_check(c, tokens, n_tokens, offsets, n, loads, out,
                                        "dm_route_batch");
        st != DM_OK || n == 0)
        return st;
    DeviceGuard g(c->device);
    hipError_t e = route(c, tokens, n_tokens, offsets, n, loads, out);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_route_batch");
}

dm_status dm_rebalance(dm_ctx* c, const dm_queues* q, int64_t* loads_out,
                       const dm_migrations* out, uint64_t cap)
{
    if (!c)
        return DM_EINVAL;
    if (!q || !q->qoff || !q->base_work || !loads_out || !out || !out->count)
        return fail(c, DM_EINVAL, "dm_rebalance: null argument");
    if (cap && (!out->rec_id || !out->from || !out->to || !out->benefit_us || !out->ttft_to_us))
        return fail(c, DM_EINVAL, "dm_rebalance: null migration array");
    if (!aligned(q->qoff) || !aligned(q->base_work) || !aligned(loads_out) ||
        !aligned(out->count) || (q->prefill_interval && !aligned(q->prefill_interval)))
        return fail(c, DM_EINVAL, "dm_rebalance: misaligned pointer");
    if (q->prefill_interval && q->decode_threshold_us < 0)
        return fail(c, DM_EINVAL, "dm_rebalance: negative decode threshold");
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_rebalance");
    // The record count sizes the work arrays: read qoff[max_slots].
    int64_t Qs = 0, q0 = 0;
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess)
        e = hipMemcpy(&Qs, q->qoff + c->cfg.max_slots, sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e == hipSuccess)
        e = hipMemcpy(&q0, q->qoff, sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_rebalance");
    if (q0 != 0 || Qs < 0 || Qs >= (1ll << 32))
        return fail(c, DM_EINVAL, "dm_rebalance: qoff[0] must be 0 and the record count < 2^32");
    if (Qs && (!q->rec_id || !q->unc_here || !q->alt || !q->unc_alt))
        return fail(c, DM_EINVAL, "dm_rebalance: null record array");
    e = rebalance(c, q, loads_out, out, cap, (uint64_t)Qs);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_rebalance");
}

dm_status dm_scale(dm_ctx* c, const uint32_t* add, uint32_t n_add, const uint32_t* rm,
                   uint32_t n_rm, const uint64_t* keys, uint64_t n, uint32_t* old_owner,
                   uint32_t* new_owner, uint64_t* moved, uint64_t* violations)
{
    if (!c)
        return DM_EINVAL;
    if (c->n_live == 0)
        return fail(c, DM_ESTATE, "dm_scale: rings not built");
    if ((n_add && !add) || (n_rm && !rm) || !moved || !violations ||
        (n && (!keys || !old_owner || !new_owner)))
        return fail(c, DM_EINVAL, "dm_scale: null argument");
    if (!aligned(moved) || !aligned(violations) || (n && (!aligned(keys) || !aligned(old_owner) ||
                                                          !aligned(new_owner))))
        return fail(c, DM_EINVAL, "dm_scale: misaligned pointer");
    const uint32_t S = c->cfg.max_slots;
    std::vector<uint8_t> fa(S, 0), fr(S, 0);
    for (uint32_t k = 0; k < n_add; k++) {
        if (add[k] >= S || c->live[add[k]] || fa[add[k]])
            return fail(c, DM_EINVAL, "dm_scale: added id is live, repeated or out of range");
        fa[add[k]] = 1;
    }
    for (uint32_t k = 0; k < n_rm; k++) {
        if (rm[k] >= S || !c->live[rm[k]] || fr[rm[k]])
            return fail(c, DM_EINVAL, "dm_scale: removed id is not live or repeated");
        fr[rm[k]] = 1;
    }
    if (c->n_live - n_rm + n_add == 0)
        return fail(c, DM_EINVAL, "dm_scale: no instance would remain");
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_scale");
    std::vector<uint8_t> live = c->live;
    for (uint32_t i = 0; i < S; i++)
        live[i] = (live[i] && !fr[i]) || fa[i];
    const std::vector<uint8_t> old_live = c->live;
    const uint32_t old_n = c->n_live;
    c->live = live;
    c->n_live = old_n - n_rm + n_add;
    hipError_t e = upload_live(c);
    if (e == hipSuccess)
        e = hipMemcpy(c->d_flag_add, fa.data(), S, hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(c->d_flag_rm, fr.data(), S, hipMemcpyHostToDevice);
    const int nb = 1 - c->cur;
    for (int s = 0; s < 2 && e == hipSuccess; s++)
        e = ring_build(c, c->ring[nb][s], s, c->d_live_ids, c->n_live);
    if (e == hipSuccess)
        e = ring_remap(c, c->ring[c->cur], c->ring[nb], keys, n, old_owner, new_owner, moved,
                       violations);
    if (e == hipSuccess) {
        std::vector<uint32_t> changed;
        for (uint32_t i = 0; i < S; i++)
            if (fa[i] || fr[i])
                changed.push_back(i);
        e = index_clear_many(c, changed.data(), (uint32_t)changed.size());
        if (e == hipSuccess && c->kv.n) {
            // the saved-key record of the emptied caches goes with them
            std::vector<uint8_t> gone(S, 0);
            for (uint32_t i : changed)
                gone[i] = 1;
            if ((e = hipMemcpy(c->d_flag_add, gone.data(), S, hipMemcpyHostToDevice)) ==
                hipSuccess)
                e = kv_forget(c, c->d_flag_add);
        }
    }
    if (e != hipSuccess) {
        c->live = old_live;
        c->n_live = old_n;
        (void)upload_live(c);
        return hip_fail(c, e, "dm_scale");
    }
    c->cur = nb;
    return DM_OK;
}

dm_status dm_set_timing(dm_ctx* c, int on)
{
    if (!c)
        return DM_EINVAL;
    DeviceGuard g(c->device);
    if (on && c->tev.empty()) {
        c->tev.assign(dm_ctx::kTimingRing * 5, nullptr);
        for (auto& ev : c->tev) {
            hipError_t e = hipEventCreate(&ev);
            if (e != hipSuccess)
                return hip_fail(c, e, "dm_set_timing");
        }
    }
    c->timing = on != 0;
    c->tcount = 0;
    return DM_OK;
}

dm_status dm_route_stage_ms(dm_ctx* c, float* ms, int n)
{
    if (!c)
        return DM_EINVAL;
    if (!ms || n < 1)
        return fail(c, DM_EINVAL, "dm_route_stage_ms: bad output");
    if (!c->timing || c->tev.empty() || c->tcount == 0)
        return fail(c, DM_ESTATE, "dm_route_stage_ms: timing is off or no batch was timed");
    DeviceGuard g(c->device);
    const uint64_t R = dm_ctx::kTimingRing;
    const uint64_t nrec = c->tcount < R ? c->tcount : R;
    // the last batch's selection ends after every earlier recorded event
    hipError_t e = hipEventSynchronize(c->tev[((c->tcount - 1) % R) * 5 + 4]);
    double t[4] = {0, 0, 0, 0};
    for (uint64_t b = c->tcount - nrec; b < c->tcount && e == hipSuccess; b++) {
        hipEvent_t* ev = &c->tev[(b % R) * 5];
        float x[4] = {0, 0, 0, 0};
        if (e == hipSuccess) e = hipEventElapsedTime(&x[0], ev[1], ev[2]);
        if (e == hipSuccess) e = hipEventElapsedTime(&x[1], ev[2], ev[3]);
        if (e == hipSuccess) e = hipEventElapsedTime(&x[2], ev[3], ev[4]);
        if (e == hipSuccess) e = hipEventElapsedTime(&x[3], ev[0], ev[1]);
        for (int k = 0; k < 4; k++)
            t[k] += x[k];
    }
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_route_stage_ms");
    for (int k = 0; k < n && k < 4; k++)
        ms[k] = (float)(t[k] / (double)nrec);
    return DM_OK;
}

// Streams of pipelined routing: the serial selection gets one compute unit
// of its own and the work and output streams all the others, so that the
// next batches' kernels never share the selection's unit.  Without CU
// masks (a runtime that refuses them), plain streams are used.
static hipError_t make_streams(dm_ctx* c)
{
    int cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, c->device);
    if (e != hipSuccess)
        return e;
    std::vector<uint32_t> one((cus + 31) / 32, 0u), rest((cus + 31) / 32, 0u);
    for (int i = 0; i < cus; i++)
        (i == 0 ? one : rest)[i / 32] |= 1u << (i % 32);
    const bool masked = cus >= 2 &&
        hipExtStreamCreateWithCUMask(&c->sel_stream, (uint32_t)one.size(), one.data()) == hipSuccess &&
        hipExtStreamCreateWithCUMask(&c->work_stream, (uint32_t)rest.size(), rest.data()) == hipSuccess &&
        hipExtStreamCreateWithCUMask(&c->out_stream, (uint32_t)rest.size(), rest.data()) == hipSuccess;
    if (!masked) {
        for (hipStream_t* s : {&c->work_stream, &c->sel_stream, &c->out_stream}) {
            if (*s)
                (void)hipStreamDestroy(*s);
            *s = nullptr;
        }
        (void)hipGetLastError();
        for (hipStream_t* s : {&c->work_stream, &c->sel_stream, &c->out_stream})
            if (e == hipSuccess)
                e = hipStreamCreateWithFlags(s, hipStreamNonBlocking);
    }
    for (hipEvent_t* ev : {&c->in_ready, &c->prep_done, &c->sel_done, &c->out_done[0], &c->out_done[1]})
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
    return e;
}

dm_status dm_keylen_enable(dm_ctx* c, uint64_t max_nodes, uint64_t max_window_blocks)
{
    if (!c)
        return DM_EINVAL;
    DeviceGuard g(c->device);
    return keylen_enable(c, max_nodes, max_window_blocks);
}

dm_status dm_keylen_window(dm_ctx* c)
{
    if (!c)
        return DM_EINVAL;
    DeviceGuard g(c->device);
    return keylen_window(c);
}

dm_status dm_keylen_export(dm_ctx* c, uint64_t* keys_host, uint64_t cap, uint64_t* n_host)
{
    if (!c)
        return DM_EINVAL;
    if (!n_host || (cap && !keys_host))
        return fail(c, DM_EINVAL, "dm_keylen_export: null argument");
    DeviceGuard g(c->device);
    return keylen_export(c, keys_host, cap, n_host);
}

dm_status dm_set_policy(dm_ctx* c, int policy)
{
    if (!c)
        return DM_EINVAL;
    if (policy < DM_POLICY_SLO_AWARE || policy > DM_POLICY_MIN_TTFT)
        return fail(c, DM_EINVAL, "dm_set_policy: unknown selection rule");
    c->policy = (uint32_t)policy;
    return DM_OK;
}

dm_status dm_set_pipelining(dm_ctx* c, int on)
{
    if (!c)
        return DM_EINVAL;
    DeviceGuard g(c->device);
    hipError_t e = hipSuccess;
    if (on && !c->sel_stream && (e = make_streams(c)) != hipSuccess)
        return hip_fail(c, e, "dm_set_pipelining");
    // later work on the context's stream follows the last pipelined batch
    if ((e = join_selection(c)) != hipSuccess)
        return hip_fail(c, e, "dm_set_pipelining");
    c->pipelined = on != 0;
    c->batches = 0;
    return DM_OK;
}

dm_status dm_sync(dm_ctx* c)
{
    if (!c)
        return DM_EINVAL;
    DeviceGuard g(c->device);
    if (hipError_t je = join_selection(c); je != hipSuccess)
        return hip_fail(c, je, "dm_sync");
    hipError_t e = hipStreamSynchronize(c->stream);
    uint32_t st = 0;
    if (e == hipSuccess)
        e = hipMemcpy(&st, c->d_status, sizeof(uint32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess)
        return hip_fail(c, e, "dm_sync");
    if (st) {
        uint32_t zero = 0;
        e = hipMemcpy(c->d_status, &zero, sizeof(uint32_t), hipMemcpyHostToDevice);
        if (e != hipSuccess)
            return hip_fail(c, e, "dm_sync");
        if (st & kErrInval)
            return fail(c, DM_EINVAL, "device: malformed input (offsets or queue records)");
        return fail(c, DM_EFULL, "device: index table full or migration list over capacity");
    }
    return DM_OK;
}

const char* dm_last_error(const dm_ctx* c) { return c ? c->err.c_str() : "null context"; }

}  // extern "C"
