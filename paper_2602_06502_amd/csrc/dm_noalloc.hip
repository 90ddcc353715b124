// dm_route_batch_noalloc: routing for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops).
//
// Its work arrays come from one fixed static device array per GPU instead of
// the context's growable scratch.  The array's device address is looked up
// once per device (dm_create, with that device current) and kept; host code
// never uses the array's name as an address.  A call first plans every
// stage's work array from n and n_tokens, rejects the batch if the plan
// does not fit, and only then launches, so a rejected call does nothing.
// Every call on one GPU shares that GPU's array: calls that overlap on one
// GPU (two contexts, two host threads, or streams that are not ordered)
// race on it.  Nothing in it has to start at zero: each stage clears what
// it needs with kernels of its own.
#include <mutex>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr size_t kNoAllocBytes = size_t(64) << 20;  // 64 MiB per GPU
constexpr int kMaxDevices = 64;

__device__ __align__(256) static unsigned char scratch[kNoAllocBytes];

std::mutex g_lock;
uint8_t* g_area[kMaxDevices] = {};  // device address of `scratch` per device

}  // namespace

size_t noalloc_capacity() { return kNoAllocBytes; }

hipError_t noalloc_attach(dm_ctx* c)
{
    if (c->device < 0 || c->device >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> g(g_lock);
    if (!g_area[c->device]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        g_area[c->device] = static_cast<uint8_t*>(ptr);
    }
    c->noalloc_area = g_area[c->device];
    return hipSuccess;
}

}  // namespace dm

using namespace dm;

extern "C" dm_status dm_route_batch_noalloc(dm_ctx* c, const int32_t* tokens, uint64_t n_tokens,
                                            const int64_t* offsets, uint64_t n, int64_t* loads,
                                            const dm_route_out* out)
{
    if (!c)
        return DM_EINVAL;
    if (dm_status st = route_args_check(c, tokens, n_tokens, offsets, n, loads, out,
                                        "dm_route_batch_noalloc");
        st != DM_OK || n == 0)
        return st;
    if (!c->noalloc_area)
        return fail(c, DM_EDEVICE, "dm_route_batch_noalloc: no static work area on this device");
    // Plan: each stage's region, 256-byte aligned, in slot order.
    size_t need[kScratchSlots];
    route_scratch_plan(c, n, n_tokens, out->block_keys == nullptr, need);
    Arena a;
    size_t used = 0;
    for (int i = 0; i < kScratchSlots; i++) {
        a.off[i] = used;
        a.len[i] = need[i];
        used += (need[i] + 255) & ~size_t(255);
    }
    if (used > kNoAllocBytes)
        return fail(c, DM_EINVAL,
                    "dm_route_batch_noalloc: the batch needs " + std::to_string(used) +
                        " bytes of work area; the static area holds " +
                        std::to_string(kNoAllocBytes) + " (use dm_route_batch)");
    int prev = -1;
    if (hipGetDevice(&prev) != hipSuccess)
        prev = -1;
    if (prev != c->device && hipSetDevice(c->device) != hipSuccess)
        return fail(c, DM_EDEVICE, "dm_route_batch_noalloc: cannot select the context's device");
    // Unpipelined on the context's stream, after any pipelined batch.
    hipError_t e = join_selection(c);
    const bool pipe = c->pipelined;
    if (e == hipSuccess) {
        a.base = c->noalloc_area;
        a.on = true;
        c->arena = a;
        c->pipelined = false;
        e = route(c, tokens, n_tokens, offsets, n, loads, out);
        c->pipelined = pipe;
        c->arena = Arena{};
    }
    if (prev >= 0 && prev != c->device)
        (void)hipSetDevice(prev);
    return e == hipSuccess ? DM_OK : hip_fail(c, e, "dm_route_batch_noalloc");
}
