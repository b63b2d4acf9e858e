// wsk_decode_step_noalloc: the decode step with its chunk-partial workspace
// in a file-scope device array instead of a caller-provided buffer, for
// callers that cannot allocate device memory.
//
// The array lives in the library's code object, so every GPU the library
// runs on holds its own copy, at its own address, until the process ends.
// Host code never uses the array's name as an address (on the host it is a
// stand-in, not device memory): the device address is resolved once per
// device with hipGetSymbolAddress, with that device current, and kept.

#include <hip/hip_runtime.h>

#include <mutex>

#include "cache.h"

namespace wsk {
namespace {

static __device__ __align__(256) unsigned char scratch[WSK_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};   // device address of `scratch` per device, once resolved

}  // namespace

// Device address of `scratch` on `device` (resolved on the first call for that
// device, with it current).  Returns WSK_OK or WSK_EHIP / WSK_EINVAL.
int noalloc_scratch(int device, void **out) {
    if (device < 0 || device >= kMaxDevices) return fail(WSK_EINVAL, "device %d outside 0..%d", device, kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        DeviceGuard guard(device);
        if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p || ((uintptr_t)p & 255)) return fail(WSK_EHIP, "scratch resolved to an unusable address");
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return WSK_OK;
}

}  // namespace wsk

extern "C" int wsk_decode_step_noalloc(wsk_cache *c, int32_t n, const int32_t *ids, const void *q,
                                       const void *k_new, const void *v_new, const float *o_x, const float *lse_x,
                                       float *o, float *lse, void *stream) {
    if (!c) return wsk::fail(WSK_EINVAL, "cache is NULL");
    if (c->device < 0) return wsk::fail(WSK_ESTATE, "host-only cache");
    size_t need = 0;
    int rc = wsk_decode_step_workspace(c, n, ids, &need);
    if (rc) return rc;
    if (need > (size_t)WSK_NOALLOC_SCRATCH_BYTES)
        return wsk::fail(WSK_ERANGE,
                         "this step needs %zu bytes of chunk partials; wsk_decode_step_noalloc holds at most %zu "
                         "(use wsk_decode_step with a workspace)",
                         need, (size_t)WSK_NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    rc = wsk::noalloc_scratch(c->device, &ws);
    if (rc) return rc;
    // pass 1 writes every chunk partial that pass 2 reads, so nothing in the
    // scratch has to start at zero
    return wsk_decode_step(c, n, ids, q, k_new, v_new, o_x, lse_x, o, lse, ws, (size_t)WSK_NOALLOC_SCRATCH_BYTES,
                           stream);
}
