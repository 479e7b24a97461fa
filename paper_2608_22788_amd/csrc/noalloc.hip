// noalloc.hip -- ts_decode_attn_noalloc: ts_decode_attn for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops).
//
// The split partials, the arrival counters of the in-kernel combine and the
// TS_DEBUG flag word go to `scratch`, a file-scope device array of
// kScratchBytes that every GPU the library runs on holds until the process
// ends.  In host code `scratch` names a host-side stand-in, not a device
// address, so its address on each device is looked up once, with that device
// current, and only that address is handed to kernels.  Every call on one GPU
// shares that GPU's array, so calls that overlap on one GPU race.  The array
// has static storage and starts zeroed; the arrival counters of the in-kernel
// combine (its first 1 MiB) are the only part that must start at zero, and
// every call leaves them zero again (the last arriver of each unit resets its
// counter), exactly as a zero-filled caller workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {

namespace {

constexpr size_t kScratchBytes = TS_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device, once looked up

// The current device's address of `scratch` (looked up on its first use).
int scratch_address(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(TS_ERR_UNSUPPORTED, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p)
            return fail(TS_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return TS_OK;
}

}  // namespace

}  // namespace tsattn

using namespace tsattn;

extern "C" int ts_decode_attn_noalloc(const ts_attn_shape *shape, const void *q, const void *k_pages,
                                      const void *v_pages, const int32_t *page_table,
                                      const int32_t *ctx_lens, const int32_t *q_lens, void *out,
                                      float scale, void *stream) {
    try {
        clear_error();
        const size_t need = ts_decode_attn_workspace_size(shape);
        if (need == 0)
            return check_shape(shape);   // sets the message of the unsupported shape
        if (need > kScratchBytes)
            return fail(TS_ERR_WORKSPACE,
                        "this shape needs %zu bytes of scratch; ts_decode_attn_noalloc holds %zu "
                        "(use ts_decode_attn with a workspace, or fewer workers)",
                        need, kScratchBytes);
        int st = check_device();
        if (st)
            return st;
        void *ws = nullptr;
        st = scratch_address(&ws);
        if (st)
            return st;
        return launch_attn(shape, q, k_pages, v_pages, page_table, ctx_lens, q_lens, out, scale, ws,
                           kScratchBytes, stream, nullptr, nullptr);
    } catch (...) {
        return fail(TS_ERR_HIP, "unexpected C++ exception");
    }
}
