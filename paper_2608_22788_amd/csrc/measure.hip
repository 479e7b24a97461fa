// measure.hip -- measurement helpers: a plain copy kernel (to calibrate
// hardware byte counters against a transfer of known size) and thin wrappers
// over HIP events so callers can time the attention kernel on its own stream.
#include <hip/hip_runtime.h>

#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {
namespace {

__global__ __launch_bounds__(256) void copy_kernel(uint4 *dst, const uint4 *src, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

// Reads every 16-byte word once and folds it into one word per thread, so the
// loads cannot be dropped; the folds are written to `sink`.
__global__ __launch_bounds__(256) void read_kernel(const uint4 *src, int64_t n, uint32_t *sink) {
    uint32_t acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

}  // namespace
}  // namespace tsattn

using namespace tsattn;

extern "C" {

int ts_copy_bytes(void *dst, const void *src, size_t bytes, void *stream) {
    clear_error();
    if (!dst || !src)
        return fail(TS_ERR_NULL, "NULL pointer");
    if ((bytes & 15) || ((uintptr_t)dst & 15) || ((uintptr_t)src & 15))
        return fail(TS_ERR_ARG, "copy needs 16-byte sizes and alignment");
    int st = check_device();
    if (st)
        return st;
    const int64_t n = (int64_t)(bytes / 16);
    if (n == 0)
        return TS_OK;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 256 * 16)
        blocks = 256 * 16;
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0,
                       reinterpret_cast<hipStream_t>(stream), static_cast<uint4 *>(dst),
                       static_cast<const uint4 *>(src), n);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "copy launch");
}

int ts_stream_read(const void *src, size_t bytes, void *sink, size_t sink_bytes, void *stream) {
    clear_error();
    if (!src || !sink)
        return fail(TS_ERR_NULL, "NULL pointer");
    if ((bytes & 15) || ((uintptr_t)src & 15))
        return fail(TS_ERR_ARG, "stream read needs 16-byte sizes and alignment");
    const int64_t blocks = 256 * 8;
    if (sink_bytes < (size_t)blocks * 256 * sizeof(uint32_t))
        return fail(TS_ERR_ARG, "sink needs %lld bytes", (long long)(blocks * 256 * 4));
    int st = check_device();
    if (st)
        return st;
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)blocks), dim3(256), 0,
                       reinterpret_cast<hipStream_t>(stream), static_cast<const uint4 *>(src),
                       (int64_t)(bytes / 16), static_cast<uint32_t *>(sink));
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "stream read launch");
}

int ts_event_create(void **ev) {
    clear_error();
    if (!ev)
        return fail(TS_ERR_NULL, "ev is NULL");
    hipEvent_t h;
    hipError_t e = hipEventCreate(&h);
    if (e != hipSuccess)
        return hip_fail(e, "hipEventCreate");
    *ev = h;
    return TS_OK;
}

int ts_event_destroy(void *ev) {
    clear_error();
    if (!ev)
        return TS_OK;
    hipError_t e = hipEventDestroy(reinterpret_cast<hipEvent_t>(ev));
    return e == hipSuccess ? TS_OK : hip_fail(e, "hipEventDestroy");
}

int ts_event_record(void *ev, void *stream) {
    clear_error();
    if (!ev)
        return fail(TS_ERR_NULL, "ev is NULL");
    hipError_t e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev), reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? TS_OK : hip_fail(e, "hipEventRecord");
}

int ts_event_elapsed_ms(void *start, void *stop, float *ms) {
    clear_error();
    if (!start || !stop || !ms)
        return fail(TS_ERR_NULL, "NULL argument");
    hipError_t e = hipEventSynchronize(reinterpret_cast<hipEvent_t>(stop));
    if (e != hipSuccess)
        return hip_fail(e, "hipEventSynchronize");
    e = hipEventElapsedTime(ms, reinterpret_cast<hipEvent_t>(start), reinterpret_cast<hipEvent_t>(stop));
    return e == hipSuccess ? TS_OK : hip_fail(e, "hipEventElapsedTime");
}

}  // extern "C"
