// debug.hip -- optional device-side precondition check (TS_DEBUG=1).
//
// The fast path never reads ctx_lens, q_lens or the page table on the host.
// When debugging, one block scans them (and the workspace's split counters,
// which must be zero between calls) on the device, sets bits in a flag word
// that lives in the call's own workspace (so concurrent calls with their own
// workspaces cannot see each other's flags), and the host synchronises and
// reports the first class of violation.
#include <hip/hip_runtime.h>

#include "attn_common.h"
#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {

namespace {

enum : int {
    kBadQLen = 1,      // q_len < 0, > max_q_len or > ctx_len
    kBadCtx = 2,       // ctx_len < 1 with q_len > 0, > max_ctx_len, or > max_pages * 16
    kBadPage = 4,      // referenced page id outside [0, num_pages)
    kDirtyWs = 8,      // a split counter of the workspace is not zero
};

__global__ __launch_bounds__(256) void check_kernel(ts_attn_shape s, const int32_t *page_table,
                                                    const int32_t *ctx_lens, const int32_t *q_lens,
                                                    const int *counters, int *flags) {
    if (threadIdx.x == 0)
        *flags = 0;
    __syncthreads();
    int bad = 0;
    for (int b = threadIdx.x; b < s.num_seqs; b += blockDim.x) {
        const int L = ctx_lens[b], Q = q_lens[b];
        if (Q < 0 || Q > s.max_q_len || Q > L)
            bad |= kBadQLen;
        if ((Q > 0 && L < 1) || L > s.max_ctx_len || (int64_t)L > (int64_t)s.max_pages_per_seq * 16)
            bad |= kBadCtx;
        if (Q > 0 && L > 0 && (int64_t)L <= (int64_t)s.max_pages_per_seq * 16) {
            const int np = (L + 15) / 16;
            for (int j = 0; j < np; j++) {
                const int pid = page_table[(size_t)b * s.max_pages_per_seq + j];
                if (pid < 0 || (int64_t)pid >= s.num_pages)
                    bad |= kBadPage;
            }
        }
    }
    for (int u = threadIdx.x; u < (int)(kCounterBytes / sizeof(int)); u += blockDim.x)
        if (counters[u] != 0)
            bad |= kDirtyWs;
    if (bad)
        atomicOr(flags, bad);
}

}  // namespace

int debug_check(const ts_attn_shape *s, const int32_t *page_table, const int32_t *ctx_lens,
                const int32_t *q_lens, const int *counters, int *flags, hipStream_t stream) {
    hipError_t e;
    hipLaunchKernelGGL(check_kernel, dim3(1), dim3(256), 0, stream, *s, page_table, ctx_lens,
                       q_lens, counters, flags);
    if ((e = hipGetLastError()) != hipSuccess)
        return hip_fail(e, "debug check launch");
    int host = 0;
    if ((e = hipMemcpyAsync(&host, flags, sizeof host, hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return hip_fail(e, "hipMemcpyAsync(debug flags)");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    if (host & kBadQLen)
        return fail(TS_ERR_SHAPE, "TS_DEBUG: some q_lens[b] outside [0, min(max_q_len, ctx_lens[b])]");
    if (host & kBadCtx)
        return fail(TS_ERR_SHAPE, "TS_DEBUG: some ctx_lens[b] outside [1, max_ctx_len] or beyond the page table");
    if (host & kBadPage)
        return fail(TS_ERR_SHAPE, "TS_DEBUG: a referenced page id is outside [0, num_pages)");
    if (host & kDirtyWs)
        return fail(TS_ERR_WORKSPACE, "TS_DEBUG: workspace split counters are not zero "
                                      "(zero-fill a workspace before its first use)");
    return TS_OK;
}

}  // namespace tsattn
