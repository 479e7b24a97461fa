// measure.hip -- measurement helpers: a plain copy kernel (to calibrate
// hardware byte counters against a transfer of known size), two read-only
// kernels that give the bandwidth ceilings the attention kernels are compared
// with, and thin wrappers over HIP events so callers can time a kernel on its
// own stream.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "attn_common.h"
#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {
namespace {

__global__ __launch_bounds__(256) void copy_kernel(uint4 *dst, const uint4 *src, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

__device__ __forceinline__ uint32_t fold(u32x4_t v) { return v.x ^ v.y ^ v.z ^ v.w; }

// Reads every 16-byte word once and folds it into one word per thread, so the
// loads cannot be dropped; the folds are written to `sink`.  The grid sweeps
// the buffer front to back: in step k block b reads the contiguous tile
// k * gridDim.x + b of kReadThreads * kReadBatch words, every lane keeping
// kReadBatch non-temporal loads in flight.
constexpr int kReadThreads = 256;
constexpr int kReadBatch = 8;

__global__ __launch_bounds__(kReadThreads) void read_kernel(const u32x4_t *src, int64_t n, uint32_t *sink) {
    constexpr int64_t kTile = (int64_t)kReadThreads * kReadBatch;
    uint32_t acc = 0;
    for (int64_t t0 = (int64_t)blockIdx.x * kTile; t0 < n; t0 += (int64_t)gridDim.x * kTile) {
        u32x4_t v[kReadBatch];
#pragma unroll
        for (int u = 0; u < kReadBatch; u++) {
            const int64_t i = t0 + (int64_t)kReadThreads * u + threadIdx.x;
            v[u] = ld_stream16(src + (i < n ? i : n - 1));   // clamped, not folded twice
        }
#pragma unroll
        for (int u = 0; u < kReadBatch; u++)
            if (t0 + (int64_t)kReadThreads * u + threadIdx.x < n)
                acc ^= fold(v[u]);
    }
    sink[(size_t)blockIdx.x * kReadThreads + threadIdx.x] = acc;
}

// Reads, for every page an attention call with the same arguments streams,
// the whole K block and V block of each KV head, in the attention kernels'
// worker partition (attn_common.h) and with their loads: the same lanes read
// the same 16-byte pieces through a buffer resource bounded to the block, one
// page in flight while the previous one is consumed, and a prefetch past the
// segment end reads nothing.  Nothing is computed beyond folding the words
// into one per lane (written to `sink`), so its bandwidth is the ceiling of
// the paged access pattern itself: random 32 D-byte blocks found through the
// page table.
template <int D>
struct GatherPage {
    static constexpr int KS = D / 32;          // 16-byte K pieces per lane
    static constexpr int VE = D / 16;          // value dims per lane
    static constexpr int kBlockBytes = kPage * D * 2;
    u32x4_t k[KS];
    u32x4_t v[4];      // at D = 64 only .x, .y are loaded (8 bytes per row)

    __device__ __forceinline__ void load(const AttnParams &p, const int32_t *pt, int j, int j1, int g, int lane) {
        const int n = lane & 15, kq = lane >> 4;
        const bool in = j < j1;
        const int pid = ld_meta(pt, in ? j : j1 - 1);
        const size_t base = ((size_t)pid * p.Hkv + g) * (size_t)(kPage * D);
        const block_rsrc_t rk = block_rsrc(p.k_pages + base, in ? kBlockBytes : 0);
        const block_rsrc_t rv = block_rsrc(p.v_pages + base, in ? kBlockBytes : 0);
#pragma unroll
        for (int s = 0; s < KS; s++)
            k[s] = ld_block16(rk, 2 * (n * D + 8 * kq + 32 * s));
#pragma unroll
        for (int i = 0; i < 4; i++) {
            if constexpr (VE == 8) {
                v[i] = ld_block16(rv, 2 * ((4 * kq + i) * D + VE * n));
            } else {
                const u32x2_t t = ld_block8(rv, 2 * ((4 * kq + i) * D + VE * n));
                v[i] = u32x4_t{t.x, t.y, 0u, 0u};
            }
        }
    }
    __device__ __forceinline__ uint32_t fold() const {
        uint32_t a = 0;
#pragma unroll
        for (int s = 0; s < KS; s++)
            a ^= k[s].x ^ k[s].y ^ k[s].z ^ k[s].w;
#pragma unroll
        for (int i = 0; i < 4; i++)
            a ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
        return a;
    }
};

template <int D>
__global__ __launch_bounds__(kWave) void page_gather_kernel(AttnParams p, uint32_t *sink) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    const int lane = threadIdx.x;
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int w = xcd_worker(blockIdx.x, p.W);
    const int64_t end = worker_begin(ptot, w + 1, p.W);
    uint32_t acc = 0;
    for (int64_t x = worker_begin(ptot, w, p.W); x < end;) {
        const Segment s = locate(p, s_pre, x, end);
        const int32_t *pt = p.page_table + (size_t)s.b * p.max_pages;
        GatherPage<D> r0, r1;
        r0.load(p, pt, s.j0, s.j1, s.g, lane);
        sched_fence();
        for (int j = s.j0; j < s.j1; j += 2) {
            r1.load(p, pt, j + 1, s.j1, s.g, lane);
            sched_fence();
            acc ^= r0.fold();
            sched_fence();
            r0.load(p, pt, j + 2, s.j1, s.g, lane);
            sched_fence();
            acc ^= r1.fold();   // zeros for a page past the segment
            sched_fence();
        }
        x = s.next;
    }
    sink[(size_t)w * kWave + lane] = acc;
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
    if ((bytes & 15) || ((uintptr_t)src & 15) || ((uintptr_t)sink & 3))
        return fail(TS_ERR_ARG, "stream read needs 16-byte sizes and alignment");
    const int64_t blocks = 256 * 8;
    if (sink_bytes < (size_t)blocks * kReadThreads * sizeof(uint32_t))
        return fail(TS_ERR_ARG, "sink needs %lld bytes", (long long)(blocks * kReadThreads * 4));
    int st = check_device();
    if (st)
        return st;
    const int64_t n = (int64_t)(bytes / 16);
    if (n == 0)
        return TS_OK;
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)blocks), dim3(kReadThreads), 0,
                       reinterpret_cast<hipStream_t>(stream), static_cast<const u32x4_t *>(src), n,
                       static_cast<uint32_t *>(sink));
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "stream read launch");
}

int ts_page_gather_read(const ts_attn_shape *s, const void *k_pages, const void *v_pages,
                        const int32_t *page_table, const int32_t *ctx_lens, const int32_t *q_lens,
                        void *sink, size_t sink_bytes, void *stream, void *ev_begin, void *ev_end) {
    clear_error();
    int st = check_shape(s);
    if (st)
        return st;
    if (!k_pages || !v_pages || !page_table || !ctx_lens || !q_lens || !sink)
        return fail(TS_ERR_NULL, "NULL pointer");
    if (((uintptr_t)k_pages & 15) || ((uintptr_t)v_pages & 15) || ((uintptr_t)sink & 3))
        return fail(TS_ERR_ARG, "misaligned pointer (pools need 16 B)");
    const int W = s->num_workers > 0 ? s->num_workers : 256 * 4;
    if (sink_bytes < (size_t)W * kWave * sizeof(uint32_t))
        return fail(TS_ERR_ARG, "sink needs %zu bytes", (size_t)W * kWave * sizeof(uint32_t));
    st = check_device();
    if (st)
        return st;
    AttnParams p = {};
    p.k_pages = static_cast<const uint16_t *>(k_pages);
    p.v_pages = static_cast<const uint16_t *>(v_pages);
    p.page_table = page_table;
    p.ctx_lens = ctx_lens;
    p.q_lens = q_lens;
    p.B = s->num_seqs;
    p.Hq = s->num_q_heads;
    p.Hkv = s->num_kv_heads;
    p.D = s->head_dim;
    p.Qmax = s->max_q_len;
    p.max_pages = s->max_pages_per_seq;
    p.W = W;
    void (*k)(AttnParams, uint32_t *) = p.D == 64 ? page_gather_kernel<64> : page_gather_kernel<128>;
    uint32_t *out = static_cast<uint32_t *>(sink);
    void *args[] = {&p, &out};
    hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void *>(k), dim3(W), dim3(kWave), args,
                                      (size_t)(p.B + 1) * sizeof(int), reinterpret_cast<hipStream_t>(stream),
                                      reinterpret_cast<hipEvent_t>(ev_begin), reinterpret_cast<hipEvent_t>(ev_end), 0);
    if (e == hipSuccess)
        e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "page gather launch");
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
