// api.hip -- host side of libtsattn: shape validation, kernel selection,
// the work-partition size, launches and error reporting behind the C ABI
// declared in include/ts_attn.h.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <string>

#include "attn_common.h"
#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {

kernel_fn decode_q1_variant(int D, int G);
kernel_fn verify_variant(int D, int NB);
kernel_fn verify_team_variant(int rows, int *lds_bytes, int *nbe);
kernel_fn merge_variant(int D, bool few);
int debug_check(const ts_attn_shape *s, const int32_t *page_table, const int32_t *ctx_lens,
                const int32_t *q_lens, const int *counters, int *flags, hipStream_t stream);

static thread_local std::string g_last_error;

int fail(int status, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

void clear_error() { g_last_error.clear(); }

int hip_fail(hipError_t e, const char *what) {
    return fail(TS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Device architecture check, once per device.
int check_device() {
    static std::mutex mu;
    static int known[64] = {0};   // 0 unknown, 1 ok, -1 unsupported
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= 64)
        return fail(TS_ERR_UNSUPPORTED, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lock(mu);
    if (known[dev] == 0) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, dev);
        if (e != hipSuccess)
            return hip_fail(e, "hipGetDeviceProperties");
        known[dev] = (std::strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : -1;
        if (known[dev] < 0)
            return fail(TS_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950",
                        dev, prop.gcnArchName);
    }
    if (known[dev] < 0)
        return fail(TS_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
    return TS_OK;
}

struct Plan {
    bool q1;          // one-token VALU kernel, else a matrix-core verify kernel
    bool team;        // verify by four-wavefront teams sharing pages in LDS (head_dim 128)
    bool auto_w;      // worker count chosen by the library (W is then an upper bound)
    int G, NB, rows_per_unit, W;
    size_t ws_cnt_off, ws_dbg_off, ws_o_off, ws_lse_off, ws_bytes;
};

// Number of workers sharing the KV stream.  MI355X has 256 compute units.
// Measured (after a clock warm-up of a few hundred calls) on the bulk, MTP and
// block-draft workloads: the VALU decode kernel is best with 4 wavefronts per
// compute unit (1024); the single-wavefront matrix-core kernel with 4 for up
// to 8 rows per unit (one-token decode; at head_dim 64 the 4th is worth 7 %)
// and with 3 for more (768 on the MTP workload; 1024 is within 1 %); the
// team kernel with 2 teams per compute unit (512), although its registers
// would allow 3: the third team lowers throughput by 8 %.  The auto count is further capped at launch by
// the occupancy the HIP runtime reports for the compiled kernel, so all
// workers run in one round.
static int per_cu_bound(bool q1, bool team, int rows) {
    if (q1)
        return 4;
    if (team)
        return 2;
    return rows <= 8 ? 4 : 3;
}

static int auto_workers(const ts_attn_shape *s, bool q1, bool team, int rows) {
    int64_t w = 256LL * per_cu_bound(q1, team, rows);
    // Small shapes get fewer workers so that each has at least a few pages.
    const int64_t pages_ub = (int64_t)s->num_seqs * s->num_kv_heads *
                             ((s->max_ctx_len + kPage - 1) / kPage);
    const int64_t by_size = (pages_ub + 7) / 8;
    if (by_size < w)
        w = by_size;
    // But one or two sequences are bound by each worker's chain of dependent
    // page loads: give them up to one worker per compute unit, while every
    // worker keeps two pages and a unit is split into at most 24 pieces, which
    // one merge pass reads in one memory round trip.  At one sequence this
    // measured 14-16 % faster than 8 pages per worker (103-192 workers); 30
    // pieces per unit was 4 % slower than 24.
    const int64_t units = (int64_t)s->num_seqs * s->num_kv_heads;
    const int64_t floor_w = std::min<int64_t>(std::min<int64_t>(256, 24 * units), pages_ub / 2);
    if (w < floor_w)
        w = floor_w;
    // Above one worker per compute unit, a whole number per compute unit: with
    // k on some and k + 1 on others the fuller ones stream slower and the
    // launch waits for them (640 workers measured 5-9 % slower than 512 or
    // 768 at 16-64 sequences).
    if (w > 256)
        w -= w % 256;
    return (int)(w < 1 ? 1 : w);
}

// Workgroups of `k` resident per compute unit times the compute units, or 0
// if the runtime cannot tell.  The LDS size is rounded up to 4 KiB (the
// answer is then a lower bound, never an overestimate), so the cache keeps
// one entry per kernel, device, block size and LDS bucket however many batch
// sizes a caller uses.
static int resident_workers(kernel_fn k, int threads, size_t lds) {
    static std::mutex mu;
    static std::map<std::tuple<kernel_fn, int, int, size_t>, int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return 0;
    const size_t bucket = (lds + 4095) & ~(size_t)4095;
    const auto key = std::make_tuple(k, dev, threads, bucket);
    std::lock_guard<std::mutex> lock(mu);
    const auto it = cache.find(key);
    if (it != cache.end())
        return it->second;
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(k), threads, bucket) !=
            hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    const int n = per_cu * cus;
    cache.emplace(key, n);
    return n;
}

int check_shape(const ts_attn_shape *s) {
    if (!s)
        return fail(TS_ERR_NULL, "shape is NULL");
    if (s->num_seqs < 1 || s->num_seqs > kMaxSeqs)
        return fail(TS_ERR_SHAPE, "num_seqs %d outside [1, %d]", s->num_seqs, kMaxSeqs);
    if (s->num_kv_heads < 1 || s->num_q_heads < 1 || s->num_q_heads % s->num_kv_heads)
        return fail(TS_ERR_SHAPE, "num_q_heads %d must be a positive multiple of num_kv_heads %d",
                    s->num_q_heads, s->num_kv_heads);
    if ((int64_t)s->num_seqs * s->num_kv_heads > kMaxUnits)
        return fail(TS_ERR_SHAPE, "num_seqs * num_kv_heads = %lld exceeds %d",
                    (long long)s->num_seqs * s->num_kv_heads, kMaxUnits);
    if (s->head_dim != 64 && s->head_dim != 128)
        return fail(TS_ERR_SHAPE, "head_dim %d unsupported (64 or 128)", s->head_dim);
    if (s->page_size != kPage)
        return fail(TS_ERR_SHAPE, "page_size %d unsupported (16)", s->page_size);
    if (s->max_q_len < 1 || s->max_q_len > 16)
        return fail(TS_ERR_SHAPE, "max_q_len %d outside [1, 16]", s->max_q_len);
    const int G = s->num_q_heads / s->num_kv_heads;
    if (G > 16 || G * s->max_q_len > 64)
        return fail(TS_ERR_SHAPE, "group size %d x max_q_len %d exceeds 64 rows per KV head", G,
                    s->max_q_len);
    if (s->max_pages_per_seq < 1)
        return fail(TS_ERR_SHAPE, "max_pages_per_seq %d < 1", s->max_pages_per_seq);
    if ((int64_t)s->num_seqs * s->max_pages_per_seq >= (1LL << 31))
        return fail(TS_ERR_SHAPE, "num_seqs x max_pages_per_seq exceeds 2^31");
    if (s->max_ctx_len < 1 || (int64_t)s->max_ctx_len > (int64_t)s->max_pages_per_seq * kPage)
        return fail(TS_ERR_SHAPE, "max_ctx_len %d outside [1, max_pages_per_seq x 16]", s->max_ctx_len);
    if (s->num_pages < 1 || s->num_pages > (1LL << 31))
        return fail(TS_ERR_SHAPE, "num_pages %lld outside [1, 2^31]", (long long)s->num_pages);
    if (s->num_workers < 0 || s->num_workers > (1 << 20))
        return fail(TS_ERR_SHAPE, "num_workers %d outside [0, 2^20]", s->num_workers);
    if (s->variant < TS_VARIANT_AUTO || s->variant > TS_VARIANT_VALU)
        return fail(TS_ERR_SHAPE, "variant %d unknown", s->variant);
    if (s->variant == TS_VARIANT_TEAM && s->head_dim != 128)
        return fail(TS_ERR_SHAPE, "the team verify kernel needs head_dim 128");
    return TS_OK;
}

int make_plan(const ts_attn_shape *s, Plan *pl) {
    const int st = check_shape(s);
    if (st)
        return st;
    const int G = s->num_q_heads / s->num_kv_heads;
    pl->G = G;
    // The one-token VALU kernel runs only on request: the single-wavefront
    // matrix-core kernel was measured faster on one-token decode too (bulk
    // workload 2.5 %, 16-128 sequences 5-14 %, group size 8 by 19 %).
    pl->q1 = s->variant == TS_VARIANT_VALU;
    if (pl->q1 && !(s->max_q_len == 1 && (G == 1 || G == 2 || G == 4 || G == 8)))
        return fail(TS_ERR_SHAPE, "the VALU decode kernel needs max_q_len 1 and a group size of 1, 2, 4 or 8");
    pl->rows_per_unit = G * s->max_q_len;
    pl->NB = (pl->rows_per_unit + 15) / 16;
    // Up to two row blocks (32 rows) run best on one wavefront (MTP workload;
    // 20-24 rows at 4-512 sequences: 3-7 % ahead of the team kernel); from
    // three row blocks on the team kernel, which shares each page through LDS
    // (block-draft workload, 64 rows: 12 % ahead at 4 sequences).
    pl->team = !pl->q1 && s->head_dim == 128 &&
               (s->variant == TS_VARIANT_TEAM || (s->variant == TS_VARIANT_AUTO && pl->NB >= 3));
    pl->auto_w = s->num_workers == 0;
    pl->W = s->num_workers > 0 ? s->num_workers : auto_workers(s, pl->q1, pl->team, pl->rows_per_unit);
    // Workspace: the split counters first, at a fixed size whatever the shape,
    // so that no call's partial results ever land on them (they are zero
    // between calls); then 256 bytes for the TS_DEBUG check's flag word; then
    // the partial outputs and their log-sum-exp.
    const size_t slots = 2 * (size_t)pl->W;
    pl->ws_cnt_off = 0;
    pl->ws_dbg_off = kCounterBytes;
    pl->ws_o_off = pl->ws_dbg_off + 256;
    const size_t o_bytes = slots * pl->rows_per_unit * s->head_dim * sizeof(float);
    pl->ws_lse_off = pl->ws_o_off + ((o_bytes + 255) & ~(size_t)255);
    pl->ws_bytes = pl->ws_lse_off + ((slots * pl->rows_per_unit * sizeof(float) + 255) & ~(size_t)255);
    return TS_OK;
}

static bool debug_enabled() {
    static int v = -1;
    if (v < 0) {
        const char *e = std::getenv("TS_DEBUG");
        v = (e && e[0] == '1') ? 1 : 0;
    }
    return v == 1;
}

// Everything a call launches, decided from the shape and the device.
struct Launch {
    kernel_fn main_k = nullptr;   // the streaming kernel
    kernel_fn merge_k = nullptr;  // the merge kernel (kCombineKernel only)
    size_t lds = 0;               // dynamic LDS of the merge kernel (the partition prefix)
    size_t main_lds = 0;          // dynamic LDS of the streaming kernel
    int main_threads = kWave;
    unsigned grid = 0;            // workgroups of the streaming launch: workers, then merge ones
    int combine = kCombineKernel;
    int cnt_shift = 0;
    int ws_o_bytes = 0;
    int64_t merge_blocks = 0;     // workgroups of the merge kernel
};

// Completes a plan for the current device: kernel, worker count, how the
// splits are combined and the launch sizes.  Launches nothing.
static int finish_plan(const ts_attn_shape *s, Plan &pl, Launch &L) {
    int st = check_device();
    if (st)
        return st;
    const int B = s->num_seqs, Hkv = s->num_kv_heads, D = s->head_dim;
    L.lds = (size_t)(B + 1) * sizeof(int);
    L.main_lds = L.lds;
    L.main_threads = kWave;
    if (pl.q1) {
        L.main_k = decode_q1_variant(D, pl.G);
    } else if (pl.team) {
        int extra = 0, nbe = 0;
        L.main_k = verify_team_variant(pl.rows_per_unit, &extra, &nbe);
        L.main_lds = ((L.lds + 15) & ~(size_t)15) + (size_t)extra;
        L.main_threads = 4 * kWave;
    } else {
        L.main_k = verify_variant(D, pl.NB);
    }
    if (!L.main_k || !merge_variant(D, false))
        return fail(TS_ERR_UNSUPPORTED, "no kernel for head_dim %d, G %d, rows %d", D, pl.G, pl.rows_per_unit);
    if (pl.auto_w) {
        // one full round of resident workers (the workspace is sized for pl.W)
        const int resident = resident_workers(L.main_k, L.main_threads, L.main_lds);
        if (resident > 0 && resident < pl.W)
            pl.W = resident;
    }
    // Who combines the splits (attn_split.h):
    //  * the last worker of a unit, for the single-wavefront kernels with at
    //    least twice as many units as workers (a unit has one or two pieces);
    //  * merge wavefronts appended to the grid, one per row of each unit, when
    //    units have many pieces (a unit meets about W / units + 1 workers;
    //    here W >= 8 units) and that takes at most kMaxMergeWgs workgroups;
    //  * otherwise the merge kernel after the launch, and always when the
    //    partial area is too large for 32-bit buffer offsets.
    // Measured against the merge kernel (per call; 32/8 heads, head_dim 128):
    // in the launch it is 2-6 % faster for 1-4 sequences with q_len 4, 4-7 %
    // for 1-8 sequences with q_len 1 (1 % at 16) and 1 % on the block-draft
    // workload (4 sequences, 64 rows).  With 1,024 merge wavefronts (8
    // sequences with q_len 4, the MTP workload) it was 1-2 % slower, and so
    // was it with 2-4 pieces per unit (64-128 sequences), hence the bounds.
    constexpr int64_t kMaxMergeWgs = 512;
    const size_t o_bytes = pl.ws_lse_off - pl.ws_o_off;
    const int64_t units = (int64_t)B * Hkv;
    const int ngroups = (pl.rows_per_unit + 3) / 4;
    const int64_t merge_wgs = units * (pl.team ? ngroups : pl.rows_per_unit);
    L.combine = kCombineKernel;
    if (o_bytes < ((size_t)1 << 31)) {
        if (!pl.team && units >= 2 * (int64_t)pl.W)
            L.combine = kCombineLast;
        else if ((int64_t)pl.W >= 8 * units && merge_wgs <= kMaxMergeWgs)
            L.combine = kCombineInLaunch;
    }
    L.ws_o_bytes = L.combine != kCombineKernel ? (int)o_bytes : 0;
    // Counters of consecutive units up to 4 KiB apart (inside the counter
    // area) when merge wavefronts poll them.
    L.cnt_shift = 0;
    if (L.combine == kCombineInLaunch)
        while (L.cnt_shift < 10 && units << (L.cnt_shift + 1) <= kMaxUnits)
            L.cnt_shift++;
    L.grid = (unsigned)(pl.W + (L.combine == kCombineInLaunch ? merge_wgs : 0));
    if (L.combine == kCombineInLaunch && pl.team && pl.auto_w) {
        // Reserve enough LDS that only the workers' teams fit on a compute
        // unit (their registers would allow one more): a merge workgroup then
        // starts where a team has finished instead of polling beside two
        // streaming teams from the start, which measured 1 % faster.
        const size_t lds_cu = (size_t)160 * 1024;
        const int teams = per_cu_bound(false, true, pl.rows_per_unit);
        const size_t gate = ((lds_cu / teams + lds_cu / (teams + 1)) / 2) & ~(size_t)1023;
        if (L.main_lds < gate)
            L.main_lds = gate;
    }
    if (L.combine == kCombineKernel) {
        // A unit meets about W / units + 1 workers.  Up to about three pieces
        // a unit, one wavefront per 4 rows takes every piece itself (a fourth
        // of the blocks); beyond that four wavefronts share each row group's
        // pieces.  Measured: 1,024 units with 16-32 rows, 768-1,024 workers,
        // 1.5-6 % faster per call; at 4 pieces a unit (32 skewed sequences)
        // the long sequences' units made it 2 % slower, hence the bound.
        const bool few = (int64_t)pl.W <= 2 * units;
        L.merge_k = merge_variant(D, few);
        L.merge_blocks = units * (few ? (ngroups + 3) / 4 : ngroups);
    }
    return TS_OK;
}

int launch_attn(const ts_attn_shape *s, const void *q, const void *k_pages, const void *v_pages,
                  const int32_t *page_table, const int32_t *ctx_lens, const int32_t *q_lens,
                  void *out, float scale, void *workspace, size_t workspace_bytes, void *stream,
                  void *ev_begin, void *ev_end) {
    clear_error();
    Plan pl;
    int st = make_plan(s, &pl);
    if (st)
        return st;
    if (!q || !k_pages || !v_pages || !page_table || !ctx_lens || !q_lens || !out)
        return fail(TS_ERR_NULL, "a tensor pointer is NULL");
    if (!workspace)
        return fail(TS_ERR_NULL, "workspace is NULL (need %zu bytes)", pl.ws_bytes);
    if (workspace_bytes < pl.ws_bytes)
        return fail(TS_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, pl.ws_bytes);
    if (((uintptr_t)workspace & 255) || ((uintptr_t)q & 15) || ((uintptr_t)out & 15) ||
        ((uintptr_t)k_pages & 15) || ((uintptr_t)v_pages & 15))
        return fail(TS_ERR_ARG, "misaligned pointer (workspace needs 256 B, tensors 16 B)");
    if (!std::isfinite(scale))
        return fail(TS_ERR_ARG, "scale is not finite");
    Launch L;
    st = finish_plan(s, pl, L);
    if (st)
        return st;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);

    int *counters = reinterpret_cast<int *>(static_cast<char *>(workspace) + pl.ws_cnt_off);
    if (debug_enabled()) {
        int *flags = reinterpret_cast<int *>(static_cast<char *>(workspace) + pl.ws_dbg_off);
        st = debug_check(s, page_table, ctx_lens, q_lens, counters, flags, hs);
        if (st)
            return st;
    }

    AttnParams p;
    p.q = static_cast<const uint16_t *>(q);
    p.k_pages = static_cast<const uint16_t *>(k_pages);
    p.v_pages = static_cast<const uint16_t *>(v_pages);
    p.page_table = page_table;
    p.ctx_lens = ctx_lens;
    p.q_lens = q_lens;
    p.out = static_cast<uint16_t *>(out);
    p.ws_o = reinterpret_cast<float *>(static_cast<char *>(workspace) + pl.ws_o_off);
    p.ws_lse = reinterpret_cast<float *>(static_cast<char *>(workspace) + pl.ws_lse_off);
    p.counters = counters;
    p.B = s->num_seqs;
    p.Hq = s->num_q_heads;
    p.Hkv = s->num_kv_heads;
    p.D = s->head_dim;
    p.Qmax = s->max_q_len;
    p.max_pages = s->max_pages_per_seq;
    p.G = pl.G;
    p.rows_per_unit = pl.rows_per_unit;
    p.W = pl.W;
    p.ws_o_bytes = L.ws_o_bytes;
    p.combine = (int16_t)L.combine;
    p.cnt_shift = (int16_t)L.cnt_shift;
    p.scale_log2 = scale * 1.4426950408889634f;

    hipError_t e;
    if (ev_begin || ev_end) {
        // the events take the kernel's own start and end timestamps
        void *args[] = {&p};
        e = hipExtLaunchKernel(reinterpret_cast<const void *>(L.main_k), dim3(L.grid), dim3(L.main_threads), args,
                               L.main_lds, hs, reinterpret_cast<hipEvent_t>(ev_begin),
                               reinterpret_cast<hipEvent_t>(ev_end), 0);
        if (e != hipSuccess)
            return hip_fail(e, "attention kernel launch");
    } else {
        hipLaunchKernelGGL(L.main_k, dim3(L.grid), dim3(L.main_threads), L.main_lds, hs, p);
    }
    if ((e = hipGetLastError()) != hipSuccess)
        return hip_fail(e, "attention kernel launch");
    if (L.combine != kCombineKernel)
        return TS_OK;   // the launch combined its own splits
    hipLaunchKernelGGL(L.merge_k, dim3((unsigned)L.merge_blocks), dim3(4 * kWave), L.lds, hs, p);
    if ((e = hipGetLastError()) != hipSuccess)
        return hip_fail(e, "merge kernel launch");
    return TS_OK;
}

}  // namespace tsattn

using namespace tsattn;

extern "C" {

size_t ts_decode_attn_workspace_size(const ts_attn_shape *shape) {
    clear_error();
    Plan pl;
    if (make_plan(shape, &pl))
        return 0;
    return pl.ws_bytes;
}

int ts_decode_attn_plan(const ts_attn_shape *shape, ts_attn_plan *plan) {
    try {
        clear_error();
        if (!plan)
            return fail(TS_ERR_NULL, "plan is NULL");
        Plan pl;
        int st = make_plan(shape, &pl);
        if (st)
            return st;
        Launch L;
        st = finish_plan(shape, pl, L);
        if (st)
            return st;
        plan->variant = pl.q1 ? TS_VARIANT_VALU : pl.team ? TS_VARIANT_TEAM : TS_VARIANT_WAVE;
        plan->num_workers = pl.W;
        plan->combine = L.combine == kCombineLast       ? TS_COMBINE_LAST_ARRIVER
                        : L.combine == kCombineInLaunch ? TS_COMBINE_IN_LAUNCH
                                                        : TS_COMBINE_MERGE_KERNEL;
        plan->grid = (int32_t)L.grid;
        plan->threads = L.main_threads;
        plan->merge_blocks = (int32_t)L.merge_blocks;
        plan->lds_bytes = (int64_t)L.main_lds;
        plan->workspace_bytes = (int64_t)pl.ws_bytes;
        return TS_OK;
    } catch (...) {
        return fail(TS_ERR_HIP, "unexpected C++ exception");
    }
}

int ts_decode_attn(const ts_attn_shape *shape, const void *q, const void *k_pages,
                   const void *v_pages, const int32_t *page_table, const int32_t *ctx_lens,
                   const int32_t *q_lens, void *out, float scale, void *workspace,
                   size_t workspace_bytes, void *stream) {
    try {
        return launch_attn(shape, q, k_pages, v_pages, page_table, ctx_lens, q_lens, out, scale,
                      workspace, workspace_bytes, stream, nullptr, nullptr);
    } catch (...) {
        return fail(TS_ERR_HIP, "unexpected C++ exception");
    }
}

int ts_decode_attn_events(const ts_attn_shape *shape, const void *q, const void *k_pages,
                          const void *v_pages, const int32_t *page_table,
                          const int32_t *ctx_lens, const int32_t *q_lens, void *out,
                          float scale, void *workspace, size_t workspace_bytes, void *stream,
                          void *ev_begin, void *ev_end) {
    try {
        return launch_attn(shape, q, k_pages, v_pages, page_table, ctx_lens, q_lens, out, scale,
                      workspace, workspace_bytes, stream, ev_begin, ev_end);
    } catch (...) {
        return fail(TS_ERR_HIP, "unexpected C++ exception");
    }
}

const char *ts_status_string(int status) {
    switch (status) {
    case TS_OK: return "ok";
    case TS_ERR_NULL: return "null pointer";
    case TS_ERR_SHAPE: return "unsupported or inconsistent shape";
    case TS_ERR_WORKSPACE: return "workspace too small";
    case TS_ERR_UNSUPPORTED: return "unsupported device or configuration";
    case TS_ERR_HIP: return "HIP runtime error";
    case TS_ERR_ARG: return "invalid argument";
    default: return "unknown status";
    }
}

const char *ts_last_error(void) { return g_last_error.c_str(); }

int ts_version(void) { return TS_ATTN_ABI_VERSION; }

}  // extern "C"
