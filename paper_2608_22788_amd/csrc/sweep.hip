// sweep.hip -- ts_concurrency_sweep: the attention share of the
// concurrency-throughput curve v(b) and per-token time tau(b) = 1 / v(b) that
// the paper's hierarchical controller consumes (Sec. 2.1, Sec. 3.2, App. C.2).
//
// For each batch size b and seed: draw the sweep's context lengths and page
// permutation on the host, fill q/K/V on the device with the seeded
// generator, then time ts_decode_attn with HIP events around groups of 10
// back-to-back calls.  Calls rotate over
// enough distinct KV pools (at least min_rotation_bytes in total) that the
// 256 MB last-level cache cannot serve a pool from the previous call, so small
// batches report HBM, not cache, bandwidth.  The same pools are then read by
// ts_page_gather_read, the call's read-only twin, timed the same way: the
// floor that latency alone sets at small batches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {

int synth_fill(void *dst, int64_t n, uint64_t seed, uint32_t stream_id, int64_t offset,
               hipStream_t stream);
void sweep_lengths(int32_t batch, uint64_t seed, int32_t *ctx_lens);
int build_page_table(int32_t batch, const int32_t *ctx_lens, int32_t page_size,
                     int32_t max_pages_per_seq, uint64_t seed, int32_t *page_table);

namespace {

constexpr uint32_t kStreamQ = 4, kStreamK = 5, kStreamV = 6;
constexpr int kGroup = 10;   // back-to-back calls per timed group

struct DevBuf {
    void *p = nullptr;
    ~DevBuf() {
        if (p)
            (void)hipFree(p);
    }
    int alloc(size_t bytes, const char *what) {
        hipError_t e = hipMalloc(&p, bytes < 256 ? 256 : bytes);
        return e == hipSuccess ? TS_OK : hip_fail(e, what);
    }
};

struct Events {
    std::vector<hipEvent_t> ev;
    ~Events() {
        for (hipEvent_t e : ev)
            (void)hipEventDestroy(e);
    }
};

struct Stream {
    hipStream_t s = nullptr;
    ~Stream() {
        if (s)
            (void)hipStreamDestroy(s);
    }
};

double quantile(std::vector<double> v, double q) {
    std::sort(v.begin(), v.end());
    const double pos = q * (double)(v.size() - 1);
    const size_t lo = (size_t)std::floor(pos);
    const size_t hi = std::min(lo + 1, v.size() - 1);
    return v[lo] + (pos - (double)lo) * (v[hi] - v[lo]);
}

// Host description of one sweep point.
struct Point {
    int32_t batch, seed, Q, maxp, maxl;
    int64_t total_pages, sum_ctx, pools, pool_bytes;
    std::vector<int32_t> lens, qlens, table;
    ts_attn_shape sh;
    size_t ws_bytes;
};

int plan_point(const ts_sweep_config &c, int32_t batch, int32_t seed, Point *pt) {
    Point &P = *pt;
    P.batch = batch;
    P.seed = seed;
    P.Q = batch <= c.verify_max_batch ? c.verify_q_len : 1;
    P.lens.assign((size_t)batch, 0);
    P.qlens.assign((size_t)batch, P.Q);
    sweep_lengths(batch, (uint64_t)seed, P.lens.data());
    P.maxp = 1;
    P.maxl = 1;
    P.total_pages = 0;
    P.sum_ctx = 0;
    for (int32_t L : P.lens) {
        P.maxp = std::max(P.maxp, (L + 15) / 16);
        P.maxl = std::max(P.maxl, L);
        P.total_pages += (L + 15) / 16;
        P.sum_ctx += L;
    }
    P.table.assign((size_t)batch * P.maxp, 0);
    int st = build_page_table(batch, P.lens.data(), 16, P.maxp, (uint64_t)seed, P.table.data());
    if (st)
        return st;
    const int64_t pool_elems = P.total_pages * c.num_kv_heads * 16 * c.head_dim;
    P.pool_bytes = pool_elems * 2;                  // one of K or V
    P.pools = (c.min_rotation_bytes + 2 * P.pool_bytes - 1) / (2 * P.pool_bytes);
    P.pools = std::max<int64_t>(1, std::min<int64_t>(P.pools, 512));
    P.sh = ts_attn_shape{};
    P.sh.num_seqs = batch;
    P.sh.num_q_heads = c.num_q_heads;
    P.sh.num_kv_heads = c.num_kv_heads;
    P.sh.head_dim = c.head_dim;
    P.sh.page_size = 16;
    P.sh.max_q_len = P.Q;
    P.sh.max_pages_per_seq = P.maxp;
    P.sh.max_ctx_len = P.maxl;
    P.sh.num_pages = P.total_pages;
    P.ws_bytes = ts_decode_attn_workspace_size(&P.sh);
    return P.ws_bytes ? TS_OK : TS_ERR_SHAPE;
}

// Device memory for every point of a sweep, allocated once at the largest
// size (memory obtained again from the driver after a free can stream a few
// per cent slower, which would bias later points).
struct Arena {
    DevBuf kv, q, out, ws, tab, len, ql, sink;
    size_t kv_bytes = 0;
};

constexpr int kGatherWorkers = 1024;   // ts_page_gather_read's default

int run_point(const ts_sweep_config &c, const Point &P, Arena &A, hipStream_t stream,
              ts_sweep_point *pt) {
    const int32_t batch = P.batch, Q = P.Q;
    const int64_t pools = P.pools, pool_bytes = P.pool_bytes;
    const int64_t pool_elems = pool_bytes / 2;
    char *kbase = static_cast<char *>(A.kv.p);
    char *vbase = kbase + (size_t)(pool_bytes * pools);
    const size_t qelems = (size_t)batch * Q * c.num_q_heads * c.head_dim;
    hipError_t e;
    int st;
    if ((e = hipMemcpyAsync(A.tab.p, P.table.data(), P.table.size() * 4, hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(A.len.p, P.lens.data(), (size_t)batch * 4, hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(A.ql.p, P.qlens.data(), (size_t)batch * 4, hipMemcpyHostToDevice, stream)))
        return hip_fail(e, "hipMemcpyAsync(sweep inputs)");
    if ((st = synth_fill(kbase, pool_elems * pools, (uint64_t)P.seed, kStreamK, 0, stream)) ||
        (st = synth_fill(vbase, pool_elems * pools, (uint64_t)P.seed, kStreamV, 0, stream)) ||
        (st = synth_fill(A.q.p, (int64_t)qelems, (uint64_t)P.seed, kStreamQ, 0, stream)))
        return st;

    const float scale = 1.0f / std::sqrt((float)c.head_dim);
    auto call = [&](int64_t i) {
        const size_t off = (size_t)((i % pools) * pool_bytes);
        return ts_decode_attn(&P.sh, A.q.p, kbase + off, vbase + off, static_cast<const int32_t *>(A.tab.p),
                              static_cast<const int32_t *>(A.len.p), static_cast<const int32_t *>(A.ql.p),
                              A.out.p, scale, A.ws.p, P.ws_bytes, stream);
    };
    auto gather = [&](int64_t i) {
        const size_t off = (size_t)((i % pools) * pool_bytes);
        return ts_page_gather_read(&P.sh, kbase + off, vbase + off, static_cast<const int32_t *>(A.tab.p),
                                   static_cast<const int32_t *>(A.len.p), static_cast<const int32_t *>(A.ql.p),
                                   A.sink.p, (size_t)kGatherWorkers * 64 * 4, stream, nullptr, nullptr);
    };
    // Timed calls run back to back in groups of up to kGroup, at least five
    // groups, with an event after each group; a point's times are the
    // groups' mean call times (median, p10, p90 over the groups), so a group
    // that a host-side stall stretched does not move the median.  An event
    // after every call measured 2.5-4 us more per call at 1-64 sequences
    // (calls of 12-125 us), which is the cost of the event, not of the call.
    const int group = std::max(1, std::min(kGroup, c.iters / 5));
    const int groups = c.iters / group;
    Events evs;
    evs.ev.resize((size_t)groups + 1);
    for (auto &ev : evs.ev)
        if ((e = hipEventCreate(&ev)))
            return hip_fail(e, "hipEventCreate");
    auto timed = [&](auto &&fn, std::vector<double> &us) -> int {
        int rc;
        hipError_t he;
        for (int i = 0; i < c.warmup; i++)
            if ((rc = fn(i)))
                return rc;
        if ((he = hipEventRecord(evs.ev[0], stream)))
            return hip_fail(he, "hipEventRecord");
        for (int g = 0; g < groups; g++) {
            for (int k = 0; k < group; k++)
                if ((rc = fn(c.warmup + (int64_t)g * group + k)))
                    return rc;
            if ((he = hipEventRecord(evs.ev[(size_t)g + 1], stream)))
                return hip_fail(he, "hipEventRecord");
        }
        if ((he = hipStreamSynchronize(stream)))
            return hip_fail(he, "hipStreamSynchronize");
        us.assign((size_t)groups, 0.0);
        for (int g = 0; g < groups; g++) {
            float ms = 0.f;
            if ((he = hipEventElapsedTime(&ms, evs.ev[(size_t)g], evs.ev[(size_t)g + 1])))
                return hip_fail(he, "hipEventElapsedTime");
            us[(size_t)g] = 1000.0 * ms / group;
        }
        return TS_OK;
    };
    std::vector<double> us, gus;
    if ((st = timed(call, us)) || (st = timed(gather, gus)))
        return st;
    pt->batch = batch;
    pt->q_len = Q;
    pt->seed = P.seed;
    pt->num_pools = (int32_t)pools;
    pt->sum_ctx = P.sum_ctx;
    pt->kv_bytes = P.sum_ctx * c.num_kv_heads * c.head_dim * 2 * 2;
    pt->t_median_us = quantile(us, 0.5);
    pt->t_p10_us = quantile(us, 0.1);
    pt->t_p90_us = quantile(us, 0.9);
    pt->kv_gbps = (double)pt->kv_bytes / (pt->t_median_us * 1e-6) / 1e9;
    pt->hbm_frac = pt->kv_gbps / 8000.0;
    // Tokens emitted per sequence and step: one for plain decode; a verify
    // step emits its accepted drafts plus one, which the caller states
    // (acceptance is not modelled here), so drafts are never counted as
    // emitted tokens by default.
    const double per_step = (Q > 1 && c.verify_tokens_per_step > 0.0) ? c.verify_tokens_per_step : 1.0;
    pt->tokens_per_s = (double)batch * per_step / (pt->t_median_us * 1e-6);
    pt->tau_us = pt->t_median_us / per_step;
    pt->gather_median_us = quantile(gus, 0.5);
    return TS_OK;
}

}  // namespace
}  // namespace tsattn

using namespace tsattn;

extern "C" int ts_concurrency_sweep(const ts_sweep_config *cfg, ts_sweep_point *pts, int32_t cap,
                                    int32_t *n_out) {
    clear_error();
    if (!cfg || !pts || !n_out)
        return fail(TS_ERR_NULL, "NULL argument");
    const ts_sweep_config &c = *cfg;
    if (c.num_batches < 1 || c.num_batches > 32 || c.num_seeds < 1 || c.iters < 1 || c.warmup < 0)
        return fail(TS_ERR_ARG, "invalid batch list, seed count or iteration counts");
    for (int i = 0; i < c.num_batches; i++)
        if (c.batches[i] < 1 || c.batches[i] > 4096)
            return fail(TS_ERR_ARG, "batch size %d outside [1, 4096]", c.batches[i]);
    if (c.verify_q_len < 1 || c.verify_q_len > 16 || c.min_rotation_bytes < 0)
        return fail(TS_ERR_ARG, "invalid verify_q_len or rotation size");
    if ((int64_t)c.num_batches * c.num_seeds > cap)
        return fail(TS_ERR_ARG, "cap %d < %d points", cap, c.num_batches * c.num_seeds);
    int st = check_device();
    if (st)
        return st;
    try {
        // plan every point on the host, then size one arena for the largest
        std::vector<Point> plan((size_t)c.num_batches * c.num_seeds);
        size_t kv = 0, qe = 0, ws = 0, tab = 0, bmax = 0;
        for (int i = 0; i < c.num_batches; i++) {
            for (int seed = 0; seed < c.num_seeds; seed++) {
                Point &P = plan[(size_t)i * c.num_seeds + seed];
                if ((st = plan_point(c, c.batches[i], seed, &P)))
                    return st;
                kv = std::max(kv, (size_t)(2 * P.pool_bytes * P.pools));
                qe = std::max(qe, (size_t)P.batch * P.Q * c.num_q_heads * c.head_dim);
                ws = std::max(ws, P.ws_bytes);
                tab = std::max(tab, P.table.size());
                bmax = std::max(bmax, (size_t)P.batch);
            }
        }
        Arena A;
        Stream s;
        hipError_t e = hipStreamCreate(&s.s);
        if (e != hipSuccess)
            return hip_fail(e, "hipStreamCreate");
        if ((st = A.kv.alloc(kv, "hipMalloc(KV pools)")) || (st = A.q.alloc(qe * 2, "hipMalloc(q)")) ||
            (st = A.out.alloc(qe * 2, "hipMalloc(out)")) || (st = A.ws.alloc(ws, "hipMalloc(workspace)")) ||
            (st = A.tab.alloc(tab * 4, "hipMalloc(page table)")) ||
            (st = A.len.alloc(bmax * 4, "hipMalloc(ctx_lens)")) ||
            (st = A.ql.alloc(bmax * 4, "hipMalloc(q_lens)")) ||
            (st = A.sink.alloc((size_t)kGatherWorkers * 64 * 4, "hipMalloc(gather sink)")))
            return st;
        if ((e = hipMemsetAsync(A.ws.p, 0, ws, s.s)))   // zero before its first use
            return hip_fail(e, "hipMemsetAsync(workspace)");
        int32_t n = 0;
        for (const Point &P : plan) {
            if ((st = run_point(c, P, A, s.s, &pts[n])))
                return st;
            n++;
        }
        *n_out = n;
        return TS_OK;
    } catch (...) {
        return fail(TS_ERR_HIP, "out of host memory");
    }
}
