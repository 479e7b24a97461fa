// attn_merge.hip -- combines the split partial results of units that more
// than one wavefront worked on (see the work partition in attn_common.h).
//
// For a row with partials (o_s, lse_s), lse in log2 units:
//   M = max_s lse_s,  w_s = 2^(lse_s - M),  out = sum_s w_s o_s / sum_s w_s,
// and a split that saw no visible key (lse = -inf) has weight 0.  Partials
// are visited in worker order, so the result is deterministic.  (The sums
// are kept relative to the running maximum and rescaled when it grows, which
// gives the same value up to rounding.)
//
// One wavefront handles 4 rows of one unit: lane (row, part) owns D/16
// consecutive dims of one row.  The partial slots of a unit are found by
// walking its workers once (workers with an empty range wrote nothing and are
// skipped); the walk is wavefront-uniform.  Loads of up to kBatch partials
// are issued before any is consumed, so the merge costs a few memory
// latencies rather than one per partial.
#include "attn_common.h"

namespace tsattn {

namespace {

constexpr int kBatch = 8;   // partials in flight per lane

// Slots of the workers wlo..whi that touched a unit starting at global page
// us.  When every worker has at least one page (ptot >= W), worker w > wlo
// began inside the unit (slot 2w) and only wlo needs its start compared with
// us; otherwise workers with an empty range are skipped one by one.
struct SlotWalk {
    int64_t ptot, us, wb;
    int w, whi, W;
    bool dense;
    __device__ SlotWalk(int64_t ptot_, int64_t us_, int wlo, int whi_, int W_)
        : ptot(ptot_), us(us_), wb(worker_begin(ptot_, wlo, W_)), w(wlo), whi(whi_), W(W_),
          dense(ptot_ >= W_) {}
    // Next up to kBatch slots; returns how many.
    __device__ int next(int *slots) {
        int n = 0;
        if (dense) {
            while (n < kBatch && w <= whi) {
                slots[n++] = (wb >= us) ? 2 * w : 2 * w + 1;
                wb = us;   // every later worker begins inside the unit
                w++;
            }
            return n;
        }
        while (n < kBatch && w <= whi) {
            const int64_t we = worker_begin(ptot, w + 1, W);
            if (we > wb)
                slots[n++] = wb >= us ? 2 * w : 2 * w + 1;
            wb = we;
            w++;
        }
        return n;
    }
};

template <int D>
__global__ __launch_bounds__(64) void merge_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    constexpr int VE = D / 16;
    const int ngroups = (p.rows_per_unit + 3) / 4;
    const int unit = blockIdx.x / ngroups;
    const int rg = blockIdx.x % ngroups;
    const int b = unit / p.Hkv;
    const int g = unit % p.Hkv;
    const int np = s_pre[b + 1] - s_pre[b];
    if (np == 0)
        return;
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int64_t us = (int64_t)p.Hkv * s_pre[b] + (int64_t)g * np;
    const int64_t ue = us + np;
    const int wlo = worker_of(ptot, us, p.W);
    const int whi = worker_of(ptot, ue - 1, p.W);
    if (wlo == whi)
        return;   // one worker saw the whole unit and wrote `out` itself

    const int lane = threadIdx.x;
    const int r = rg * 4 + (lane >> 4);
    const int part = lane & 15;
    const int Q = ld_meta(p.q_lens, b);
    const bool row_ok = r < p.rows_per_unit && r / p.G < Q;
    const int rr = row_ok ? r : 0;   // keep addresses inside the workspace

    // One pass: each batch of partials is loaded at once; the running sums
    // are rescaled to the batch's new maximum before the batch is added.
    float acc[VE];
#pragma unroll
    for (int e = 0; e < VE; e++)
        acc[e] = 0.0f;
    float den = 0.0f, M = -INFINITY;
    SlotWalk walk(ptot, us, wlo, whi, p.W);
    int slots[kBatch];
    for (int n; (n = walk.next(slots)) > 0;) {
        float l[kBatch];
        float4 v[kBatch][VE / 4];
#pragma unroll
        for (int k = 0; k < kBatch; k++) {
            const size_t row = (size_t)(k < n ? slots[k] : slots[0]) * p.rows_per_unit + rr;
            l[k] = k < n ? p.ws_lse[row] : -INFINITY;
            const float *src = p.ws_o + row * D + VE * part;
#pragma unroll
            for (int e = 0; e < VE / 4; e++)
                v[k][e] = *reinterpret_cast<const float4 *>(src + 4 * e);
        }
        float Mb = M;
#pragma unroll
        for (int k = 0; k < kBatch; k++)
            Mb = fmaxf(Mb, l[k]);
        if (Mb == -INFINITY)
            continue;
        const float a = M == -INFINITY ? 0.0f : fast_exp2(M - Mb);
        den *= a;
#pragma unroll
        for (int e = 0; e < VE; e++)
            acc[e] *= a;
        M = Mb;
#pragma unroll
        for (int k = 0; k < kBatch; k++) {
            const float wt = l[k] == -INFINITY ? 0.0f : fast_exp2(l[k] - M);
            den += wt;
#pragma unroll
            for (int e = 0; e < VE / 4; e++) {
                acc[4 * e + 0] += wt * v[k][e].x;
                acc[4 * e + 1] += wt * v[k][e].y;
                acc[4 * e + 2] += wt * v[k][e].z;
                acc[4 * e + 3] += wt * v[k][e].w;
            }
        }
    }
    if (!row_ok)
        return;
    const float inv = den > 0.0f ? 1.0f / den : 0.0f;
    const int i = r / p.G;
    uint16_t *dst = p.out + (((size_t)b * p.Qmax + i) * p.Hq + (size_t)g * p.G + r % p.G) * D + VE * part;
    uint32_t w2[VE / 2];
#pragma unroll
    for (int e = 0; e < VE / 2; e++)
        w2[e] = pack_bf16x2(acc[2 * e] * inv, acc[2 * e + 1] * inv);
    if constexpr (VE == 8)
        *reinterpret_cast<uint4 *>(dst) = make_uint4(w2[0], w2[1], w2[2], w2[3]);
    else
        *reinterpret_cast<uint2 *>(dst) = make_uint2(w2[0], w2[1]);
}

}  // namespace

typedef void (*kernel_fn)(AttnParams);

kernel_fn merge_variant(int D) {
    if (D == 64)
        return merge_kernel<64>;
    if (D == 128)
        return merge_kernel<128>;
    return nullptr;
}

}  // namespace tsattn
