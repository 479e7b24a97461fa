// attn_merge.hip -- combines the split partial results of units that more
// than one wavefront worked on (see the work partition in attn_common.h).
//
// For a row with partials (o_s, lse_s), lse in log2 units:
//   M = max_s lse_s,  w_s = 2^(lse_s - M),  out = sum_s w_s o_s / sum_s w_s,
// and a split that saw no visible key (lse = -inf) has weight 0.  The slots
// are visited in worker order, so the result is deterministic.  One block
// of 256 threads handles 16 rows of one unit: thread (row, part) owns D/16
// consecutive dims of one row.
#include "attn_common.h"

namespace tsattn {

namespace {

template <int D>
__global__ __launch_bounds__(256) void merge_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    constexpr int VE = D / 16;
    const int nrb = (p.rows_per_unit + 15) / 16;
    const int unit = blockIdx.x / nrb;
    const int rb = blockIdx.x % nrb;
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

    const int r = rb * 16 + (threadIdx.x >> 4);
    const int part = threadIdx.x & 15;
    const int Q = p.q_lens[b];
    if (r >= p.rows_per_unit || r / p.G >= Q)
        return;

    // Workers with an empty range (more workers than pages) wrote nothing.
    float M = -INFINITY;
    for (int w = wlo; w <= whi; w++) {
        const int64_t wb = worker_begin(ptot, w, p.W);
        if (worker_begin(ptot, w + 1, p.W) == wb)
            continue;
        const int slot = wb >= us ? 2 * w : 2 * w + 1;
        M = fmaxf(M, p.ws_lse[(size_t)slot * p.rows_per_unit + r]);
    }
    float acc[VE];
#pragma unroll
    for (int e = 0; e < VE; e++)
        acc[e] = 0.0f;
    float den = 0.0f;
    for (int w = wlo; w <= whi; w++) {
        const int64_t wb = worker_begin(ptot, w, p.W);
        if (worker_begin(ptot, w + 1, p.W) == wb)
            continue;
        const int slot = wb >= us ? 2 * w : 2 * w + 1;
        const size_t row = (size_t)slot * p.rows_per_unit + r;
        const float lse = p.ws_lse[row];
        if (lse == -INFINITY)
            continue;
        const float wt = fast_exp2(lse - M);
        den += wt;
        const float *src = p.ws_o + row * D + VE * part;
#pragma unroll
        for (int e = 0; e < VE; e += 4) {
            const float4 v = *reinterpret_cast<const float4 *>(src + e);
            acc[e] += wt * v.x;
            acc[e + 1] += wt * v.y;
            acc[e + 2] += wt * v.z;
            acc[e + 3] += wt * v.w;
        }
    }
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
