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
// One block of four wavefronts handles 4 rows of one unit: in each wave, lane
// (row, part) owns D/16 consecutive dims of one row, and the four waves take
// interleaved partials, kBatch at a time with all loads issued before any is
// consumed, so a unit with up to 32 partials costs one memory latency; the
// waves' running sums are then combined through LDS.  Workers with an empty
// range (more workers than pages) wrote nothing and are skipped.
#include "attn_common.h"

namespace tsattn {

namespace {

constexpr int kBatch = 8;    // partials in flight per lane
constexpr int kWaves = 4;    // wavefronts per merge block

// The k-th partial slot (k = 0, 1, ...) of a unit that starts at global page
// us and spans workers wlo..whi.  When every worker has at least one page
// (ptot >= W) worker wlo + k began inside the unit for k > 0 (slot 2w), and
// only wlo's start needs comparing with us.
struct DenseSlots {
    int wlo, first_slot;
    __device__ int operator()(int k) const { return k == 0 ? first_slot : 2 * (wlo + k); }
};

// Running log-sum-exp combination of partials for one lane's D/16 dims.
template <int VE>
struct Acc {
    float acc[VE];
    float den, M;
    __device__ void init() {
#pragma unroll
        for (int e = 0; e < VE; e++)
            acc[e] = 0.0f;
        den = 0.0f;
        M = -INFINITY;
    }
    // Adds a batch of up to kBatch partials (n valid) given their rows.
    template <int D>
    __device__ void add_batch(const AttnParams &p, const size_t *rows, int n, int part) {
        float l[kBatch];
        float4 v[kBatch][VE / 4];
#pragma unroll
        for (int k = 0; k < kBatch; k++) {
            const size_t row = rows[k < n ? k : 0];
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
            return;
        rescale(Mb);
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
    __device__ void rescale(float Mnew) {
        const float a = M == -INFINITY ? 0.0f : fast_exp2(M - Mnew);
        den *= a;
#pragma unroll
        for (int e = 0; e < VE; e++)
            acc[e] *= a;
        M = Mnew;
    }
};

template <int D>
__global__ __launch_bounds__(kWaves * 64) void merge_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    constexpr int VE = D / 16;
    const int ngroups = (p.rows_per_unit + 3) / 4;
    const int unit = blockIdx.x / ngroups;
    const int rg = blockIdx.x % ngroups;
    const int b = unit / p.Hkv;
    const int g = unit % p.Hkv;
    const int np = s_pre[b + 1] - s_pre[b];
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int64_t us = (int64_t)p.Hkv * s_pre[b] + (int64_t)g * np;
    const int wlo = np ? worker_of(ptot, us, p.W) : 0;
    const int whi = np ? worker_of(ptot, us + np - 1, p.W) : 0;
    if (np == 0 || wlo == whi)
        return;   // nothing to do, or one worker saw the whole unit and wrote `out`

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = rg * 4 + (lane >> 4);
    const int part = lane & 15;
    const int Q = ld_meta(p.q_lens, b);
    const bool row_ok = r < p.rows_per_unit && r / p.G < Q;
    const size_t rr = row_ok ? r : 0;   // keep addresses inside the workspace
    const size_t R = p.rows_per_unit;

    Acc<VE> a;
    a.init();
    if (ptot >= p.W) {
        // wave w takes partials w, w + 4, ... in batches of kBatch
        const DenseSlots slot{wlo, worker_begin(ptot, wlo, p.W) >= us ? 2 * wlo : 2 * wlo + 1};
        const int nparts = whi - wlo + 1;
        for (int k0 = wave; k0 < nparts; k0 += kWaves * kBatch) {
            size_t rows[kBatch];
            int n = 0;
#pragma unroll
            for (int k = 0; k < kBatch; k++) {
                const int kk = k0 + kWaves * k;
                rows[k] = (size_t)slot(kk < nparts ? kk : k0) * R + rr;
                n += kk < nparts;
            }
            a.template add_batch<D>(p, rows, n, part);
        }
    } else if (wave == 0) {
        // more workers than pages: skip the workers whose range is empty
        int64_t wb = worker_begin(ptot, wlo, p.W);
        for (int w = wlo; w <= whi;) {
            size_t rows[kBatch];
            int n = 0;
            while (n < kBatch && w <= whi) {
                const int64_t we = worker_begin(ptot, w + 1, p.W);
                if (we > wb)
                    rows[n++] = (size_t)(wb >= us ? 2 * w : 2 * w + 1) * R + rr;
                wb = we;
                w++;
            }
            if (n)
                a.template add_batch<D>(p, rows, n, part);
        }
    }

    // combine the waves' running sums (lane-wise) through LDS
    __shared__ float s_comb[kWaves - 1][VE + 2][64];
    if (wave > 0) {
#pragma unroll
        for (int e = 0; e < VE; e++)
            s_comb[wave - 1][e][lane] = a.acc[e];
        s_comb[wave - 1][VE][lane] = a.den;
        s_comb[wave - 1][VE + 1][lane] = a.M;
    }
    __syncthreads();
    if (wave != 0 || !row_ok)
        return;
    float Mall = a.M;
#pragma unroll
    for (int w = 0; w < kWaves - 1; w++)
        Mall = fmaxf(Mall, s_comb[w][VE + 1][lane]);
    a.rescale(Mall);
#pragma unroll
    for (int w = 0; w < kWaves - 1; w++) {
        const float Mw = s_comb[w][VE + 1][lane];
        const float f = Mw == -INFINITY ? 0.0f : fast_exp2(Mw - Mall);
        a.den += f * s_comb[w][VE][lane];
#pragma unroll
        for (int e = 0; e < VE; e++)
            a.acc[e] += f * s_comb[w][e][lane];
    }
    const float inv = a.den > 0.0f ? 1.0f / a.den : 0.0f;
    const int i = r / p.G;
    uint16_t *dst = p.out + (((size_t)b * p.Qmax + i) * p.Hq + (size_t)g * p.G + r % p.G) * D + VE * part;
    uint32_t w2[VE / 2];
#pragma unroll
    for (int e = 0; e < VE / 2; e++)
        w2[e] = pack_bf16x2(a.acc[2 * e] * inv, a.acc[2 * e + 1] * inv);
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
