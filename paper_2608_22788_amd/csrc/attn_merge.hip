// attn_merge.hip -- combines the split partial results of units that more
// than one worker processed, whenever the streaming launch did not combine
// them itself (kCombineKernel).  The combination rule and the lane layout
// are in attn_split.h.
//
// Two shapes of the same work, chosen on the host from the expected number
// of pieces per unit:
//   * merge_kernel (many pieces, e.g. a few long sequences split over the
//     whole chip): one block of four wavefronts per 4 rows of a unit; the
//     waves take interleaved pieces, so up to 32 pieces cost one memory
//     latency, and their running sums are combined through LDS;
//   * merge_few_kernel (a handful of pieces per unit, many units): one
//     wavefront per 4 rows, taking every piece itself, four row groups per
//     block.  Four times fewer blocks, no LDS exchange, and still one memory
//     latency for up to 8 pieces.
#include "attn_split.h"

namespace tsattn {

namespace {

constexpr int kWaves = 4;    // wavefronts per merge block

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
    if (np == 0)
        return;
    const UnitSplit u = unit_split(ptot, us, np, p.W);
    if (u.wlo == u.whi)
        return;   // one worker saw the whole unit and wrote `out`

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = rg * 4 + (lane >> 4);
    const int part = lane & 15;
    const int Q = ld_meta(p.q_lens, b);
    const bool row_ok = r < p.rows_per_unit && r / p.G < Q;
    const size_t rr = row_ok ? r : 0;   // keep addresses inside the workspace

    Acc<VE> a;
    a.init();
    gather_partials<D, false>(p, u, rr, part, wave, kWaves, a);   // wave w takes partials w, w + 4, ...

    // combine the waves' running sums (lane-wise) through LDS
    __shared__ float s_comb[(kWaves - 1) * (VE + 2) * 64];
    combine_waves<VE, kWaves>(a, s_comb, wave, lane);
    if (wave != 0 || !row_ok)
        return;
    write_merged<D>(p, b, g, r, part, a);
}

template <int D>
__global__ __launch_bounds__(kWaves * 64) void merge_few_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    const int ngroups = (p.rows_per_unit + 3) / 4;
    const int nblk = (ngroups + kWaves - 1) / kWaves;   // blocks per unit
    const int unit = blockIdx.x / nblk;
    const int b = unit / p.Hkv;
    const int g = unit % p.Hkv;
    const int np = s_pre[b + 1] - s_pre[b];
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int64_t us = (int64_t)p.Hkv * s_pre[b] + (int64_t)g * np;
    if (np == 0)
        return;
    const UnitSplit u = unit_split(ptot, us, np, p.W);
    if (u.wlo == u.whi)
        return;   // one worker saw the whole unit and wrote `out`

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int rg = (blockIdx.x % nblk) * kWaves + wave;
    if (rg >= ngroups)
        return;
    const int r = rg * 4 + (lane >> 4);
    const int part = lane & 15;
    const int Q = ld_meta(p.q_lens, b);
    const bool row_ok = r < p.rows_per_unit && r / p.G < Q;
    Acc<D / 16> a;
    a.init();
    gather_partials<D, false>(p, u, row_ok ? r : 0, part, 0, 1, a);
    if (row_ok)
        write_merged<D>(p, b, g, r, part, a);
}

}  // namespace

typedef void (*kernel_fn)(AttnParams);

kernel_fn merge_variant(int D, bool few) {
    if (D == 64)
        return few ? merge_few_kernel<64> : merge_kernel<64>;
    if (D == 128)
        return few ? merge_few_kernel<128> : merge_kernel<128>;
    return nullptr;
}

}  // namespace tsattn
