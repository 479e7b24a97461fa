// attn_split.h -- combining the split partial results of a unit (the work
// partition is described in attn_common.h).
//
// For a row with partials (o_s, lse_s), lse in log2 units:
//   M = max_s lse_s,  w_s = 2^(lse_s - M),  out = sum_s w_s o_s / sum_s w_s,
// and a split that saw no visible key (lse = -inf) has weight 0.  Partials
// are visited in worker order, so the result is deterministic.  (The sums
// are kept relative to the running maximum and rescaled when it grows, which
// gives the same value up to rounding.)
//
// Lane layout of a combining wavefront: lane (row, part) = 16 * row + part
// owns dims VE * part .. VE * part + VE - 1 (VE = D / 16) of row `row` of a
// group of 4 rows.  Partials are loaded kMergeBatch at a time (4 in the
// streaming kernels' own combine, whose registers are shared with the page
// pipeline), all loads issued before any is consumed.
#pragma once

#include "attn_common.h"

namespace tsattn {

constexpr int kMergeBatch = 8;

// Loads and stores coherent across the whole device (the L2 caches of all
// XCDs), so that the worker combining a unit sees the partials the others
// wrote in the same launch.  Scalar ones are relaxed atomics at agent scope;
// the 16-byte ones are buffer loads and stores over the partial area with the
// device-scope cache policy (the host combines in the kernel only while that
// area is below 2 GiB, so byte offsets fit the buffer's 32-bit offsets).  On
// gfx950 both are plain memory operations with that policy bit, and a store
// is visible device-wide once the issuing wavefront's vector memory counter
// has drained.
constexpr int kDeviceScope = 16;   // cache policy of buffer operations: sc1

__device__ __forceinline__ float ld_coherent(const float *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ block_rsrc_t partial_rsrc(const AttnParams &p) {
    return block_rsrc(p.ws_o, p.ws_o_bytes);
}
// Partial-area elements elem .. elem + 3 (elem a multiple of 4).
__device__ __forceinline__ void st_partial16(const AttnParams &p, size_t elem, f32x4_t v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), partial_rsrc(p),
                                           (int)(elem * sizeof(float)), 0, kDeviceScope);
}
// Partial-area element elem.
__device__ __forceinline__ void st_partial4(const AttnParams &p, size_t elem, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), partial_rsrc(p), (int)(elem * sizeof(float)), 0,
                                          kDeviceScope);
}
__device__ __forceinline__ f32x4_t ld_partial16(const AttnParams &p, size_t elem) {
    return __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                           partial_rsrc(p), (int)(elem * sizeof(float)), 0, kDeviceScope));
}
// Waits until every vector memory operation this wavefront issued is
// complete.  The wait itself is not a memory operation to the compiler, so
// compiler-only fences on both sides keep every memory access written before
// it above it and every one written after it below it (they emit no
// instruction; no cache is written back or invalidated).
__device__ __forceinline__ void wait_vmem() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0); expcnt, lgkmcnt left at their maximum
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// The workers whose ranges meet the unit that occupies global pages
// [us, us + np), and the workspace slot of the k-th piece (k = 0 .. nparts-1,
// in worker order).  When every worker has at least one page (ptot >= W),
// worker wlo + k, k > 0, began inside the unit (slot 2 (wlo + k)) and only
// wlo's start needs comparing with us.  Otherwise every range holds at most
// one page, so page us + k of the unit is the whole range of worker
// worker_of(us + k), which began there (slot 2 worker_of(us + k)).
struct UnitSplit {
    int64_t ptot;     // pages of the whole call
    int64_t us;       // global index of the unit's first page
    int W;            // workers
    int wlo, whi;     // first and last worker whose range meets the unit
    int first_slot;   // slot of worker wlo's piece
    bool dense;       // ptot >= W
    int nparts;       // workers with a non-empty piece of the unit
    __device__ __forceinline__ int slot(int k) const {
        if (dense)
            return k == 0 ? first_slot : 2 * (wlo + k);
        return 2 * worker_of(ptot, us + k, W);
    }
};

__device__ __forceinline__ UnitSplit unit_split(int64_t ptot, int64_t us, int np, int W) {
    UnitSplit u;
    u.ptot = ptot;
    u.us = us;
    u.W = W;
    u.wlo = worker_of(ptot, us, W);
    u.whi = worker_of(ptot, us + np - 1, W);
    u.dense = ptot >= W;
    u.first_slot = worker_begin(ptot, u.wlo, W) >= us ? 2 * u.wlo : 2 * u.wlo + 1;
    u.nparts = u.dense ? u.whi - u.wlo + 1 : np;
    return u;
}

// Running log-sum-exp combination of partials for one lane's VE dims.
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
    // Adds a batch of up to kB partials (n valid) given their rows.
    // kCoherent: read them with device-coherent loads (partials written by
    // other workers of the same launch), else with plain vector loads.
    template <int D, bool kCoherent, int kB>
    __device__ void add_batch(const AttnParams &p, const size_t *rows, int n, int part) {
        float l[kB];
        float4 v[kB][VE / 4];
#pragma unroll
        for (int k = 0; k < kB; k++) {
            const size_t row = rows[k < n ? k : 0];
            const float *src = p.ws_o + row * D + VE * part;
            if constexpr (kCoherent) {
                l[k] = k < n ? ld_coherent(p.ws_lse + row) : -INFINITY;
#pragma unroll
                for (int e = 0; e < VE / 4; e++) {
                    const f32x4_t t = ld_partial16(p, row * D + VE * part + 4 * e);
                    v[k][e] = make_float4(t[0], t[1], t[2], t[3]);
                }
            } else {
                l[k] = k < n ? p.ws_lse[row] : -INFINITY;
#pragma unroll
                for (int e = 0; e < VE / 4; e++)
                    v[k][e] = *reinterpret_cast<const float4 *>(src + 4 * e);
            }
        }
        float Mb = M;
#pragma unroll
        for (int k = 0; k < kB; k++)
            Mb = fmaxf(Mb, l[k]);
        if (Mb == -INFINITY)
            return;
        rescale(Mb);
#pragma unroll
        for (int k = 0; k < kB; k++) {
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

// Adds to `a` the partials k = k0, k0 + kstep, ... of row rr of the unit,
// kB at a time.
template <int D, bool kCoherent, int kB = kMergeBatch>
__device__ void gather_partials(const AttnParams &p, const UnitSplit &u, size_t rr, int part,
                                int k0, int kstep, Acc<D / 16> &a) {
    const size_t R = p.rows_per_unit;
    for (int kb = k0; kb < u.nparts; kb += kstep * kB) {
        size_t rows[kB];
        int n = 0;
#pragma unroll
        for (int k = 0; k < kB; k++) {
            const int kk = kb + kstep * k;
            rows[k] = (size_t)u.slot(kk < u.nparts ? kk : kb) * R + rr;
            n += kk < u.nparts;
        }
        a.template add_batch<D, kCoherent, kB>(p, rows, n, part);
    }
}

// Normalises and writes row r (of the unit's rows_per_unit) as bf16.
template <int D>
__device__ __forceinline__ void write_merged(const AttnParams &p, int b, int g, int r, int part,
                                             const Acc<D / 16> &a) {
    constexpr int VE = D / 16;
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

// Combines all pieces of unit (b, g) and writes its rows (one wavefront;
// rows_per_unit rows, 4 per pass; rows of draft positions >= q_len are
// skipped).  Called by the worker that counted the last arrival on the unit,
// which then sets the counter back to zero for the next call.
template <int D>
__device__ void combine_unit(const AttnParams &p, int b, int g, const UnitSplit &u, int lane) {
    const int part = lane & 15;
    const int R = p.rows_per_unit;
    const int Q = ld_meta(p.q_lens, b);
    for (int r0 = 0; r0 < R; r0 += 4) {
        const int r = r0 + (lane >> 4);
        const bool row_ok = r < R && r / p.G < Q;
        Acc<D / 16> a;
        a.init();
        gather_partials<D, true, 4>(p, u, row_ok ? r : 0, part, 0, 1, a);
        if (row_ok)
            write_merged<D>(p, b, g, r, part, a);
    }
    // every arrival has been counted: leave the counter zero for the next call
    __hip_atomic_store(unit_counter(p, b * p.Hkv + g), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// kCombineLast: counts this wavefront's arrival on the unit of a piece whose
// partial it has just written with device-coherent stores; the last arriver
// combines the unit.  The stores are complete once the vector memory counter
// has drained, so no cache-wide fence is needed, and the last arriver's loads
// are issued after its count returned.  The counters are zero between calls
// (the workspace is zero-filled before its first use, and each call leaves
// them zero).
template <int D>
__device__ void arrive_and_combine(const AttnParams &p, const Segment &s, int64_t ptot, int lane) {
    wait_vmem();
    int old = 0;
    if (lane == 0)
        old = atomicAdd(unit_counter(p, s.b * p.Hkv + s.g), 1);
    old = first_lane_int(old);
    const UnitSplit u = unit_split(ptot, s.us, s.np, p.W);
    if (old == u.nparts - 1)
        combine_unit<D>(p, s.b, s.g, u, lane);
}

// kCombineInLaunch: a worker has split pieces in at most two units (the first
// and the last segment of its range) and counts its arrivals on them once,
// after its whole range: every piece of a split unit ends near the end of
// the launch anyway, and a drain of the stores between segments would stall
// the worker for a memory round trip.
struct Arrivals {
    int u0, u1;   // units of the pending arrivals, -1 for none
    __device__ __forceinline__ void init() { u0 = u1 = -1; }
    __device__ __forceinline__ void add(const AttnParams &p, const Segment &s) {
        if (!s.whole && p.combine == kCombineInLaunch) {
            const int u = s.b * p.Hkv + s.g;
            if (u0 < 0)
                u0 = u;
            else
                u1 = u;
        }
    }
    // Called by every thread of the workgroup; the first thread counts.
    template <bool kBlock>
    __device__ __forceinline__ void flush(const AttnParams &p) {
        if (u0 < 0)
            return;
        wait_vmem();
        if constexpr (kBlock)
            __syncthreads();   // every wavefront's stores are complete
        if (threadIdx.x == 0) {
            atomicAdd(unit_counter(p, u0), 1);
            if (u1 >= 0)
                atomicAdd(unit_counter(p, u1), 1);
        }
    }
};

// Sums of waves 1 .. kWaves - 1 of a workgroup added into wave 0's `a` (the
// same lanes of each wave hold the same rows and dims), through LDS at
// `comb` (3 * (VE + 2) * 64 floats).  Every thread of the workgroup calls it.
template <int VE, int kWaves>
__device__ void combine_waves(Acc<VE> &a, float *comb, int wave, int lane) {
    float(*c)[VE + 2][64] = reinterpret_cast<float(*)[VE + 2][64]>(comb);
    if (wave > 0) {
#pragma unroll
        for (int e = 0; e < VE; e++)
            c[wave - 1][e][lane] = a.acc[e];
        c[wave - 1][VE][lane] = a.den;
        c[wave - 1][VE + 1][lane] = a.M;
    }
    __syncthreads();
    if (wave != 0)
        return;
    float Mall = a.M;
#pragma unroll
    for (int w = 0; w < kWaves - 1; w++)
        Mall = fmaxf(Mall, c[w][VE + 1][lane]);
    if (Mall == -INFINITY)
        return;   // no partial saw a visible key: the sums stay zero
    a.rescale(Mall);
#pragma unroll
    for (int w = 0; w < kWaves - 1; w++) {
        const float Mw = c[w][VE + 1][lane];
        const float f = Mw == -INFINITY ? 0.0f : fast_exp2(Mw - Mall);
        a.den += f * c[w][VE][lane];
#pragma unroll
        for (int e = 0; e < VE; e++)
            a.acc[e] += f * c[w][e][lane];
    }
}

// ---------------------------------------------------------------------------
// Merge wavefronts in the streaming launch (kCombineInLaunch).
//
// The grid holds the W workers and then the merge workgroups, one wavefront
// per row of each unit (single-wavefront kernels: workgroup W + m is row
// m % R of unit m / R; four-wavefront kernels: wave w of workgroup W + m is
// row 4 (m % ceil(R / 4)) + w of unit m / ceil(R / 4)).  A merge wavefront
// waits until every worker with a piece of its unit has counted its arrival,
// then its four 16-lane groups read pieces k, k + 4, ... (k = lane / 16)
// with device-coherent loads, so up to 4 * kMergeBatch pieces cost one
// memory round trip; the groups' sums meet through cross-lane exchanges and
// group 0 writes the row.  The host takes this mode for units with many
// pieces (a few long sequences), where the merge kernel's launch after the
// whole grid was a large share of a short call.
//
// Forward progress: the dispatcher starts the workgroups of each XCD in
// increasing order, so every worker has started before any merge workgroup
// of its XCD, and workers never wait.  A merge wavefront therefore only
// waits for workgroups that are running.  The wait is bounded all the same
// (kMergeSpins polls); a wavefront that gives up writes NaN, so such a
// failure shows in the output instead of as a hang.
//
// Counter protocol: the unit's counter reaches nparts once every worker has
// arrived; then each merge wavefront of the unit with a valid row adds one
// after it has read the partials, and the last of them sets the counter back
// to zero for the next call.  The host spaces the counters of the units
// apart (cnt_shift): with all of them on one line, every worker's arrival
// and every merge wavefront's poll queued on that line, which made the
// block-draft call 38 % slower.
constexpr int kMergeSpins = 1 << 22;

// Waits until *c >= target; false if kMergeSpins polls saw less.
__device__ __forceinline__ bool wait_count(const int *c, int target) {
    for (int i = 0; i < kMergeSpins; i++) {
        const int v = first_lane_int(__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        if (v >= target) {
            __atomic_signal_fence(__ATOMIC_SEQ_CST);   // later loads stay after the poll
            return true;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    return false;
}

// Sums of the four 16-lane groups (same part, different pieces) combined;
// every group gets the total.
template <int VE>
__device__ __forceinline__ void combine_lane_groups(Acc<VE> &a) {
    float Mall = fmaxf(a.M, __shfl_xor(a.M, 16));
    Mall = fmaxf(Mall, __shfl_xor(Mall, 32));
    const float f = a.M == -INFINITY ? 0.0f : fast_exp2(a.M - Mall);
    float den = a.den * f;
    den += __shfl_xor(den, 16);
    den += __shfl_xor(den, 32);
    a.den = den;
#pragma unroll
    for (int e = 0; e < VE; e++) {
        float v = a.acc[e] * f;
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        a.acc[e] = v;
    }
    a.M = Mall;
}

// Combines and writes row r of unit `unit` (one wavefront).
template <int D>
__device__ void merge_in_launch(const AttnParams &p, const int *s_pre, int unit, int r) {
    const int b = unit / p.Hkv, g = unit % p.Hkv;
    const int np = s_pre[b + 1] - s_pre[b];
    if (np == 0)
        return;
    const int nvalid = min(p.rows_per_unit, ld_meta(p.q_lens, b) * p.G);   // rows with i < q_len
    if (r >= nvalid)
        return;
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int64_t us = (int64_t)p.Hkv * s_pre[b] + (int64_t)g * np;
    const UnitSplit u = unit_split(ptot, us, np, p.W);
    if (u.wlo == u.whi)
        return;   // one worker saw the whole unit and wrote `out`
    const int lane = threadIdx.x & 63;
    int *cnt = unit_counter(p, unit);
    const bool ok = wait_count(cnt, u.nparts);
    Acc<D / 16> a;
    a.init();
    if (ok) {
        gather_partials<D, true>(p, u, r, lane & 15, lane >> 4, 4, a);
    } else {
#pragma unroll
        for (int e = 0; e < D / 16; e++)
            a.acc[e] = __builtin_nanf("");
        a.den = 1.0f;
        a.M = 0.0f;
    }
    combine_lane_groups(a);
    if (lane < 16)
        write_merged<D>(p, b, g, r, lane, a);
    if (lane == 0) {
        const int old = atomicAdd(cnt, 1);
        if (old == u.nparts + nvalid - 1)   // nvalid merge wavefronts per unit
            __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

}  // namespace tsattn
