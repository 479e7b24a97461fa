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
// group of 4 rows.  Partials are loaded kMergeBatch at a time, all loads
// issued before any is consumed.
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
    // Adds a batch of up to kMergeBatch partials (n valid) given their rows.
    // kCoherent: read them with device-coherent loads (partials written by
    // other workers of the same launch), else with plain vector loads.
    template <int D, bool kCoherent>
    __device__ void add_batch(const AttnParams &p, const size_t *rows, int n, int part) {
        float l[kMergeBatch];
        float4 v[kMergeBatch][VE / 4];
#pragma unroll
        for (int k = 0; k < kMergeBatch; k++) {
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
        for (int k = 0; k < kMergeBatch; k++)
            Mb = fmaxf(Mb, l[k]);
        if (Mb == -INFINITY)
            return;
        rescale(Mb);
#pragma unroll
        for (int k = 0; k < kMergeBatch; k++) {
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

// Adds to `a` the partials k = k0, k0 + kstep, ... of row rr of the unit.
template <int D, bool kCoherent>
__device__ void gather_partials(const AttnParams &p, const UnitSplit &u, size_t rr, int part,
                                int k0, int kstep, Acc<D / 16> &a) {
    const size_t R = p.rows_per_unit;
    for (int kb = k0; kb < u.nparts; kb += kstep * kMergeBatch) {
        size_t rows[kMergeBatch];
        int n = 0;
#pragma unroll
        for (int k = 0; k < kMergeBatch; k++) {
            const int kk = kb + kstep * k;
            rows[k] = (size_t)u.slot(kk < u.nparts ? kk : kb) * R + rr;
            n += kk < u.nparts;
        }
        a.template add_batch<D, kCoherent>(p, rows, n, part);
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
        gather_partials<D, true>(p, u, row_ok ? r : 0, part, 0, 1, a);
        if (row_ok)
            write_merged<D>(p, b, g, r, part, a);
    }
    // every arrival has been counted: leave the counter zero for the next call
    __hip_atomic_store(p.counters + (size_t)b * p.Hkv + g, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Counts this wavefront's arrival on the unit of a piece whose partial it has
// just written with device-coherent stores; the last arriver combines the
// unit.  The stores are complete once the vector memory counter has drained,
// so no cache-wide fence is needed, and the last arriver's loads are issued
// after its count returned.  The counters are zero between calls (the
// workspace is zero-filled before its first use, and the last arriver of each
// unit resets its counter).
template <int D>
__device__ void arrive_and_combine(const AttnParams &p, const Segment &s, int64_t ptot, int lane) {
    wait_vmem();
    int old = 0;
    if (lane == 0)
        old = atomicAdd(p.counters + (size_t)s.b * p.Hkv + s.g, 1);
    old = first_lane_int(old);
    const UnitSplit u = unit_split(ptot, s.us, s.np, p.W);
    if (old == u.nparts - 1)
        combine_unit<D>(p, s.b, s.g, u, lane);
}

}  // namespace tsattn
