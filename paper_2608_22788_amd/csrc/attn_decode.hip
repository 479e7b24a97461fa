// attn_decode.hip -- paged decode attention for one query token per sequence
// on the vector ALUs (TS_VARIANT_VALU).  The default for one-token decode is
// the matrix-core kernel of attn_verify.hip, which measured faster on every
// shape tried; this kernel stays as an explicit variant and a cross-check.
//
// One wavefront streams one KV head of one sequence at a time (a segment of
// the work partition in attn_common.h) and serves all G query heads that
// share that KV head, so each K/V byte is fetched from HBM once per group.
//
// Lane layout for a 16-token page: lane = 8 * slot + part.  Token slot
// `slot` (0..7) holds tokens slot and slot + 8 of the page; `part` (0..7)
// holds 8 of every 64 head dimensions (d = 64c + 8 part + 0..7), so the 8
// lanes of a slot read 128 contiguous bytes of a key row per load.
//   * scores: v_dot2_f32_bf16 on packed bf16 pairs of K and q (fp32
//     accumulate), then a 3-step DPP butterfly over the 8 parts;
//   * online softmax per lane (each slot keeps its own running reference
//     m_ref, row sum and output), in log2 units with scale * log2(e) folded
//     into the scores; the reference is only raised when a score exceeds it
//     by more than 8 (a factor 256), so the rescale of the accumulators is
//     skipped by the whole wavefront on almost every page, and the result is
//     the same up to rounding because the final normalisation uses the same
//     reference;
//   * P.V: the two tokens of a slot are packed as one bf16 pair per head
//     dimension, so v_dot2_f32_bf16 multiplies a probability pair by a value
//     pair; the row sum is accumulated from the same rounded probabilities;
//   * at the end of a segment the 8 slots are merged with log-sum-exp
//     weights through cross-lane shuffles.
// Unless p.combine is kCombineKernel, splits are combined in this launch: a
// wavefront that wrote a partial (a piece of a unit that other workers share)
// with device-coherent stores waits for them to complete, then counts its
// arrival on the unit's counter.  With kCombineLast it counts right after the
// piece, and the one that arrives last combines all partials of the unit
// (device-coherent loads), writes the output rows and sets the counter back
// to zero; with kCombineInLaunch it counts after its whole range, and the
// merge wavefronts that follow the workers in the grid combine (attn_split.h).
// No cache-wide write-back or invalidation is needed.  kCombineLast saves
// the merge kernel's launch but puts four dependent memory round trips
// (store, count, partial loads, output) at the end of the last pieces; the
// host takes it when units are at least twice as many as workers (a unit
// then has one or two pieces), where it was measured faster (4-5 % at 256
// sequences).
// Masking: only the last page of a sequence has slots past the context end;
// their probabilities are forced to 0 and their value rows to 0, so stale
// data (even NaN) in unused slots never reaches the output.
#include "attn_split.h"

#include <type_traits>

namespace tsattn {

namespace {

template <int NC>
struct PageRegs {
    u32x4_t k[2][NC];
    u32x4_t v[2][NC];
};

// Calls f(std::integral_constant<int, I>) for I = B .. E - 1 (compile-time).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

template <int D, int G>
struct DecodeQ1 {
    static constexpr int NC = D / 64;   // 16-byte chunks per token row per lane
    static constexpr int NO = NC * 8;   // output dims per lane
    static constexpr int kAhead = 2;    // pages in flight while one is computed

    struct Ring {
        PageRegs<NC> r0, r1, r2;
        template <int K>
        __device__ __forceinline__ PageRegs<NC> &at() {
            static_assert(K >= 0 && K < 3, "ring slot");
            if constexpr (K == 0) return r0;
            else if constexpr (K == 1) return r1;
            else return r2;
        }
    };

    __device__ __forceinline__ static void load_page(const AttnParams &p, const int32_t *pt, int j, int g,
                                     int slot, int part, PageRegs<NC> &r) {
        const int pid = ld_meta(pt, j);
        const size_t base = ((size_t)pid * p.Hkv + g) * (size_t)(kPage * D);
        const uint16_t *kb = p.k_pages + base;
        const uint16_t *vb = p.v_pages + base;
#pragma unroll
        for (int h = 0; h < 2; h++) {
#pragma unroll
            for (int c = 0; c < NC; c++) {
                const int off = (slot + 8 * h) * D + 64 * c + 8 * part;
                r.k[h][c] = ld_stream16(kb + off);
                r.v[h][c] = ld_stream16(vb + off);
            }
        }
    }

    // One 16-token page: scores, online softmax, P.V for all G rows.
    __device__ __forceinline__ static void page(const AttnParams &p, PageRegs<NC> &cur, int j, int L,
                                                int slot, const uint32_t (&qv)[G][NC][4],
                                                float (&o)[G][NO], float (&m_ref)[G], float (&lsum)[G]) {
        // scores of the two tokens of this slot, all G rows
        float x0[G], x1[G];
#pragma unroll
        for (int r = 0; r < G; r++) {
            float a = 0.0f, c1 = 0.0f;
#pragma unroll
            for (int c = 0; c < NC; c++) {
                a = dot2_bf16(cur.k[0][c].x, qv[r][c][0], a);
                c1 = dot2_bf16(cur.k[1][c].x, qv[r][c][0], c1);
                a = dot2_bf16(cur.k[0][c].y, qv[r][c][1], a);
                c1 = dot2_bf16(cur.k[1][c].y, qv[r][c][1], c1);
                a = dot2_bf16(cur.k[0][c].z, qv[r][c][2], a);
                c1 = dot2_bf16(cur.k[1][c].z, qv[r][c][2], c1);
                a = dot2_bf16(cur.k[0][c].w, qv[r][c][3], a);
                c1 = dot2_bf16(cur.k[1][c].w, qv[r][c][3], c1);
            }
            x0[r] = sum8(a) * p.scale_log2;
            x1[r] = sum8(c1) * p.scale_log2;
        }

        const bool tail = (j + 1) * kPage > L;       // wavefront-uniform
        const int tok0 = j * kPage + slot;
        const bool ok0 = !tail || tok0 < L;
        const bool ok1 = !tail || tok0 + 8 < L;

        bool need = false;
        float mx[G];
#pragma unroll
        for (int r = 0; r < G; r++) {
            mx[r] = fmaxf(ok0 ? x0[r] : -INFINITY, ok1 ? x1[r] : -INFINITY);
            need |= mx[r] > m_ref[r] + kRescaleSlack;
        }
        if (__any(need)) {
#pragma unroll
            for (int r = 0; r < G; r++) {
                const bool up = mx[r] > m_ref[r] + kRescaleSlack;
                const float alpha = up ? fast_exp2(m_ref[r] - mx[r]) : 1.0f;
                m_ref[r] = up ? mx[r] : m_ref[r];
                lsum[r] *= alpha;
#pragma unroll
                for (int k = 0; k < NO; k++)
                    o[r][k] *= alpha;
            }
        }

        if (tail) {
#pragma unroll
            for (int c = 0; c < NC; c++) {
                if (!ok0)
                    cur.v[0][c] = u32x4_t{0u, 0u, 0u, 0u};
                if (!ok1)
                    cur.v[1][c] = u32x4_t{0u, 0u, 0u, 0u};
            }
        }

        uint32_t pk[G];
#pragma unroll
        for (int r = 0; r < G; r++) {
            const float p0 = ok0 ? fast_exp2(x0[r] - m_ref[r]) : 0.0f;
            const float p1 = ok1 ? fast_exp2(x1[r] - m_ref[r]) : 0.0f;
            pk[r] = pack_bf16x2(p0, p1);
            lsum[r] = dot2_bf16(pk[r], 0x3F803F80u, lsum[r]);
        }

#pragma unroll
        for (int c = 0; c < NC; c++) {
            const uint32_t va[4] = {cur.v[0][c].x, cur.v[0][c].y, cur.v[0][c].z, cur.v[0][c].w};
            const uint32_t vb[4] = {cur.v[1][c].x, cur.v[1][c].y, cur.v[1][c].z, cur.v[1][c].w};
#pragma unroll
            for (int w = 0; w < 4; w++) {
                // (token slot, token slot + 8) pairs for dims 2w and 2w + 1
                const uint32_t even = (va[w] & 0xffffu) | (vb[w] << 16);
                const uint32_t odd = (va[w] >> 16) | (vb[w] & 0xffff0000u);
#pragma unroll
                for (int r = 0; r < G; r++) {
                    o[r][8 * c + 2 * w] = dot2_bf16(even, pk[r], o[r][8 * c + 2 * w]);
                    o[r][8 * c + 2 * w + 1] = dot2_bf16(odd, pk[r], o[r][8 * c + 2 * w + 1]);
                }
            }
        }
    }

    __device__ static void segment(const AttnParams &p, const Segment &s, int slot_id, int64_t ptot) {
        const int lane = threadIdx.x;
        const int slot = lane >> 3;
        const int part = lane & 7;
        const int b = s.b, g = s.g;
        const int L = ld_meta(p.ctx_lens, b);
        const int32_t *pt = p.page_table + (size_t)b * p.max_pages;

        // query rows of the group, packed bf16 pairs
        uint32_t qv[G][NC][4];
#pragma unroll
        for (int r = 0; r < G; r++) {
            const uint16_t *qr = p.q + ((size_t)b * p.Qmax * p.Hq + (size_t)g * G + r) * D;
#pragma unroll
            for (int c = 0; c < NC; c++) {
                uint4 t = *reinterpret_cast<const uint4 *>(qr + 64 * c + 8 * part);
                qv[r][c][0] = t.x;
                qv[r][c][1] = t.y;
                qv[r][c][2] = t.z;
                qv[r][c][3] = t.w;
            }
        }

        float o[G][NO];
        float m_ref[G], lsum[G];
#pragma unroll
        for (int r = 0; r < G; r++) {
            m_ref[r] = -INFINITY;
            lsum[r] = 0.0f;
#pragma unroll
            for (int k = 0; k < NO; k++)
                o[r][k] = 0.0f;
        }

        // Pages are prefetched kAhead ahead into a ring of register sets
        // addressed by compile-time index.  Every prefetch is issued
        // unconditionally (past the segment the last page is loaded again): a
        // load under a branch would make the compiler wait for it before the
        // current page is computed.
        Ring ring;
        static_for<0, kAhead>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            load_page(p, pt, min(s.j0 + k, s.j1 - 1), g, slot, part, ring.template at<k>());
        });
        for (int j0 = s.j0; j0 < s.j1; j0 += kAhead + 1) {
            static_for<0, kAhead + 1>([&](auto kc) {
                constexpr int k = decltype(kc)::value;
                const int j = j0 + k;
                if (j < s.j1) {
                    load_page(p, pt, min(j + kAhead, s.j1 - 1), g, slot, part,
                              ring.template at<(k + kAhead) % (kAhead + 1)>());
                    page(p, ring.template at<k>(), j, L, slot, qv, o, m_ref, lsum);
                }
            });
        }

        // merge the 8 token slots (lanes part, part + 8, ..., part + 56)
#pragma unroll
        for (int r = 0; r < G; r++) {
            float M = m_ref[r];
            M = fmaxf(M, __shfl_xor(M, 8));
            M = fmaxf(M, __shfl_xor(M, 16));
            M = fmaxf(M, __shfl_xor(M, 32));
            const float a = (m_ref[r] == -INFINITY) ? 0.0f : fast_exp2(m_ref[r] - M);
            float l = lsum[r] * a;
            l += __shfl_xor(l, 8);
            l += __shfl_xor(l, 16);
            l += __shfl_xor(l, 32);
#pragma unroll
            for (int k = 0; k < NO; k++) {
                float v = o[r][k] * a;
                v += __shfl_xor(v, 8);
                v += __shfl_xor(v, 16);
                v += __shfl_xor(v, 32);
                o[r][k] = v;
            }
            const float inv = l > 0.0f ? 1.0f / l : 0.0f;
            if (slot == 0) {
                const int h = g * G + r;
                if (s.whole) {
                    uint16_t *dst = p.out + ((size_t)b * p.Qmax * p.Hq + h) * D;
#pragma unroll
                    for (int c = 0; c < NC; c++) {
                        uint4 w4;
                        w4.x = pack_bf16x2(o[r][8 * c + 0] * inv, o[r][8 * c + 1] * inv);
                        w4.y = pack_bf16x2(o[r][8 * c + 2] * inv, o[r][8 * c + 3] * inv);
                        w4.z = pack_bf16x2(o[r][8 * c + 4] * inv, o[r][8 * c + 5] * inv);
                        w4.w = pack_bf16x2(o[r][8 * c + 6] * inv, o[r][8 * c + 7] * inv);
                        *reinterpret_cast<uint4 *>(dst + 64 * c + 8 * part) = w4;
                    }
                } else {
                    const size_t row = (size_t)slot_id * p.rows_per_unit + r;
                    float *dst = p.ws_o + row * D;
                    const float lse = l > 0.0f ? M + __log2f(l) : -INFINITY;
                    if (p.combine != kCombineKernel) {
                        // device-coherent stores: another wavefront of this
                        // launch combines them
#pragma unroll
                        for (int c = 0; c < NC; c++) {
                            const f32x4_t lo = {o[r][8 * c + 0] * inv, o[r][8 * c + 1] * inv,
                                                o[r][8 * c + 2] * inv, o[r][8 * c + 3] * inv};
                            const f32x4_t hi = {o[r][8 * c + 4] * inv, o[r][8 * c + 5] * inv,
                                                o[r][8 * c + 6] * inv, o[r][8 * c + 7] * inv};
                            st_partial16(p, row * D + 64 * c + 8 * part, lo);
                            st_partial16(p, row * D + 64 * c + 8 * part + 4, hi);
                        }
                        if (part == 0)
                            st_coherent(p.ws_lse + row, lse);
                    } else {
#pragma unroll
                        for (int c = 0; c < NC; c++) {
                            float4 lo = make_float4(o[r][8 * c + 0] * inv, o[r][8 * c + 1] * inv,
                                                    o[r][8 * c + 2] * inv, o[r][8 * c + 3] * inv);
                            float4 hi = make_float4(o[r][8 * c + 4] * inv, o[r][8 * c + 5] * inv,
                                                    o[r][8 * c + 6] * inv, o[r][8 * c + 7] * inv);
                            *reinterpret_cast<float4 *>(dst + 64 * c + 8 * part) = lo;
                            *reinterpret_cast<float4 *>(dst + 64 * c + 8 * part + 4) = hi;
                        }
                        if (part == 0)
                            p.ws_lse[row] = lse;
                    }
                }
            }
        }
        if (!s.whole && p.combine == kCombineLast)
            arrive_and_combine<D>(p, s, ptot, lane);
    }
};

template <int D, int G>
__global__ __launch_bounds__(64) void decode_q1_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    if (__builtin_expect((int)blockIdx.x >= p.W, 0)) {   // merge workgroups, laid out after the workers' code
        const int m = (int)blockIdx.x - p.W;
        merge_in_launch<D>(p, s_pre, m / p.rows_per_unit, m % p.rows_per_unit);
        return;
    }
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int w = xcd_worker(blockIdx.x, p.W);
    const int64_t begin = worker_begin(ptot, w, p.W);
    const int64_t end = worker_begin(ptot, w + 1, p.W);
    Arrivals arr;
    arr.init();
    for (int64_t x = begin; x < end;) {
        const Segment s = locate(p, s_pre, x, end);
        DecodeQ1<D, G>::segment(p, s, x == begin ? 2 * w : 2 * w + 1, ptot);
        arr.add(p, s);
        x = s.next;
    }
    arr.flush<false>(p);
}

}  // namespace

typedef void (*kernel_fn)(AttnParams);

kernel_fn decode_q1_variant(int D, int G) {
#define TS_Q1(DD, GG) \
    if (D == DD && G == GG) return decode_q1_kernel<DD, GG>;
    TS_Q1(64, 1) TS_Q1(64, 2) TS_Q1(64, 4) TS_Q1(64, 8)
    TS_Q1(128, 1) TS_Q1(128, 2) TS_Q1(128, 4) TS_Q1(128, 8)
#undef TS_Q1
    return nullptr;
}

}  // namespace tsattn
