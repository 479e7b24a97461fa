// attn_verify.hip -- paged speculative-verify attention: each sequence
// brings q_len = 1 + gamma query rows (the draft block) that attend to the
// whole cache and causally to each other, on bf16 matrix cores.
//
// The G query heads of a KV group times the q_len draft rows form
// R = G * Qmax rows per (sequence, KV head) unit, padded to NB blocks of 16;
// row r is draft position i = r / G of query head g * G + r % G.  One
// wavefront streams the unit's pages and keeps every row block in registers,
// so each K/V byte is read once for all rows of the group.
//
// With l = lane, n = l % 16, kq = l / 16, per 16-token page:
//   * scores S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (A: row l%16, k
//     8(l/16)..+7; B: col l%16, k 8(l/16)..+7; C: row 4(l/16)+i, col l%16):
//     A = 16 key rows x 32 dims loaded straight from the page (16 bytes per
//     lane), B = Q^T kept in registers.  Lane (n, kq) receives tokens
//     4kq..4kq+3 of the page for query row n;
//   * probabilities P = exp2(scale*log2e * S - m_ref), packed to bf16 in the
//     lane that computed them, are exactly the A operand of O = P V on
//     v_mfma_f32_16x16x16_bf16 (A: row l%16, k 4(l/16)..+3);
//   * V is loaded as rows (lane (n, kq) reads D/16 consecutive dims of tokens
//     4kq..4kq+3) and transposed in registers, so the B operand of the j-th
//     P.V product holds dims (D/16) n + j of those four tokens;
//   * row sums come from one more product of P with a ones operand, so they
//     use exactly the rounded probabilities that weight V;
//   * the running reference m_ref of each row is only raised when a score
//     exceeds it by more than 8 in log2 units, which leaves the accumulators
//     untouched on almost every page;
//   * the next page is loaded into a second register set while the current
//     one is computed; loads go through a buffer resource bounded to the
//     page's block, so a prefetch past the end reads nothing (it used to
//     re-read the last page: about 0.8 % of the bulk call's traffic).  With
//     one row block the prefetch runs on across the end of a segment into
//     the next segment's first page, whose lengths and query rows are
//     fetched when the current segment starts, so the pipeline is not
//     drained at a unit boundary.
// Masks: key t is visible to draft row i iff t <= L - Q + i; keys past the
// segment end or the context end get probability 0 and their value rows are
// zeroed before the product, so stale data never reaches the output.
// Splits are combined as p.combine says (attn_split.h): by the last worker to
// finish a piece of the unit, by the merge wavefronts that follow the workers
// in the grid (workgroups W and up), or by the separate merge kernel.
#include "attn_split.h"

namespace tsattn {

namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }
__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t u) { return __builtin_bit_cast(bf16x8_t, u); }
__device__ __forceinline__ s16x4_t as_s16x4(uint2 u) { return __builtin_bit_cast(s16x4_t, u); }

template <int VE>
struct VRow;
template <>
struct VRow<8> {
    uint32_t w[4];
    __device__ void load(block_rsrc_t r, int byte_off) {
        const u32x4_t t = ld_block16(r, byte_off);
        w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
    }
    __device__ void zero() { w[0] = w[1] = w[2] = w[3] = 0; }
};
template <>
struct VRow<4> {
    uint32_t w[2];
    __device__ void load(block_rsrc_t r, int byte_off) {
        const u32x2_t t = ld_block8(r, byte_off);
        w[0] = t.x; w[1] = t.y;
    }
    __device__ void zero() { w[0] = w[1] = 0; }
};

template <int D, int NB>
struct Verify {
    static constexpr int KS = D / 32;   // k-steps of the score product
    static constexpr int VE = D / 16;   // value dims per lane = P.V products per row block
    static constexpr int kBlockBytes = kPage * D * 2;   // one (page, KV head) block

    struct PageRegs {
        u32x4_t k[KS];      // A operands of the score product
        VRow<VE> v[4];      // value rows of the lane's 4 tokens
    };

    // The K and V blocks of KV head g in physical page pid.  With !in the
    // buffer resources hold no records: the loads return zeros and touch no
    // memory, so a prefetch past the worker's range needs no branch.
    __device__ static void load_block(const AttnParams &p, int pid, bool in, int g, int n, int kq, PageRegs &r) {
        const size_t base = ((size_t)pid * p.Hkv + g) * (size_t)(kPage * D);
        const block_rsrc_t rk = block_rsrc(p.k_pages + base, in ? kBlockBytes : 0);
        const block_rsrc_t rv = block_rsrc(p.v_pages + base, in ? kBlockBytes : 0);
#pragma unroll
        for (int s = 0; s < KS; s++)
            r.k[s] = ld_block16(rk, 2 * (n * D + 8 * kq + 32 * s));
#pragma unroll
        for (int i = 0; i < 4; i++)
            r.v[i].load(rv, 2 * ((4 * kq + i) * D + VE * n));
    }

    // Element e (0..VE-1) of a VE-wide bf16 row held in dwords.
    __device__ static uint32_t half_of(const VRow<VE> &v, int e) {
        const uint32_t w = v.w[e >> 1];
        return (e & 1) ? (w >> 16) : (w & 0xffffu);
    }

    struct State {
        uint4 qf[NB][KS];
        int lim[NB];
        f32x4_t acc[NB][VE];
        f32x4_t lacc[NB];
        float m_ref[NB];
    };

    __device__ static void page_step(const AttnParams &p, State &st, PageRegs &cur, int j,
                                     int full_end, int seg_end_tok, int kq) {
        const int t0 = j * kPage;
        const bool masked = t0 + kPage > full_end;          // wavefront-uniform
        if (t0 + kPage > seg_end_tok) {
#pragma unroll
            for (int i = 0; i < 4; i++)
                if (t0 + 4 * kq + i >= seg_end_tok)
                    cur.v[i].zero();
        }
        // transpose the lane's 4 value rows: vt[jj] = dim (VE n + jj) of its 4 tokens
        uint2 vt[VE];
#pragma unroll
        for (int jj = 0; jj < VE; jj++)
            vt[jj] = make_uint2(half_of(cur.v[0], jj) | (half_of(cur.v[1], jj) << 16),
                                half_of(cur.v[2], jj) | (half_of(cur.v[3], jj) << 16));
        const uint2 ones = make_uint2(0x3F803F80u, 0x3F803F80u);

#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            f32x4_t sc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ks++)
                sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.k[ks]), as_bf16x8(st.qf[rb][ks]),
                                                             sc, 0, 0, 0);
            float x[4];
            bool ok[4];
#pragma unroll
            for (int e = 0; e < 4; e++) {
                x[e] = sc[e] * p.scale_log2;
                ok[e] = !masked || (t0 + 4 * kq + e < st.lim[rb]);
            }
            // Lane-local check first: the row maximum (a cross-lane reduction over the
            // four lanes of a row) is only needed when some score exceeds its row's
            // reference by more than the slack, which is rare after the first page.
            float mx = fmaxf(fmaxf(ok[0] ? x[0] : -INFINITY, ok[1] ? x[1] : -INFINITY),
                             fmaxf(ok[2] ? x[2] : -INFINITY, ok[3] ? x[3] : -INFINITY));
            if (__any(mx > st.m_ref[rb] + kRescaleSlack)) {
                mx = fmaxf(mx, __shfl_xor(mx, 16));
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const bool up = mx > st.m_ref[rb] + kRescaleSlack;
                const float alpha = up ? fast_exp2(st.m_ref[rb] - mx) : 1.0f;
                st.m_ref[rb] = up ? mx : st.m_ref[rb];
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const float ai = __shfl(alpha, 4 * kq + i);
                    st.lacc[rb][i] *= ai;
#pragma unroll
                    for (int jj = 0; jj < VE; jj++)
                        st.acc[rb][jj][i] *= ai;
                }
            }
            const float p0 = ok[0] ? fast_exp2(x[0] - st.m_ref[rb]) : 0.0f;
            const float p1 = ok[1] ? fast_exp2(x[1] - st.m_ref[rb]) : 0.0f;
            const float p2 = ok[2] ? fast_exp2(x[2] - st.m_ref[rb]) : 0.0f;
            const float p3 = ok[3] ? fast_exp2(x[3] - st.m_ref[rb]) : 0.0f;
            const s16x4_t pa = as_s16x4(make_uint2(pack_bf16x2(p0, p1), pack_bf16x2(p2, p3)));
            st.lacc[rb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, as_s16x4(ones), st.lacc[rb], 0, 0, 0);
#pragma unroll
            for (int jj = 0; jj < VE; jj++)
                st.acc[rb][jj] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, as_s16x4(vt[jj]),
                                                                           st.acc[rb][jj], 0, 0, 0);
        }
    }

    // The segment being computed, with its lengths and masks.
    struct Cur {
        Segment s;
        const int32_t *pt;   // the sequence's page-table row
        int L, Q;
        int seg_end_tok, full_end;
    };

    __device__ static void head(const AttnParams &p, const Segment &s, Cur &c) {
        c.s = s;
        c.pt = p.page_table + (size_t)s.b * p.max_pages;
        c.L = ld_meta(p.ctx_lens, s.b);
        c.Q = ld_meta(p.q_lens, s.b);
    }

    // Query rows of unit (b, g) in the lane's B-operand layout.  Rows past
    // R = G * Qmax read row R - 1 (inside q); start() zeroes every row that
    // is not a draft row of the sequence.
    __device__ static void load_q(const AttnParams &p, int b, int g, int n, int kq, uint4 (&q)[NB][KS]) {
        const int G = p.G, R = p.rows_per_unit;
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            const int rc = min(rb * 16 + n, R - 1);
            const uint16_t *qr = p.q + (((size_t)b * p.Qmax + rc / G) * p.Hq + (size_t)g * G + rc % G) * D + 8 * kq;
#pragma unroll
            for (int ks = 0; ks < KS; ks++)
                q[rb][ks] = *reinterpret_cast<const uint4 *>(qr + 32 * ks);
        }
    }

    // Masks and empty accumulators for segment c.
    __device__ static void start(const AttnParams &p, Cur &c, const uint4 (&q)[NB][KS], State &st, int n) {
        const int G = p.G, R = p.rows_per_unit, L = c.L, Q = c.Q;
        c.seg_end_tok = min(L, c.s.j1 * kPage);
        // keys below this bound are visible to every row of the block
        c.full_end = min(L - Q + 1, c.seg_end_tok);
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            const int r = rb * 16 + n;
            const bool row_ok = r < R && r / G < Q;
            st.lim[rb] = min(row_ok ? L - Q + r / G + 1 : L, c.seg_end_tok);
#pragma unroll
            for (int ks = 0; ks < KS; ks++)
                st.qf[rb][ks] = row_ok ? q[rb][ks] : make_uint4(0, 0, 0, 0);
            st.m_ref[rb] = -INFINITY;
            st.lacc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int jj = 0; jj < VE; jj++)
                st.acc[rb][jj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
    }

    // Writes segment c's rows: to `out` when the segment is its whole unit,
    // else as a normalised partial with its log2-sum-exp in slot slot_id.
    __device__ static void finish(const AttnParams &p, const Cur &c, const State &st, int slot_id, int64_t ptot,
                                  int n, int kq) {
        const int b = c.s.b, g = c.s.g, G = p.G, R = p.rows_per_unit, Q = c.Q;
        // lane holds rows 16 rb + 4 kq + i, dims VE n .. VE n + VE - 1
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int r = rb * 16 + 4 * kq + i;
                const float m = __shfl(st.m_ref[rb], 4 * kq + i);
                const float l = st.lacc[rb][i];
                const int di = r / G;
                if (r >= R || di >= Q)
                    continue;
                const float inv = l > 0.0f ? 1.0f / l : 0.0f;
                if (c.s.whole) {
                    uint16_t *dst = p.out + (((size_t)b * p.Qmax + di) * p.Hq + (size_t)g * G + r % G) * D + VE * n;
                    uint32_t w[VE / 2];
#pragma unroll
                    for (int e = 0; e < VE / 2; e++)
                        w[e] = pack_bf16x2(st.acc[rb][2 * e][i] * inv, st.acc[rb][2 * e + 1][i] * inv);
                    if constexpr (VE == 8)
                        *reinterpret_cast<uint4 *>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
                    else
                        *reinterpret_cast<uint2 *>(dst) = make_uint2(w[0], w[1]);
                } else {
                    const size_t row = (size_t)slot_id * R + r;
                    float *dst = p.ws_o + row * D + VE * n;
                    const float lse = l > 0.0f ? m + __log2f(l) : -INFINITY;
                    if (p.combine != kCombineKernel) {
                        // device-coherent: another wavefront of this launch combines them
#pragma unroll
                        for (int e = 0; e < VE; e += 4)
                            st_partial16(p, row * D + VE * n + e,
                                         f32x4_t{st.acc[rb][e][i] * inv, st.acc[rb][e + 1][i] * inv,
                                                 st.acc[rb][e + 2][i] * inv, st.acc[rb][e + 3][i] * inv});
                        if (n == 0)
                            st_coherent(p.ws_lse + row, lse);
                    } else {
#pragma unroll
                        for (int e = 0; e < VE; e += 4)
                            *reinterpret_cast<float4 *>(dst + e) =
                                make_float4(st.acc[rb][e][i] * inv, st.acc[rb][e + 1][i] * inv,
                                            st.acc[rb][e + 2][i] * inv, st.acc[rb][e + 3][i] * inv);
                        if (n == 0)
                            p.ws_lse[row] = lse;
                    }
                }
            }
        }
        if (!c.s.whole && p.combine == kCombineLast)
            arrive_and_combine<D>(p, c.s, ptot, threadIdx.x);
    }

    // One segment on its own, the page after the current one in flight
    // within the segment (the layout for two or more row blocks, which have
    // no registers to spare for a pipeline across segments).
    __device__ static void segment(const AttnParams &p, const Segment &s, int slot_id, int64_t ptot) {
        const int lane = threadIdx.x;
        const int n = lane & 15;
        const int kq = lane >> 4;
        const int G = p.G, R = p.rows_per_unit;
        Cur c;
        head(p, s, c);
        c.seg_end_tok = min(c.L, s.j1 * kPage);
        c.full_end = min(c.L - c.Q + 1, c.seg_end_tok);
        State st;
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            const int r = rb * 16 + n;
            const bool row_ok = r < R && r / G < c.Q;
            const int i = row_ok ? r / G : 0;
            const int hl = row_ok ? r % G : 0;
            st.lim[rb] = min(row_ok ? c.L - c.Q + i + 1 : c.L, c.seg_end_tok);
            const uint16_t *qr = p.q + (((size_t)s.b * p.Qmax + i) * p.Hq + (size_t)s.g * G + hl) * D + 8 * kq;
#pragma unroll
            for (int ks = 0; ks < KS; ks++)
                st.qf[rb][ks] = row_ok ? *reinterpret_cast<const uint4 *>(qr + 32 * ks) : make_uint4(0, 0, 0, 0);
            st.m_ref[rb] = -INFINITY;
            st.lacc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int jj = 0; jj < VE; jj++)
                st.acc[rb][jj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        PageRegs ring[2];
        load_block(p, ld_meta(c.pt, s.j0), true, s.g, n, kq, ring[0]);
        for (int j = s.j0; j < s.j1; j += 2) {
#pragma unroll
            for (int k = 0; k < 2; k++) {
                if (j + k < s.j1) {
                    const bool in = j + k + 1 < s.j1;
                    load_block(p, ld_meta(c.pt, in ? j + k + 1 : s.j1 - 1), in, s.g, n, kq, ring[1 - k]);
                    page_step(p, st, ring[k], j + k, c.full_end, c.seg_end_tok, kq);
                }
            }
        }
        finish(p, c, st, slot_id, ptot, n, kq);
    }

    // Streams the worker's global pages [begin, end) with one row block as
    // one pipeline: the page after the current one is always in flight, also
    // across the end of a segment, where it is the next segment's first page.
    // The next segment is located, its lengths read and its query rows
    // loaded when the current one starts, so a unit boundary costs the
    // epilogue and no refill of the pipeline.
    __device__ static void run(const AttnParams &p, const int *s_pre, int64_t begin, int64_t end, int w,
                               int64_t ptot, Arrivals &arr) {
        const int lane = threadIdx.x;
        const int n = lane & 15;
        const int kq = lane >> 4;
        Cur c;
        head(p, locate(p, s_pre, begin, end), c);
        Cur nx = c;   // the next segment, once there is one
        uint4 q[NB][KS];
        load_q(p, c.s.b, c.s.g, n, kq, q);
        PageRegs ring[2];
        load_block(p, ld_meta(c.pt, c.s.j0), true, c.s.g, n, kq, ring[0]);
        bool more = c.s.next < end;
        State st;
        start(p, c, q, st, n);
        if (more) {
            head(p, locate(p, s_pre, c.s.next, end), nx);
            load_q(p, nx.s.b, nx.s.g, n, kq, q);
        }
        int slot_id = 2 * w;
        int j = c.s.j0;
        while (true) {
#pragma unroll
            for (int k = 0; k < 2; k++) {
                // The next page of the range goes into the other ring slot,
                // loaded unconditionally (after the range's last page: nothing).
                const bool last = j + 1 == c.s.j1;
                const bool to_next = last && more;
                const int32_t *tpt = to_next ? nx.pt : c.pt;
                const int tj = to_next ? nx.s.j0 : min(j + 1, c.s.j1 - 1);
                load_block(p, ld_meta(tpt, tj), !last || more, to_next ? nx.s.g : c.s.g, n, kq, ring[1 - k]);
                page_step(p, st, ring[k], j, c.full_end, c.seg_end_tok, kq);
                if (last) {
                    finish(p, c, st, slot_id, ptot, n, kq);
                    arr.add(p, c.s);
                    if (!more)
                        return;
                    slot_id = 2 * w + 1;
                    c = nx;
                    j = c.s.j0;
                    more = c.s.next < end;
                    start(p, c, q, st, n);
                    if (more) {
                        head(p, locate(p, s_pre, c.s.next, end), nx);
                        load_q(p, nx.s.b, nx.s.g, n, kq, q);
                    }
                } else {
                    j++;
                }
            }
        }
    }
};

template <int D, int NB>
__global__ __launch_bounds__(64) void verify_kernel(AttnParams p) {
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
    if constexpr (NB == 1) {
        if (begin < end)
            Verify<D, NB>::run(p, s_pre, begin, end, w, ptot, arr);
    } else {
        for (int64_t x = begin; x < end;) {
            const Segment s = locate(p, s_pre, x, end);
            Verify<D, NB>::segment(p, s, x == begin ? 2 * w : 2 * w + 1, ptot);
            arr.add(p, s);
            x = s.next;
        }
    }
    arr.flush<false>(p);
}

}  // namespace

typedef void (*kernel_fn)(AttnParams);

kernel_fn verify_variant(int D, int NB) {
#define TS_VF(DD, NN) \
    if (D == DD && NB == NN) return verify_kernel<DD, NN>;
    TS_VF(64, 1) TS_VF(64, 2) TS_VF(64, 3) TS_VF(64, 4)
    TS_VF(128, 1) TS_VF(128, 2) TS_VF(128, 3) TS_VF(128, 4)
#undef TS_VF
    return nullptr;
}

}  // namespace tsattn
