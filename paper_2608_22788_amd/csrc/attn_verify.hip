// attn_verify.hip -- paged speculative-verify attention: each sequence
// brings q_len = 1 + gamma query rows (the draft block) that attend to the
// whole cache and causally to each other, on bf16 matrix cores.
//
// The G query heads of a KV group times the q_len draft rows form
// R = G * Qmax rows per (sequence, KV head) unit, padded to NB blocks of 16;
// row r is draft position i = r / G of query head g * G + r % G.  One
// wavefront streams the unit's pages two at a time (32 tokens) and keeps
// every row block in registers, so each K/V byte is read once for all rows.
//
// With l = lane, n = l % 16, kq = l / 16, and v_mfma_f32_16x16x32_bf16
// operand layouts (A: row l%16, k 8(l/16)..+7; B: col l%16, k 8(l/16)..+7;
// C: row 4(l/16)+i, col l%16):
//   * scores S^T = K Q^T per page: A = 16 key rows x 32 dims loaded straight
//     from the page (16 bytes per lane), B = Q^T kept in registers.  Lane
//     (n, kq) receives tokens 4kq..4kq+3 of the page for query row n;
//   * probabilities P = exp2(scale*log2e * S - m_ref) are packed to bf16 in
//     the lane that computed them and used directly as the A operand of
//     O = P V, with the contraction index k = 8kq + e standing for token
//     16(e/4) + 4kq + e%4 of the page pair;
//   * V is loaded as rows (lane (n, kq) reads D/16 consecutive dims of its 8
//     tokens) and transposed in registers with byte permutes, so the B
//     operand of the j-th P.V product holds dims (D/16) n + j;
//   * row sums come from one more product of P with a ones operand, so they
//     use exactly the rounded probabilities that weight V;
//   * the running reference m_ref of each row is only raised when a score
//     exceeds it by more than 8 in log2 units, which leaves the accumulators
//     untouched on almost every page pair.
// Masks: key t is visible to draft row i iff t <= L - Q + i; keys past the
// segment end or the context end get probability 0 and their value rows are
// zeroed before the product, so stale data never reaches the output.
#include "attn_common.h"

namespace tsattn {

namespace {

template <int D>
struct VerifyTypes {
    static constexpr int KS = D / 32;   // k-steps of the score product
    static constexpr int VE = D / 16;   // value dims per lane (= P.V products per row block)
};

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

template <int VE>
struct VRow;
template <>
struct VRow<8> {
    uint32_t w[4];
    __device__ void load(const uint16_t *p) {
        uint4 t = *reinterpret_cast<const uint4 *>(p);
        w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
    }
    __device__ void zero() { w[0] = w[1] = w[2] = w[3] = 0; }
};
template <>
struct VRow<4> {
    uint32_t w[2];
    __device__ void load(const uint16_t *p) {
        uint2 t = *reinterpret_cast<const uint2 *>(p);
        w[0] = t.x; w[1] = t.y;
    }
    __device__ void zero() { w[0] = w[1] = 0; }
};

template <int D, int NB>
struct Verify {
    static constexpr int KS = VerifyTypes<D>::KS;
    static constexpr int VE = VerifyTypes<D>::VE;

    struct PairRegs {
        uint4 k[2][KS];        // A operands of the score product, per page
        VRow<VE> v[2][4];      // value rows of the lane's 8 tokens
    };

    __device__ static void load_pair(const AttnParams &p, const int32_t *pt, int jp, bool has2,
                                     int g, int n, int kq, PairRegs &r) {
#pragma unroll
        for (int pg = 0; pg < 2; pg++) {
            if (pg == 1 && !has2) {
#pragma unroll
                for (int s = 0; s < KS; s++)
                    r.k[1][s] = make_uint4(0, 0, 0, 0);
#pragma unroll
                for (int i = 0; i < 4; i++)
                    r.v[1][i].zero();
                continue;
            }
            const int pid = pt[jp + pg];
            const size_t base = ((size_t)pid * p.Hkv + g) * (size_t)(kPage * D);
            const uint16_t *kb = p.k_pages + base + (size_t)n * D + 8 * kq;
#pragma unroll
            for (int s = 0; s < KS; s++)
                r.k[pg][s] = *reinterpret_cast<const uint4 *>(kb + 32 * s);
            const uint16_t *vb = p.v_pages + base + (size_t)(4 * kq) * D + VE * n;
#pragma unroll
            for (int i = 0; i < 4; i++)
                r.v[pg][i].load(vb + (size_t)i * D);
        }
    }

    // Element e (0..VE-1) of a VE-wide bf16 row held in dwords.
    __device__ static uint32_t half_of(const VRow<VE> &v, int e) {
        const uint32_t w = v.w[e >> 1];
        return (e & 1) ? (w >> 16) : (w & 0xffffu);
    }

    __device__ static void segment(const AttnParams &p, const Segment &s, int slot_id) {
        const int lane = threadIdx.x;
        const int n = lane & 15;
        const int kq = lane >> 4;
        const int b = s.b, g = s.g;
        const int G = p.G;
        const int L = p.ctx_lens[b];
        const int Q = p.q_lens[b];
        const int R = p.rows_per_unit;
        const int32_t *pt = p.page_table + (size_t)b * p.max_pages;
        const int seg_end_tok = min(L, s.j1 * kPage);

        // query fragments (B operand of the score product) and causal limits
        uint4 qf[NB][KS];
        int lim[NB];
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            const int r = rb * 16 + n;
            const bool row_ok = r < R && r / G < Q;
            const int i = row_ok ? r / G : 0;
            const int hl = row_ok ? r % G : 0;
            lim[rb] = min(row_ok ? L - Q + i + 1 : L, seg_end_tok);
            const uint16_t *qr = p.q + (((size_t)b * p.Qmax + i) * p.Hq + (size_t)g * G + hl) * D + 8 * kq;
#pragma unroll
            for (int ks = 0; ks < KS; ks++)
                qf[rb][ks] = row_ok ? *reinterpret_cast<const uint4 *>(qr + 32 * ks) : make_uint4(0, 0, 0, 0);
        }
        // keys below this bound are visible to every row of the block
        const int full_end = min(L - Q + 1, seg_end_tok);

        f32x4_t acc[NB][VE];
        f32x4_t lacc[NB];
        float m_ref[NB];
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            m_ref[rb] = -INFINITY;
            lacc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int jj = 0; jj < VE; jj++)
                acc[rb][jj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        const uint4 ones4 = make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u);

        PairRegs cur, nxt;
        load_pair(p, pt, s.j0, s.j0 + 1 < s.j1, g, n, kq, cur);
        for (int jp = s.j0; jp < s.j1; jp += 2) {
            if (jp + 2 < s.j1)
                load_pair(p, pt, jp + 2, jp + 3 < s.j1, g, n, kq, nxt);
            const int t0 = jp * kPage;                   // first token of the pair
            const bool masked = t0 + 2 * kPage > full_end;  // wavefront-uniform

            // value rows of keys past the segment / context end become 0
            if (t0 + 2 * kPage > seg_end_tok) {
#pragma unroll
                for (int pg = 0; pg < 2; pg++)
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        if (t0 + 16 * pg + 4 * kq + i >= seg_end_tok)
                            cur.v[pg][i].zero();
            }

            // transpose the lane's 8 value rows: vt[jj] = dim (VE n + jj) of tokens k = 0..7
            uint4 vt[VE];
#pragma unroll
            for (int jj = 0; jj < VE; jj++) {
                uint32_t w[4];
#pragma unroll
                for (int q2 = 0; q2 < 4; q2++) {
                    const int pg = q2 >> 1, i0 = 2 * (q2 & 1);
                    w[q2] = half_of(cur.v[pg][i0], jj) | (half_of(cur.v[pg][i0 + 1], jj) << 16);
                }
                vt[jj] = make_uint4(w[0], w[1], w[2], w[3]);
            }

#pragma unroll
            for (int rb = 0; rb < NB; rb++) {
                f32x4_t sc[2];
#pragma unroll
                for (int pg = 0; pg < 2; pg++) {
                    sc[pg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KS; ks++)
                        sc[pg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.k[pg][ks]),
                                                                         as_bf16x8(qf[rb][ks]), sc[pg], 0, 0, 0);
                }
                float x[8];
                bool ok[8];
#pragma unroll
                for (int e = 0; e < 8; e++) {
                    x[e] = sc[e >> 2][e & 3] * p.scale_log2;
                    ok[e] = !masked || (t0 + 16 * (e >> 2) + 4 * kq + (e & 3) < lim[rb]);
                }
                float mx = -INFINITY;
#pragma unroll
                for (int e = 0; e < 8; e++)
                    mx = fmaxf(mx, ok[e] ? x[e] : -INFINITY);
                mx = fmaxf(mx, __shfl_xor(mx, 16));
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const bool up = mx > m_ref[rb] + kRescaleSlack;
                if (__any(up)) {
                    const float alpha = up ? fast_exp2(m_ref[rb] - mx) : 1.0f;
                    m_ref[rb] = up ? mx : m_ref[rb];
#pragma unroll
                    for (int i = 0; i < 4; i++) {
                        const float ai = __shfl(alpha, 4 * kq + i);
                        lacc[rb][i] *= ai;
#pragma unroll
                        for (int jj = 0; jj < VE; jj++)
                            acc[rb][jj][i] *= ai;
                    }
                }
                uint32_t pw[4];
#pragma unroll
                for (int q2 = 0; q2 < 4; q2++) {
                    const int e0 = 2 * q2, e1 = 2 * q2 + 1;
                    const float p0 = ok[e0] ? fast_exp2(x[e0] - m_ref[rb]) : 0.0f;
                    const float p1 = ok[e1] ? fast_exp2(x[e1] - m_ref[rb]) : 0.0f;
                    pw[q2] = pack_bf16x2(p0, p1);
                }
                const bf16x8_t pa = as_bf16x8(make_uint4(pw[0], pw[1], pw[2], pw[3]));
                lacc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, as_bf16x8(ones4), lacc[rb], 0, 0, 0);
#pragma unroll
                for (int jj = 0; jj < VE; jj++)
                    acc[rb][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, as_bf16x8(vt[jj]), acc[rb][jj], 0, 0, 0);
            }
            cur = nxt;
        }

        // epilogue: lane holds rows 16 rb + 4 kq + i, dims VE n .. VE n + VE - 1
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int r = rb * 16 + 4 * kq + i;
                const float m = __shfl(m_ref[rb], 4 * kq + i);
                const float l = lacc[rb][i];
                const int di = r / G;
                if (r >= R || di >= Q)
                    continue;
                const float inv = l > 0.0f ? 1.0f / l : 0.0f;
                if (s.whole) {
                    uint16_t *dst = p.out + (((size_t)b * p.Qmax + di) * p.Hq + (size_t)g * G + r % G) * D + VE * n;
                    uint32_t w[VE / 2];
#pragma unroll
                    for (int e = 0; e < VE / 2; e++)
                        w[e] = pack_bf16x2(acc[rb][2 * e][i] * inv, acc[rb][2 * e + 1][i] * inv);
                    if constexpr (VE == 8)
                        *reinterpret_cast<uint4 *>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
                    else
                        *reinterpret_cast<uint2 *>(dst) = make_uint2(w[0], w[1]);
                } else {
                    const size_t row = (size_t)slot_id * R + r;
                    float *dst = p.ws_o + row * D + VE * n;
#pragma unroll
                    for (int e = 0; e < VE; e += 4)
                        *reinterpret_cast<float4 *>(dst + e) =
                            make_float4(acc[rb][e][i] * inv, acc[rb][e + 1][i] * inv,
                                        acc[rb][e + 2][i] * inv, acc[rb][e + 3][i] * inv);
                    if (n == 0)
                        p.ws_lse[row] = l > 0.0f ? m + __log2f(l) : -INFINITY;
                }
            }
        }
    }
};

template <int D, int NB>
__global__ __launch_bounds__(64) void verify_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    const int64_t ptot = (int64_t)p.Hkv * s_pre[p.B];
    const int w = blockIdx.x;
    const int64_t begin = worker_begin(ptot, w, p.W);
    const int64_t end = worker_begin(ptot, w + 1, p.W);
    for (int64_t x = begin; x < end;) {
        const Segment s = locate(p, s_pre, x, end);
        Verify<D, NB>::segment(p, s, x == begin ? 2 * w : 2 * w + 1);
        x = s.next;
    }
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
