// attn_verify_team.hip -- speculative-verify attention (head_dim 128) by a
// team of four wavefronts that share each KV page through LDS.
//
// Rows.  The G query heads of a KV group times the Qmax draft rows form
// R = G * Qmax rows per (sequence, KV head) unit, in NBE blocks of 16
// (NBE = 1, 2 or 4; R padded up).  Row r is draft position r / G of query
// head g * G + r % G.  A group is PS * PPW consecutive pages, PS = 4 / NBE;
// wave w owns row block w % NBE of pages (w / NBE) * PPW + 0 .. PPW - 1 of
// it.  With 64 rows the four waves split the rows of two pages (two
// independent chains per wave and barrier), with 16 rows they take a page
// each.
// A workgroup is one worker of the stream-K partition (attn_common.h), or,
// from workgroup W on, a merge workgroup of the launch (attn_split.h).
//
// Staging.  A page is loaded as eight 1 KiB pieces, one 16-byte piece per
// lane, through a buffer resource bounded to the page's block (so a group
// past the segment end reads nothing).  Wave w loads K rows 4 w .. 4 w + 3
// whole (1 KiB contiguous, so each 128-byte line is fetched by one load) and
// scatters them into four K slabs (slab s holds, for consumer lane
// l = 16 kq + n, key row n dims 32 s + 8 kq .. + 7: the A operand of the
// score product, stored in lane order with the 16-byte chunk index swizzled
// so that the scattered writes and the reads are free of bank conflicts) and
// four V slabs (slab i: value row 4 kq + i, dims 8 n .. 8 n + 7), stored as
// the page's 16 value rows in natural order with a 288-byte row pitch.  The four
// waves split the loading; loads run kDepth groups ahead in registers, are
// written into one of two LDS stages, and one barrier per page group
// separates writing a stage from reading it.
//
// Value operand.  gfx950's LDS transpose read (ds_read_b64_tr_b16) hands lane
// i' of each 16-lane group element i' % 4 of the 8-byte chunk addressed by
// lane 4k + i' / 4 of that group, as element k.  So if lane (n, kq) addresses
// value row 4 kq + n / 4, dims 16 jj + 4 (n % 4) .. + 3, every lane receives
// rows 4 kq .. 4 kq + 3 of dim 16 jj + n: exactly the B operand of the j-th
// P.V product, with no register shuffles.  With the 288-byte pitch the 16
// lanes of a group touch 32 distinct banks.

// Math per page and row block (l = lane, n = l % 16, kq = l / 16):
//   S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (lane gets tokens 4kq..4kq+3 of
//   row n); P = exp2(scale log2e S - m_ref) packed to bf16 in the same lane
//   is the A operand of O += P V on v_mfma_f32_16x16x16_bf16 (product jj
//   covers dims 16 jj .. 16 jj + 15); row sums are P times a ones operand;
//   m_ref is raised only when a score exceeds it by more than 8 (log2 units).
//   Pages that need no mask (all but the last one or two of a sequence) take
//   a path without any per-token selects.
// At the end of a segment the PS waves of a row block merge their running
// states through LDS with log-sum-exp weights; the first one writes.
// Masks: key t is visible to draft row i iff t <= L - Q + i; keys past the
// segment or context end get probability 0 and zeroed value rows.
#include "attn_split.h"

#include <type_traits>

namespace tsattn {

namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t u) { return __builtin_bit_cast(bf16x8_t, u); }
__device__ __forceinline__ u32x4_t ld16(const void *p) { return *reinterpret_cast<const u32x4_t *>(p); }
__device__ __forceinline__ s16x4_t as_s16x4(uint2 u) { return __builtin_bit_cast(s16x4_t, u); }

// Calls f(std::integral_constant<int, I>) for I = B .. E - 1 (compile-time).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// Wait for this wave's LDS operations, then meet the other waves.
// Release/acquire fences limited to LDS keep outstanding global prefetches in
// flight across the barrier (only lgkmcnt is waited for).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

constexpr int kD = 128;
constexpr int kSlab = 1024;               // bytes per K slab
constexpr int kVPitch = 288;              // bytes per value row in LDS
constexpr int kVOff = 4 * kSlab;          // value rows follow the K slabs
constexpr int kPageLds = kVOff + kPage * kVPitch;   // one staged page
constexpr int kTeam = 4;                  // wavefronts per workgroup
constexpr int kBlockBytes = kPage * kD * 2;   // one (page, KV head) block

template <int NBE>
struct Team {
    static constexpr int PS = kTeam / NBE;        // page splits across the waves
    static constexpr int PPW = NBE == 4 ? 2 : 1;  // pages per wave per group
    static constexpr int GP = PS * PPW;           // pages per group
    static constexpr int SLABS = 8 * GP;          // slabs per group
    static constexpr int PER_WAVE = SLABS / kTeam;  // slabs each wave loads per group
    static constexpr int STAGE = GP * kPageLds;   // LDS bytes per stage
    static constexpr int kDepth = NBE == 2 ? 4 : 2;  // groups in flight in registers

    struct Regs {
        u32x4_t s[PER_WAVE];
    };
    // kDepth register sets addressed only by compile-time index.
    struct Ring {
        Regs r0, r1, r2, r3, r4, r5, r6, r7;
        template <int K>
        __device__ __forceinline__ Regs &at() {
            static_assert(K >= 0 && K < 8, "ring slot");
            if constexpr (K == 0) return r0;
            else if constexpr (K == 1) return r1;
            else if constexpr (K == 2) return r2;
            else if constexpr (K == 3) return r3;
            else if constexpr (K == 4) return r4;
            else if constexpr (K == 5) return r5;
            else if constexpr (K == 6) return r6;
            else return r7;
        }
    };

    // Issue this wave's loads of group `grp` (pages j0 + grp * GP + q): K slab
    // `wave` and V slab `wave` of each page, i.e. slots tau = wave + 4 t with
    // t = 2 q (K) and t = 2 q + 1 (V).  Loads go through a buffer resource
    // bounded to the page's block; for a page past the segment it has no
    // records, so the loads read nothing and yield zeros (no branch, no
    // re-read of the last page).
    __device__ __forceinline__ static void load_group(const AttnParams &p, const int32_t *pt, int g, int j0, int j1,
                                      int grp, int wave, int lane, Regs &r) {
        const int n = lane & 15, kq = lane >> 4;
#pragma unroll
        for (int q = 0; q < GP; q++) {
            const int j = j0 + grp * GP + q;
            const bool in = j < j1;
            const int pid = ld_meta(pt, in ? j : j1 - 1);
            const size_t base = ((size_t)pid * p.Hkv + g) * (size_t)(kPage * kD);
            const block_rsrc_t rk = block_rsrc(p.k_pages + base, in ? kBlockBytes : 0);
            const block_rsrc_t rv = block_rsrc(p.v_pages + base, in ? kBlockBytes : 0);
            // K rows 4 wave .. 4 wave + 3 whole (1 KiB contiguous per load):
            // lane l holds row 4 wave + l / 16, dims 8 (l % 16) .. + 7
            r.s[2 * q] = ld_block16(rk, 2 * ((4 * wave + kq) * kD + 8 * n));
            r.s[2 * q + 1] = ld_block16(rv, 2 * ((4 * kq + wave) * kD + 8 * n));
        }
    }

    // Where 16-byte chunk C of a page's K slabs is stored (C = 64 slab +
    // consumer lane): its low four bits are XORed with the next four, so that
    // both the scattered writes below and the consumers' reads touch sixteen
    // distinct bank groups per sixteen lanes.
    __device__ __forceinline__ static int k_chunk(int C) { return C ^ ((C >> 4) & 15); }

    // Writes the wave's loads of a group into a stage.  A K piece (row rho =
    // 4 wave + kq, 8-dim chunk c = n) goes where the score product's A operand
    // wants it: slab c / 4, consumer lane 16 (c % 4) + rho (swizzled).  A V
    // piece (row 4 kq + wave, dims 8 n .. + 7) goes to its row in natural order.
    __device__ __forceinline__ static void store_group(char *stage, int wave, int lane, const Regs &r) {
        const int n = lane & 15, kq = lane >> 4;
        const int k_off = k_chunk(64 * (n >> 2) + 16 * (n & 3) + 4 * wave + kq) * 16;
        const int v_off = kVOff + (4 * kq + wave) * kVPitch + 16 * n;
#pragma unroll
        for (int t = 0; t < PER_WAVE; t++) {
            char *pg = stage + (t >> 1) * kPageLds;
            *reinterpret_cast<u32x4_t *>(pg + ((t & 1) ? v_off : k_off)) = r.s[t];
        }
    }

    struct State {
        u32x4_t qf[4];
        int lim;
        f32x4_t acc[8];
        f32x4_t lacc;
        float m_ref;
    };

    // One page for this wave's row block.  `masked` (wavefront-uniform) is set
    // only for the last page or two of a sequence; elsewhere no per-token
    // select is executed.
    __device__ __forceinline__ static void page_step(const AttnParams &p, State &st, const char *pg, int j,
                                                     bool masked, int seg_end_tok, int lane) {
        const int n = lane & 15, kq = lane >> 4;
        u32x4_t kf[4];
#pragma unroll
        for (int s = 0; s < 4; s++)
            kf[s] = ld16(pg + k_chunk(64 * s + lane) * 16);
        // transpose-read address of this lane for product jj: + 32 jj bytes
        typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;
        const char *vbase = pg + kVOff + (4 * kq + (n >> 2)) * kVPitch + 8 * (n & 3);
        s16x4_t vt[8];
#pragma unroll
        for (int jj = 0; jj < 8; jj++)
            vt[jj] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_s16x4 *)(__attribute__((address_space(3))) const char *)(vbase + 32 * jj));

        f32x4_t sc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 4; s++)
            sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[s]), as_bf16x8(st.qf[s]), sc, 0, 0, 0);
        float x[4];
#pragma unroll
        for (int e = 0; e < 4; e++)
            x[e] = sc[e] * p.scale_log2;
        const int t0 = j * kPage;
        if (masked) {
            // invisible keys score -inf; keys past the segment or context end
            // also get zeroed value rows (stale data may be NaN, and 0 * NaN
            // would poison the product)
            s16x4_t keep;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                keep[e] = (t0 + 4 * kq + e < seg_end_tok) ? (short)-1 : (short)0;
                x[e] = (t0 + 4 * kq + e < st.lim) ? x[e] : -INFINITY;
            }
#pragma unroll
            for (int jj = 0; jj < 8; jj++)
                vt[jj] &= keep;
        }
        // Lane-local check first: the row maximum (a cross-lane reduction over the
        // four lanes of a row) is only needed when some score exceeds its row's
        // reference by more than the slack, which is rare after the first page.
        float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
        if (__any(mx > st.m_ref + kRescaleSlack)) {
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const bool up = mx > st.m_ref + kRescaleSlack;
            const float alpha = up ? fast_exp2(st.m_ref - mx) : 1.0f;
            st.m_ref = up ? mx : st.m_ref;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const float ai = __shfl(alpha, 4 * kq + i);
                st.lacc[i] *= ai;
#pragma unroll
                for (int jj = 0; jj < 8; jj++)
                    st.acc[jj][i] *= ai;
            }
        }
        float pr[4];
#pragma unroll
        for (int e = 0; e < 4; e++)
            pr[e] = fast_exp2(x[e] - st.m_ref);
        if (masked) {
            // a row with no visible key yet keeps m_ref = -inf: -inf - -inf
#pragma unroll
            for (int e = 0; e < 4; e++)
                pr[e] = x[e] == -INFINITY ? 0.0f : pr[e];
        }
        const s16x4_t pa = as_s16x4(make_uint2(pack_bf16x2(pr[0], pr[1]), pack_bf16x2(pr[2], pr[3])));
        const uint2 ones = make_uint2(0x3F803F80u, 0x3F803F80u);
        st.lacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, as_s16x4(ones), st.lacc, 0, 0, 0);
#pragma unroll
        for (int jj = 0; jj < 8; jj++)
            st.acc[jj] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, vt[jj], st.acc[jj], 0, 0, 0);
    }

    // Per-wave merge record in LDS (for waves po > 0).
    struct Rec {
        float acc[8][4][64];    // [jj][i][lane]
        float lacc[4][64];
        float m[16];
    };

    __device__ __forceinline__ static void segment(const AttnParams &p, const Segment &s, int slot_id, char *lds) {
        const int lane = threadIdx.x & 63;
        const int wave = first_lane_int(threadIdx.x >> 6);   // uniform within the wavefront
        const int n = lane & 15, kq = lane >> 4;
        const int po = wave / NBE, rb = wave % NBE;
        const int b = s.b, g = s.g;
        const int G = p.G;
        const int L = ld_meta(p.ctx_lens, b);
        const int Q = ld_meta(p.q_lens, b);
        const int R = p.rows_per_unit;
        const int32_t *pt = p.page_table + (size_t)b * p.max_pages;
        const int seg_end_tok = min(L, s.j1 * kPage);
        const int full_end = min(L - Q + 1, seg_end_tok);

        State st;
        {
            const int r = rb * 16 + n;
            const bool row_ok = r < R && r / G < Q;
            const int i = row_ok ? r / G : 0;
            const int hl = row_ok ? r % G : 0;
            st.lim = min(row_ok ? L - Q + i + 1 : L, seg_end_tok);
            const uint16_t *qr = p.q + (((size_t)b * p.Qmax + i) * p.Hq + (size_t)g * G + hl) * kD + 8 * kq;
#pragma unroll
            for (int ks = 0; ks < 4; ks++)
                st.qf[ks] = row_ok ? ld16(qr + 32 * ks) : u32x4_t{0u, 0u, 0u, 0u};
            st.m_ref = -INFINITY;
            st.lacc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int jj = 0; jj < 8; jj++)
                st.acc[jj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }

        const int ngroups = (s.j1 - s.j0 + GP - 1) / GP;
        Ring ring;
        static_for<0, kDepth>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            load_group(p, pt, g, s.j0, s.j1, k, wave, lane, ring.template at<k>());
        });
        // group 0 into stage 0
        store_group(lds, wave, lane, ring.template at<0>());
        load_group(p, pt, g, s.j0, s.j1, kDepth, wave, lane, ring.template at<0>());
        lds_barrier();

        for (int it0 = 0; it0 < ngroups; it0 += kDepth) {
            static_for<0, kDepth>([&](auto kc) {
                constexpr int k = decltype(kc)::value;
                constexpr int nk = (k + 1) % kDepth;   // ring slot of group it + 1
                const int it = it0 + k;
                if (it < ngroups) {
                    store_group(lds + ((it + 1) & 1) * STAGE, wave, lane, ring.template at<nk>());
                    load_group(p, pt, g, s.j0, s.j1, it + 1 + kDepth, wave, lane, ring.template at<nk>());
#pragma unroll
                    for (int pp = 0; pp < PPW; pp++) {
                        const int q = po * PPW + pp;          // page within the group
                        const int j = s.j0 + it * GP + q;
                        if (j < s.j1)
                            page_step(p, st, lds + (it & 1) * STAGE + q * kPageLds, j,
                                      (j + 1) * kPage > full_end, seg_end_tok, lane);
                    }
                    lds_barrier();
                }
            });
        }

        // merge the PS page groups of each row block through LDS
        if constexpr (PS > 1) {
            Rec *rec = reinterpret_cast<Rec *>(lds);
            if (po > 0) {
                Rec &m = rec[(po - 1) * NBE + rb];
#pragma unroll
                for (int jj = 0; jj < 8; jj++)
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        m.acc[jj][i][lane] = st.acc[jj][i];
#pragma unroll
                for (int i = 0; i < 4; i++)
                    m.lacc[i][lane] = st.lacc[i];
                if (kq == 0)
                    m.m[n] = st.m_ref;
            }
            lds_barrier();
            if (po == 0) {
                float mrow[4], M[4];
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    mrow[i] = __shfl(st.m_ref, 4 * kq + i);
                    M[i] = mrow[i];
                }
#pragma unroll
                for (int q = 1; q < PS; q++) {
                    const Rec &m = rec[(q - 1) * NBE + rb];
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        M[i] = fmaxf(M[i], m.m[4 * kq + i]);
                }
                float a0[4];
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    a0[i] = mrow[i] == -INFINITY ? 0.0f : fast_exp2(mrow[i] - M[i]);
                    st.lacc[i] *= a0[i];
#pragma unroll
                    for (int jj = 0; jj < 8; jj++)
                        st.acc[jj][i] *= a0[i];
                }
#pragma unroll
                for (int q = 1; q < PS; q++) {
                    const Rec &m = rec[(q - 1) * NBE + rb];
#pragma unroll
                    for (int i = 0; i < 4; i++) {
                        const float mq = m.m[4 * kq + i];
                        const float aq = mq == -INFINITY ? 0.0f : fast_exp2(mq - M[i]);
                        st.lacc[i] += aq * m.lacc[i][lane];
#pragma unroll
                        for (int jj = 0; jj < 8; jj++)
                            st.acc[jj][i] += aq * m.acc[jj][i][lane];
                    }
                }
                write_out(p, st, M, s, slot_id, rb, lane);
            }
            lds_barrier();
        } else {
            float M[4];
#pragma unroll
            for (int i = 0; i < 4; i++)
                M[i] = __shfl(st.m_ref, 4 * kq + i);
            write_out(p, st, M, s, slot_id, rb, lane);
            lds_barrier();
        }
    }

    // Rows 16 rb + 4 kq + i, dims 16 jj + n (jj = 0..7) of the merged state.
    __device__ __forceinline__ static void write_out(const AttnParams &p, const State &st, const float (&M)[4],
                                                     const Segment &s, int slot_id, int rb, int lane) {
        const int n = lane & 15, kq = lane >> 4;
        const int G = p.G, R = p.rows_per_unit, Q = ld_meta(p.q_lens, s.b);
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const int r = rb * 16 + 4 * kq + i;
            const int di = r / G;
            if (r >= R || di >= Q)
                continue;
            const float l = st.lacc[i];
            const float inv = l > 0.0f ? 1.0f / l : 0.0f;
            if (s.whole) {
                uint16_t *dst = p.out + (((size_t)s.b * p.Qmax + di) * p.Hq + (size_t)s.g * G + r % G) * kD + n;
#pragma unroll
                for (int jj = 0; jj < 8; jj++)
                    dst[16 * jj] = to_bf16(st.acc[jj][i] * inv);
            } else {
                const size_t row = (size_t)slot_id * R + r;
                const float lse = l > 0.0f ? M[i] + __log2f(l) : -INFINITY;
                if (p.combine != kCombineKernel) {
                    // device-coherent: merge workgroups of this launch read them
#pragma unroll
                    for (int jj = 0; jj < 8; jj++)
                        st_partial4(p, row * kD + 16 * jj + n, st.acc[jj][i] * inv);
                    if (n == 0)
                        st_coherent(p.ws_lse + row, lse);
                } else {
                    float *dst = p.ws_o + row * kD + n;
#pragma unroll
                    for (int jj = 0; jj < 8; jj++)
                        dst[16 * jj] = st.acc[jj][i] * inv;
                    if (n == 0)
                        p.ws_lse[row] = lse;
                }
            }
        }
    }
};

// LDS bytes a team of NBE row blocks needs beyond the sequence prefix.
template <int NBE>
constexpr int team_lds() {
    constexpr int stages = 2 * Team<NBE>::STAGE;
    constexpr int recs = (Team<NBE>::PS - 1) * NBE * (int)sizeof(typename Team<NBE>::Rec);
    return stages > recs ? stages : recs;
}

template <int NBE>
__global__ __launch_bounds__(256) void verify_team_kernel(AttnParams p) {
    extern __shared__ int s_pre[];
    page_prefix(p, s_pre);
    char *lds = reinterpret_cast<char *>(s_pre) + (((p.B + 1) * 4 + 15) & ~15);
    if (__builtin_expect((int)blockIdx.x >= p.W, 0)) {   // merge workgroups, laid out after the workers' code
        const int m = (int)blockIdx.x - p.W, ngroups = (p.rows_per_unit + 3) / 4;
        merge_in_launch<kD>(p, s_pre, m / ngroups, 4 * (m % ngroups) + (int)(threadIdx.x >> 6));
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
        Team<NBE>::segment(p, s, x == begin ? 2 * w : 2 * w + 1, lds);
        arr.add(p, s);
        x = s.next;
    }
    arr.flush<true>(p);
}

}  // namespace

typedef void (*kernel_fn)(AttnParams);

// Kernel and its LDS need (beyond the prefix) for R = G * Qmax rows, head_dim 128.
kernel_fn verify_team_variant(int rows, int *lds_bytes, int *nbe) {
    if (rows <= 16) {
        *nbe = 1;
        *lds_bytes = team_lds<1>();
        return verify_team_kernel<1>;
    }
    if (rows <= 32) {
        *nbe = 2;
        *lds_bytes = team_lds<2>();
        return verify_team_kernel<2>;
    }
    *nbe = 4;
    *lds_bytes = team_lds<4>();
    return verify_team_kernel<4>;
}

}  // namespace tsattn
