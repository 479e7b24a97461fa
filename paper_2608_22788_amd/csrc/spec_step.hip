// spec_step.hip -- the two steps around the verify attention in one
// speculative decoding step (paper Sec. 3.4: drafts are verified by the
// target model, losslessly, following the speculative sampling of Leviathan
// et al.):
//
//   * KV append: the step's 1 + gamma new tokens' key and value rows are
//     written into the paged pool before the attention reads them (the
//     attention's context length counts them).  One thread per 16-byte piece
//     of a row; HBM-bound and tiny.
//
//   * acceptance: per sequence, walk the drafts while u_i * q_i(d_i) <=
//     p_i(d_i); at the first rejection k draw the next token from the
//     leftover mass max(0, p_k - q_k), after full acceptance from the bonus
//     row p_gamma, by inverse CDF with the caller's uniform.  The rule is
//     stated over real numbers and is evaluated here without rounding: the
//     test u q <= p on float64 products (exact for float32 factors), and the
//     weights and their running sums as integers in units of 2^-149, the
//     smallest float32, held in three 64-bit words (Fx below).  So the result
//     does not depend on the order of the sums, and the parallel evaluation
//     gives exactly the sequential one.  The sampling row is a full
//     vocabulary of fp32 probabilities per sequence, so the work is a
//     streaming read of one or two rows:
//       - accept_blocks_kernel: every 256-element block of every sequence's
//         sampling row is summed by one wavefront (a float4 per lane, then a
//         butterfly), so the whole chip shares the read even for a handful
//         of sequences;
//       - accept_pick_kernel: one wavefront per sequence scans the block sums
//         (lane runs of consecutive blocks, a wavefront scan of the run
//         totals), finds the block where the cumulative mass first exceeds
//         floor(u * total), and scans that block's 256 elements.
//     Both kernels recompute the acceptance walk (2 gamma scalar loads)
//     rather than pass it through memory.
//   Readings: probabilities are clamped to [0, 1] and uniforms to
//   [0, 1 - 2^-24], NaN read as 0; a draft id outside [0, V) is rejected; if
//   the leftover mass is zero the next token is drawn from p_k itself; a
//   sampling row without mass gives token -1.
#include <hip/hip_runtime.h>

#include <climits>

#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {

namespace {

constexpr int kWave = 64;
constexpr int kBlk = 256;          // vocabulary elements per block (float4 per lane)
constexpr int kPickThreads = 64;   // pick workgroup: one wavefront

struct AppendParams {
    const uint16_t *k_new, *v_new;   // [B][Qmax][Hkv][D]
    uint16_t *k_pages, *v_pages;     // [num_pages][Hkv][16][D]
    const int32_t *page_table, *ctx_lens, *q_lens;
    int64_t num_pages;
    int B, Qmax, Hkv, D, max_pages;
};

__global__ __launch_bounds__(256) void kv_append_kernel(AppendParams p) {
    const int chunks = p.D / 8;   // 16-byte pieces per row
    const int64_t total = (int64_t)p.B * p.Qmax * p.Hkv * chunks;
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= total)
        return;
    const int c = (int)(id % chunks);
    int64_t r = id / chunks;
    const int g = (int)(r % p.Hkv);
    r /= p.Hkv;
    const int i = (int)(r % p.Qmax);
    const int b = (int)(r / p.Qmax);
    const int Q = p.q_lens[b];
    if (i >= Q)
        return;
    const int t = p.ctx_lens[b] - Q + i;
    if (t < 0 || t >= p.max_pages * 16)
        return;   // violated precondition: write nothing rather than out of bounds
    const int page = p.page_table[(size_t)b * p.max_pages + t / 16];
    if (page < 0 || page >= p.num_pages)
        return;
    const size_t src = (((size_t)b * p.Qmax + i) * p.Hkv + g) * p.D + 8 * c;
    const size_t dst = (((size_t)page * p.Hkv + g) * 16 + t % 16) * p.D + 8 * c;
    *reinterpret_cast<uint4 *>(p.k_pages + dst) = *reinterpret_cast<const uint4 *>(p.k_new + src);
    *reinterpret_cast<uint4 *>(p.v_pages + dst) = *reinterpret_cast<const uint4 *>(p.v_new + src);
}

struct AcceptParams {
    const float *p;          // [B][G+1][V]
    const float *q;          // [B][G][V]
    const int32_t *draft;    // [B][G]
    const int32_t *num_draft;
    const float *u_accept;   // [B][G]
    const float *u_sample;   // [B]
    int32_t *n_accepted, *next_token;
    uint64_t *bsum;          // [B][2][nblk][3] exact block sums of the sampling row
    int32_t *walk;           // [B] drafts accepted, as the block-sum kernel found them
    int B, V, G, nblk;
};

// ---- exact fixed point --------------------------------------------------------
// A float32 in [0, 1] is an integer number of units of 2^-149 (the smallest
// positive subnormal), below 2^150 of them; a row of at most 2^31 such
// weights sums to below 2^181.  Fx holds such integers in three 64-bit words,
// so every sum and comparison below is exact and independent of order.
struct Fx {
    uint64_t w0, w1, w2;
};

__device__ __forceinline__ Fx fx_zero() { return Fx{0, 0, 0}; }

__device__ __forceinline__ Fx fx_add(Fx a, Fx b) {
    Fx r;
    r.w0 = a.w0 + b.w0;
    const uint64_t c0 = r.w0 < a.w0;
    const uint64_t t = a.w1 + b.w1;
    uint64_t c1 = t < a.w1;
    r.w1 = t + c0;
    c1 += r.w1 < t;
    r.w2 = a.w2 + b.w2 + c1;
    return r;
}

__device__ __forceinline__ bool fx_gt(Fx a, Fx b) {
    if (a.w2 != b.w2)
        return a.w2 > b.w2;
    if (a.w1 != b.w1)
        return a.w1 > b.w1;
    return a.w0 > b.w0;
}

__device__ __forceinline__ bool fx_is_zero(Fx a) { return (a.w0 | a.w1 | a.w2) == 0; }

// a - b for a > b.
__device__ __forceinline__ Fx fx_sub(Fx a, Fx b) {
    Fx r;
    r.w0 = a.w0 - b.w0;
    const uint64_t b0 = a.w0 < b.w0;
    const uint64_t t = a.w1 - b.w1;
    uint64_t b1 = a.w1 < b.w1;
    r.w1 = t - b0;
    b1 += t < b0;
    r.w2 = a.w2 - b.w2 - b1;
    return r;
}

// A probability clamped to [0, 1] (NaN and negatives read as 0), in units of
// 2^-149: significand M (with the implicit bit for normal numbers) shifted
// left by (biased exponent - 1), at most 126.
__device__ __forceinline__ Fx fx_of_prob(float x) {
    x = x > 0.0f ? fminf(x, 1.0f) : 0.0f;
    const uint32_t bits = __float_as_uint(x);
    const uint32_t e = bits >> 23, f = bits & 0x7fffffu;
    const uint64_t M = e ? (uint64_t)(f | 0x800000u) : (uint64_t)f;
    const uint32_t sh = e ? e - 1 : 0;
    const uint32_t off = sh & 63;
    const uint64_t lo = M << off;
    const uint64_t hi = off ? M >> (64 - off) : 0;
    return sh < 64 ? Fx{lo, hi, 0} : Fx{0, lo, hi};
}

// A uniform clamped to [0, 1 - 2^-24] (NaN and negatives read as 0).
__device__ __forceinline__ float clamp_uniform(float u) {
    return u > 0.0f ? fminf(u, 0x1.fffffep-1f) : 0.0f;
}

// floor(u * Z) for a clamped uniform u: u = m 2^-s with m < 2^24 and
// s >= 24, so m Z < 2^205 takes four words before the shift.
__device__ __forceinline__ Fx fx_floor_mul(Fx Z, float u) {
    const uint32_t bits = __float_as_uint(u);
    const uint32_t e = bits >> 23, f = bits & 0x7fffffu;
    const uint64_t m = e ? (uint64_t)(f | 0x800000u) : (uint64_t)f;
    const uint32_t s = e ? 150 - e : 149;
    uint64_t r[4];
    const uint64_t lo0 = m * Z.w0, hi0 = __umul64hi(m, Z.w0);
    const uint64_t lo1 = m * Z.w1, hi1 = __umul64hi(m, Z.w1);
    const uint64_t lo2 = m * Z.w2, hi2 = __umul64hi(m, Z.w2);
    r[0] = lo0;
    r[1] = lo1 + hi0;
    const uint64_t c1 = r[1] < lo1;
    const uint64_t t = lo2 + hi1;
    uint64_t c2 = t < lo2;
    r[2] = t + c1;
    c2 += r[2] < t;
    r[3] = hi2 + c2;
    const uint32_t ws = s >> 6, bs = s & 63;
    uint64_t out[3];
#pragma unroll
    for (int i = 0; i < 3; i++) {
        // words i + ws and i + ws + 1 of r (zero past the top), selected
        // without dynamic indexing
        uint64_t a = 0, b = 0;
#pragma unroll
        for (int j = 0; j < 4; j++) {
            a = (uint32_t)(i + (int)ws) == (uint32_t)j ? r[j] : a;
            b = (uint32_t)(i + (int)ws + 1) == (uint32_t)j ? r[j] : b;
        }
        out[i] = (a >> bs) | (bs ? b << (64 - bs) : 0);
    }
    return Fx{out[0], out[1], out[2]};
}

__device__ __forceinline__ Fx fx_shfl_xor(Fx a, int m) {
    return Fx{__shfl_xor(a.w0, m, kWave), __shfl_xor(a.w1, m, kWave), __shfl_xor(a.w2, m, kWave)};
}
__device__ __forceinline__ Fx fx_shfl_up(Fx a, int d) {
    return Fx{__shfl_up(a.w0, d, kWave), __shfl_up(a.w1, d, kWave), __shfl_up(a.w2, d, kWave)};
}
__device__ __forceinline__ Fx fx_shfl(Fx a, int lane) {
    return Fx{__shfl(a.w0, lane, kWave), __shfl(a.w1, lane, kWave), __shfl(a.w2, lane, kWave)};
}

__device__ __forceinline__ Fx wave_sum(Fx x) {
#pragma unroll
    for (int m = 32; m > 0; m >>= 1)
        x = fx_add(x, fx_shfl_xor(x, m));
    return x;
}

// Inclusive scan over a wavefront.
__device__ __forceinline__ Fx wave_incl_scan(Fx x, int lane) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const Fx y = fx_shfl_up(x, d);
        if (lane >= d)
            x = fx_add(x, y);
    }
    return x;
}

__device__ __forceinline__ int clamp_gamma(const AcceptParams &a, int b) {
    const int g = a.num_draft[b];
    return g < 0 ? 0 : (g > a.G ? a.G : g);
}

// Drafts accepted before the first rejection (gamma if none).  The test
// u q <= p is exact: the product of two float32 values is exact in float64.
// Every lane of the calling wavefront tests one draft (i = c + lane for
// c = 0, 64, ...), so a walk costs two dependent loads per 64 drafts; the
// first failing draft is the lowest set bit of the ballot.
__device__ int accept_walk(const AcceptParams &a, int b) {
    const int lane = threadIdx.x & (kWave - 1);
    const int gamma = clamp_gamma(a, b);
    for (int c = 0; c < gamma; c += kWave) {
        const int i = c + lane;
        bool bad = false;
        if (i < gamma) {
            const int d = a.draft[(size_t)b * a.G + i];
            const float u = clamp_uniform(a.u_accept[(size_t)b * a.G + i]);
            if (d < 0 || d >= a.V) {
                bad = true;
            } else {
                const float pv = a.p[((size_t)b * (a.G + 1) + i) * a.V + d];
                const float qv = a.q[((size_t)b * a.G + i) * a.V + d];
                const float p = pv > 0.0f ? fminf(pv, 1.0f) : 0.0f;
                const float q = qv > 0.0f ? fminf(qv, 1.0f) : 0.0f;
                bad = !((double)u * (double)q <= (double)p);
            }
        }
        const unsigned long long m = __ballot(bad);
        if (m)
            return c + __ffsll((long long)m) - 1;
    }
    return gamma;
}

// Elements e .. e + 3 (zero past V) of the target row p_k and, when
// `load_q`, of the draft row q_k.
__device__ __forceinline__ void load_rows(const AcceptParams &a, int b, int k, bool load_q, int e, float pe[4],
                                          float qe[4]) {
    const float *prow = a.p + ((size_t)b * (a.G + 1) + k) * a.V;
    const float *qrow = a.q + ((size_t)b * a.G + (load_q ? k : 0)) * a.V;
    if (e + 3 < a.V && ((a.V & 3) == 0)) {
        const float4 pv = *reinterpret_cast<const float4 *>(prow + e);
        pe[0] = pv.x; pe[1] = pv.y; pe[2] = pv.z; pe[3] = pv.w;
        if (load_q) {
            const float4 qv = *reinterpret_cast<const float4 *>(qrow + e);
            qe[0] = qv.x; qe[1] = qv.y; qe[2] = qv.z; qe[3] = qv.w;
        } else {
            qe[0] = qe[1] = qe[2] = qe[3] = 0.0f;
        }
    } else {
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const bool in = e + j < a.V;
            pe[j] = in ? prow[e + j] : 0.0f;
            qe[j] = (in && load_q) ? qrow[e + j] : 0.0f;
        }
    }
}

// Exact sampling weights from the loaded elements: the leftover mass
// max(0, p_k - q_k) (resid), else the target row itself.
__device__ __forceinline__ void weights_of(const float pe[4], const float qe[4], bool resid, Fx w[4]) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
        const Fx P = fx_of_prob(pe[j]);
        if (resid) {
            const Fx Q = fx_of_prob(qe[j]);
            w[j] = fx_gt(P, Q) ? fx_sub(P, Q) : fx_zero();
        } else {
            w[j] = P;
        }
    }
}

// The weights of the sampling row at elements e .. e + 3: the leftover mass
// at a rejection (use_p = false), else the target row.
__device__ __forceinline__ void row_weights(const AcceptParams &a, int b, int k, bool rejected, bool use_p,
                                           int e, Fx w[4]) {
    const bool resid = rejected && !use_p;
    float pe[4], qe[4];
    load_rows(a, b, k, resid, e, pe, qe);
    weights_of(pe, qe, resid, w);
}

__device__ __forceinline__ Fx sum4(const Fx w[4]) {
    return fx_add(fx_add(w[0], w[1]), fx_add(w[2], w[3]));
}

__device__ __forceinline__ void store_fx(uint64_t *p, Fx x) {
    p[0] = x.w0;
    p[1] = x.w1;
    p[2] = x.w2;
}
__device__ __forceinline__ Fx load_fx(const uint64_t *p) { return Fx{p[0], p[1], p[2]}; }

// Block sums j0 .. j0 + kPickChunk - 1 of a row (zero from `hi` on), every
// load issued before any is used.
constexpr int kPickChunk = 16;
__device__ __forceinline__ void load_chunk(const uint64_t *bs, int j0, int hi, Fx v[kPickChunk]) {
#pragma unroll
    for (int c = 0; c < kPickChunk; c++) {
        const int j = j0 + c;
        v[c] = j < hi ? load_fx(bs + 3 * (size_t)j) : fx_zero();
    }
}

// One wavefront per (sequence, block): the block's exact sum of sampling
// weights.  The leftover-mass and plain-row sums are both written when a
// rejection happened, so the pick kernel can fall back without another pass.
__global__ __launch_bounds__(256) void accept_blocks_kernel(AcceptParams a) {
    const int wave = (int)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    if (wave >= a.B * a.nblk)
        return;
    const int b = wave / a.nblk, blk = wave % a.nblk;
    const int gamma = clamp_gamma(a, b);
    const int k = accept_walk(a, b);
    const bool rejected = k < gamma;
    float pe[4], qe[4];
    load_rows(a, b, k, rejected, blk * kBlk + 4 * lane, pe, qe);
    Fx w[4];
    weights_of(pe, qe, rejected, w);
    const Fx s = wave_sum(sum4(w));
    if (lane == 0)
        store_fx(a.bsum + (((size_t)b * 2 + 0) * a.nblk + blk) * 3, s);
    if (blk == 0 && lane == 0)
        a.walk[b] = k;   // read by the pick kernel, so it need not walk again
    if (rejected) {
        weights_of(pe, qe, false, w);   // the target row, from the same loads
        const Fx sp = wave_sum(sum4(w));
        if (lane == 0)
            store_fx(a.bsum + (((size_t)b * 2 + 1) * a.nblk + blk) * 3, sp);
    }
}

// One wavefront per sequence: the total, the target T = floor(u Z), the block
// whose cumulative mass first exceeds T, and the element inside it.  Since the
// cumulative weights are integers, C_v > u Z exactly when C_v > T, and u < 1
// makes T < Z, so the element exists and carries weight.
__global__ __launch_bounds__(kPickThreads) void accept_pick_kernel(AcceptParams a) {
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int gamma = clamp_gamma(a, b);
    const int k = __builtin_amdgcn_readfirstlane(a.walk[b]);
    const bool rejected = k < gamma;
    const int per = (a.nblk + kWave - 1) / kWave;   // consecutive blocks per lane
    const int lo = min(lane * per, a.nblk), hi = min(lo + per, a.nblk);
    // with at most kPickChunk blocks per lane (vocabularies up to 262,144),
    // v keeps the lane's block sums for the owner's search below
    const bool one_chunk = per <= kPickChunk;

    int pass = 0;
    Fx run, incl, Z;
    Fx v[kPickChunk];
    const uint64_t *bs = nullptr;
    for (;; pass++) {
        bs = a.bsum + ((size_t)b * 2 + pass) * a.nblk * 3;
        run = fx_zero();
        for (int j0 = lo; j0 < hi; j0 += kPickChunk) {
            load_chunk(bs, j0, hi, v);
#pragma unroll
            for (int c = 0; c < kPickChunk; c++)
                run = fx_add(run, v[c]);
        }
        incl = wave_incl_scan(run, lane);
        Z = fx_shfl(incl, kWave - 1);
        // leftover mass zero: sample p_k itself (its sums are in pass 1)
        if (pass == 0 && rejected && fx_is_zero(Z))
            continue;
        break;
    }
    if (fx_is_zero(Z)) {
        if (lane == 0) {
            a.n_accepted[b] = k;
            a.next_token[b] = -1;   // a sampling row with no mass
        }
        return;
    }
    const Fx T = fx_floor_mul(Z, clamp_uniform(a.u_sample[b]));

    // the first lane whose run ends above T owns the block
    const unsigned long long own = __ballot(fx_gt(incl, T));
    const int owner = __ffsll((long long)own) - 1;   // exists: incl of lane 63 = Z > T
    int blk = 0;
    Fx base = fx_zero();
    if (lane == owner) {
        Fx acc = fx_sub(incl, run);   // mass before this lane's run (incl >= run)
        bool found = false;
        for (int j0 = lo; j0 < hi && !found; j0 += kPickChunk) {
            if (!one_chunk)
                load_chunk(bs, j0, hi, v);
#pragma unroll
            for (int c = 0; c < kPickChunk; c++) {
                const Fx next = fx_add(acc, v[c]);
                if (!found && fx_gt(next, T)) {   // blocks past hi add zero
                    blk = j0 + c;
                    found = true;
                }
                if (!found)
                    acc = next;
            }
        }
        base = acc;
    }
    blk = __shfl(blk, owner, kWave);
    base = fx_shfl(base, owner);

    // the element inside that block
    Fx w[4];
    row_weights(a, b, k, rejected, pass == 1, blk * kBlk + 4 * lane, w);
    const Fx lane_sum = sum4(w);
    const Fx lincl = fx_add(base, wave_incl_scan(lane_sum, lane));
    const unsigned long long hit = __ballot(fx_gt(lincl, T));
    const int first = __ffsll((long long)hit) - 1;   // exists: the block's total exceeds T
    int jsel = 3;
    if (lane == first) {
        // the smallest j whose cumulative weight exceeds T
        Fx acc = fx_sub(lincl, lane_sum);
        bool found = false;
#pragma unroll
        for (int j = 0; j < 4; j++) {
            acc = fx_add(acc, w[j]);
            if (!found && fx_gt(acc, T)) {
                jsel = j;
                found = true;
            }
        }
    }
    jsel = __shfl(jsel, first, kWave);
    if (lane == 0) {
        a.n_accepted[b] = k;
        a.next_token[b] = blk * kBlk + 4 * first + jsel;
    }
}

}  // namespace

// Workspace of the acceptance: the block sums, then (256-byte aligned) the
// per-sequence walk results.
static size_t walk_offset(size_t num_seqs, size_t nblk) {
    return (num_seqs * 2 * nblk * 3 * sizeof(uint64_t) + 255) & ~(size_t)255;
}

}  // namespace tsattn

using namespace tsattn;

extern "C" {

int ts_kv_append(const ts_attn_shape *s, const void *k_new, const void *v_new, void *k_pages, void *v_pages,
                 const int32_t *page_table, const int32_t *ctx_lens, const int32_t *q_lens, void *stream) {
    clear_error();
    if (!s)
        return fail(TS_ERR_NULL, "shape is NULL");
    if (!k_new || !v_new || !k_pages || !v_pages || !page_table || !ctx_lens || !q_lens)
        return fail(TS_ERR_NULL, "a pointer is NULL");
    if (s->num_seqs < 1 || s->num_kv_heads < 1 || s->max_q_len < 1 || s->max_pages_per_seq < 1 ||
        s->num_pages < 1 || s->page_size != 16 || (s->head_dim != 64 && s->head_dim != 128))
        return fail(TS_ERR_SHAPE, "unsupported shape for the KV append");
    if (((uintptr_t)k_new | (uintptr_t)v_new | (uintptr_t)k_pages | (uintptr_t)v_pages) & 15)
        return fail(TS_ERR_ARG, "misaligned pointer (16 B needed)");
    int st = check_device();
    if (st)
        return st;
    AppendParams p;
    p.k_new = static_cast<const uint16_t *>(k_new);
    p.v_new = static_cast<const uint16_t *>(v_new);
    p.k_pages = static_cast<uint16_t *>(k_pages);
    p.v_pages = static_cast<uint16_t *>(v_pages);
    p.page_table = page_table;
    p.ctx_lens = ctx_lens;
    p.q_lens = q_lens;
    p.num_pages = s->num_pages;
    p.B = s->num_seqs;
    p.Qmax = s->max_q_len;
    p.Hkv = s->num_kv_heads;
    p.D = s->head_dim;
    p.max_pages = s->max_pages_per_seq;
    const int64_t total = (int64_t)p.B * p.Qmax * p.Hkv * (p.D / 8);
    if ((total + 255) / 256 > INT32_MAX)
        return fail(TS_ERR_SHAPE, "KV append of %lld rows is too large for one launch",
                    (long long)((int64_t)p.B * p.Qmax * p.Hkv));
    const unsigned blocks = (unsigned)((total + 255) / 256);
    hipLaunchKernelGGL(kv_append_kernel, dim3(blocks), dim3(256), 0, reinterpret_cast<hipStream_t>(stream), p);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "KV append launch");
}

size_t ts_spec_accept_workspace_size(int32_t num_seqs, int32_t vocab) {
    clear_error();
    if (num_seqs < 1 || vocab < 1) {
        fail(TS_ERR_ARG, "num_seqs and vocab must be positive");
        return 0;
    }
    const size_t nblk = ((size_t)vocab + kBlk - 1) / kBlk;
    return walk_offset(num_seqs, nblk) + (((size_t)num_seqs * sizeof(int32_t) + 255) & ~(size_t)255);
}

int ts_spec_accept(int32_t num_seqs, int32_t vocab, int32_t max_draft, const float *p_target,
                   const float *q_draft, const int32_t *draft_tokens, const int32_t *num_draft,
                   const float *u_accept, const float *u_sample, int32_t *num_accepted, int32_t *next_token,
                   void *workspace, size_t workspace_bytes, void *stream) {
    clear_error();
    if (num_seqs < 1 || vocab < 1 || max_draft < 0)
        return fail(TS_ERR_ARG, "num_seqs, vocab must be positive and max_draft >= 0");
    if (!p_target || !num_draft || !u_sample || !num_accepted || !next_token || !workspace ||
        (max_draft > 0 && (!q_draft || !draft_tokens || !u_accept)))
        return fail(TS_ERR_NULL, "a pointer is NULL");
    const size_t need = ts_spec_accept_workspace_size(num_seqs, vocab);
    if (workspace_bytes < need)
        return fail(TS_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
    if ((((uintptr_t)p_target | (uintptr_t)q_draft) & 15) || ((uintptr_t)workspace & 255))
        return fail(TS_ERR_ARG, "misaligned pointer (probabilities 16 B, workspace 256 B)");
    int st = check_device();
    if (st)
        return st;
    AcceptParams a;
    a.p = p_target;
    a.q = q_draft;
    a.draft = draft_tokens;
    a.num_draft = num_draft;
    a.u_accept = u_accept;
    a.u_sample = u_sample;
    a.n_accepted = num_accepted;
    a.next_token = next_token;
    a.bsum = static_cast<uint64_t *>(workspace);
    a.walk = reinterpret_cast<int32_t *>(static_cast<char *>(workspace) +
                                         walk_offset(num_seqs, ((size_t)vocab + kBlk - 1) / kBlk));
    a.B = num_seqs;
    a.V = vocab;
    a.G = max_draft;
    a.nblk = (vocab + kBlk - 1) / kBlk;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    const int64_t waves = (int64_t)a.B * a.nblk;
    if ((waves + 3) / 4 > INT32_MAX)
        return fail(TS_ERR_ARG, "num_seqs x vocab is too large for one launch");
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    hipLaunchKernelGGL(accept_blocks_kernel, dim3(blocks), dim3(256), 0, hs, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "acceptance block-sum launch");
    hipLaunchKernelGGL(accept_pick_kernel, dim3(a.B), dim3(kPickThreads), 0, hs, a);
    e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "acceptance pick launch");
}

}  // extern "C"
