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
//     row p_gamma, by inverse CDF with the caller's uniform.  The sampling row
//     is a full vocabulary of fp32 probabilities per sequence, so the work is
//     a streaming read of one or two rows:
//       - accept_blocks_kernel: every 256-element block of every sequence's
//         sampling row is summed by one wavefront (a float4 per lane, lane
//         sums in element order, then a butterfly), so the whole chip shares
//         the read even for a handful of sequences;
//       - accept_pick_kernel: one workgroup per sequence scans the block sums
//         (lane runs of consecutive blocks, a wavefront scan of the run
//         totals), finds the block where the cumulative mass passes
//         u * total, and scans that block's 256 elements in order.
//     Both kernels recompute the acceptance walk (2 gamma scalar loads)
//     rather than pass it through memory.
//   Readings: the acceptance test is taken in fp32 as u * q <= p; a draft id
//   outside [0, V) is rejected; if the leftover mass sums to zero the next
//   token is drawn from p_k itself; a cumulative mass that rounding leaves
//   just short of the target selects the last token with mass.
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
    float *bsum;             // [B][nblk] block sums of the sampling row
    int B, V, G, nblk;
};

__device__ __forceinline__ int clamp_gamma(const AcceptParams &a, int b) {
    const int g = a.num_draft[b];
    return g < 0 ? 0 : (g > a.G ? a.G : g);
}

// Drafts accepted before the first rejection (gamma if none), by one thread.
__device__ int accept_walk(const AcceptParams &a, int b) {
    const int gamma = clamp_gamma(a, b);
    for (int i = 0; i < gamma; i++) {
        const int d = a.draft[(size_t)b * a.G + i];
        if (d < 0 || d >= a.V)
            return i;
        const float pv = a.p[((size_t)b * (a.G + 1) + i) * a.V + d];
        const float qv = a.q[((size_t)b * a.G + i) * a.V + d];
        const float u = a.u_accept[(size_t)b * a.G + i];
        if (!(u * qv <= pv))
            return i;
    }
    return gamma;
}

// Weights of the sampling row at elements e .. e + 3 (zero past V): the
// leftover mass at a rejection (use_p = false), else the target row itself.
__device__ __forceinline__ void row_weights(const AcceptParams &a, int b, int k, bool rejected, bool use_p,
                                           int e, float w[4]) {
    const float *prow = a.p + ((size_t)b * (a.G + 1) + k) * a.V;
    const float *qrow = a.q + ((size_t)b * a.G + (rejected ? k : 0)) * a.V;
    if (e + 3 < a.V && ((a.V & 3) == 0)) {
        const float4 pv = *reinterpret_cast<const float4 *>(prow + e);
        float pe[4] = {pv.x, pv.y, pv.z, pv.w};
        if (rejected && !use_p) {
            const float4 qv = *reinterpret_cast<const float4 *>(qrow + e);
            const float qe[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
            for (int j = 0; j < 4; j++)
                pe[j] = fmaxf(0.0f, pe[j] - qe[j]);
        }
#pragma unroll
        for (int j = 0; j < 4; j++)
            w[j] = pe[j];
        return;
    }
#pragma unroll
    for (int j = 0; j < 4; j++) {
        const int v = e + j;
        if (v >= a.V) {
            w[j] = 0.0f;
            continue;
        }
        const float pv = prow[v];
        w[j] = (rejected && !use_p) ? fmaxf(0.0f, pv - qrow[v]) : pv;
    }
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        x += __shfl_xor(x, off, kWave);
    return x;
}

// One wavefront per (sequence, block): the block's sum of sampling weights.
// The leftover-mass and plain-row sums are both written when a rejection
// happened, so the pick kernel can fall back without another pass.
__global__ __launch_bounds__(256) void accept_blocks_kernel(AcceptParams a) {
    const int wave = (int)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    if (wave >= a.B * a.nblk)
        return;
    const int b = wave / a.nblk, blk = wave % a.nblk;
    const int gamma = clamp_gamma(a, b);
    const int k = accept_walk(a, b);
    const bool rejected = k < gamma;
    float w[4];
    row_weights(a, b, k, rejected, false, blk * kBlk + 4 * lane, w);
    const float s = wave_sum(((w[0] + w[1]) + w[2]) + w[3]);
    if (lane == 0)
        a.bsum[((size_t)b * 2 + 0) * a.nblk + blk] = s;
    if (rejected) {
        row_weights(a, b, k, true, true, blk * kBlk + 4 * lane, w);
        const float sp = wave_sum(((w[0] + w[1]) + w[2]) + w[3]);
        if (lane == 0)
            a.bsum[((size_t)b * 2 + 1) * a.nblk + blk] = sp;
    }
}

// Inclusive scan over a wavefront.
__device__ __forceinline__ float wave_incl_scan(float x, int lane) {
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const float y = __shfl_up(x, off, kWave);
        if (lane >= off)
            x += y;
    }
    return x;
}

__global__ __launch_bounds__(kPickThreads) void accept_pick_kernel(AcceptParams a) {
    __shared__ int s_k;
    __shared__ int s_blk;
    __shared__ float s_base;
    __shared__ int s_use_p;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    if (tid == 0) {
        s_k = accept_walk(a, b);
        s_blk = -1;
    }
    __syncthreads();
    const int gamma = clamp_gamma(a, b);
    const int k = s_k;
    const bool rejected = k < gamma;

    // which block holds the target mass
    {
        int use_p = 0;
        for (int pass = 0; pass < 2; pass++) {
            const float *bs = a.bsum + ((size_t)b * 2 + pass) * a.nblk;
            const int per = (a.nblk + kWave - 1) / kWave;   // consecutive blocks per lane
            const int lo = lane * per, hi = min(lo + per, a.nblk);
            float run = 0.0f;
            for (int j = lo; j < hi; j++)
                run += bs[j];
            const float incl = wave_incl_scan(run, lane);
            const float total = __shfl(incl, kWave - 1, kWave);
            if (pass == 0 && !(total > 0.0f) && rejected) {
                use_p = 1;   // leftover mass vanished: sample p_k itself
                continue;
            }
            const float target = a.u_sample[b] * total;
            // the lane whose run holds the target, else the last lane with mass
            const float excl = incl - run;
            const bool here = run > 0.0f && excl <= target && target < incl;
            const unsigned long long m = __ballot(here);
            const unsigned long long nz = __ballot(run > 0.0f);
            const int owner = m ? __ffsll((long long)m) - 1 : (nz ? 63 - __clzll((long long)nz) : 0);
            if (lane == owner) {
                float acc = excl;
                int pick = -1, last = -1;
                for (int j = lo; j < hi; j++) {
                    if (bs[j] > 0.0f) {
                        last = j;
                        if (pick < 0 && target < acc + bs[j])
                            pick = j;
                    }
                    if (pick < 0)
                        acc += bs[j];
                }
                if (pick < 0) {
                    pick = last < 0 ? 0 : last;
                    acc = excl;
                    for (int j = lo; j < pick; j++)
                        acc += bs[j];
                }
                s_blk = pick;
                s_base = acc;
                s_use_p = use_p;
            }
            break;
        }
    }
    __syncthreads();

    // the element inside that block, scanned in order
    {
        const int blk = s_blk;
        float w[4];
        row_weights(a, b, k, rejected, s_use_p != 0, blk * kBlk + 4 * lane, w);
        const float lane_sum = ((w[0] + w[1]) + w[2]) + w[3];
        const float incl = wave_incl_scan(lane_sum, lane);
        // the row total is taken from the block sums, as in the block search
        // above, so that both searches aim at the same target
        const float *bs = a.bsum + ((size_t)b * 2 + (s_use_p ? 1 : 0)) * a.nblk;
        float total;
        {
            const int per = (a.nblk + kWave - 1) / kWave;
            const int lo = lane * per, hi = min(lo + per, a.nblk);
            float run = 0.0f;
            for (int j = lo; j < hi; j++)
                run += bs[j];
            total = __shfl(wave_incl_scan(run, lane), kWave - 1, kWave);
        }
        const float target = a.u_sample[b] * total;
        float acc = s_base + (incl - lane_sum);
        int pick = -1;
        int j = 0;
        for (; j < 4; j++) {
            if (w[j] > 0.0f && target < acc + w[j]) {
                pick = j;
                break;
            }
            acc += w[j];
        }
        const bool found = pick >= 0;
        const unsigned long long m = __ballot(found);
        int last_lane = -1, last_j = -1;
        if (!m) {
            // rounding left the walk short: the block's last element with mass
            int lj = -1;
            for (int jj = 3; jj >= 0; jj--)
                if (w[jj] > 0.0f) {
                    lj = jj;
                    break;
                }
            const unsigned long long nz = __ballot(lj >= 0);
            last_lane = nz ? 63 - __clzll((long long)nz) : 0;
            last_j = __shfl(lj, last_lane, kWave);
        }
        const int first = m ? __ffsll((long long)m) - 1 : last_lane;
        const int jsel = m ? __shfl(pick, first, kWave) : (last_j < 0 ? 0 : last_j);
        if (lane == 0) {
            a.n_accepted[b] = k;
            a.next_token[b] = blk * kBlk + 4 * first + jsel;
        }
    }
}

}  // namespace

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
    return ((size_t)num_seqs * 2 * nblk * sizeof(float) + 255) & ~(size_t)255;
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
    a.bsum = static_cast<float *>(workspace);
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
