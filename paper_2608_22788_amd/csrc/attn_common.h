// attn_common.h -- device-side pieces shared by the paged-attention kernels:
// kernel parameters, bf16 packing, wavefront reductions and the split of the
// KV stream over wavefronts.
//
// Work partition.  A "unit" is one (sequence b, KV head g) pair; it owns
// np_b = ceil(L_b / 16) pages.  Units are laid end to end (b-major, g-minor)
// into one global page index space of Ptot = Hkv * sum_b np_b pages, and
// worker (wavefront) w of W processes the contiguous range
//   [floor(Ptot * w / W), floor(Ptot * (w + 1) / W)),
// so every worker streams the same number of KV bytes to within one page no
// matter how skewed the context lengths are.  A worker's range may start or
// end inside a unit; such a piece is a split whose normalised partial output
// and log2-sum-exp go to the workspace, slot 2w if the piece is the first of
// the worker's range and 2w+1 otherwise.  A unit processed whole by one worker
// is written straight to `out`.  The workers that touched a unit are found by
// inverting the range formula, and their slots are combined (attn_split.h) in
// one of three ways, chosen on the host: by the last of them to finish (many
// units, one or two pieces each), by merge workgroups appended to the same
// launch (few units, many pieces each), or by a separate merge kernel.
// Everything depends on ctx_lens / q_lens read on the device, so the launch
// grid depends on the shape alone.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tsattn {

constexpr int kPage = 16;          // tokens per page
constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kMaxSeqs = 4096;     // sequences per call (LDS prefix array)
constexpr int kMaxUnits = 1 << 18; // (sequence, KV head) units per call
constexpr size_t kCounterBytes = (size_t)kMaxUnits * sizeof(int);   // split counters
constexpr float kRescaleSlack = 8.0f;  // lazy rescale threshold, log2 units

// Who combines the split partials of a launch.  In the two in-launch modes
// the workers write partials with device-coherent stores and count their
// arrivals on the unit's counter.
constexpr int kCombineKernel = 0;    // a separate merge kernel (plain stores)
constexpr int kCombineLast = 1;      // the last worker to finish a piece of the unit
constexpr int kCombineInLaunch = 2;  // merge workgroups after the W workers of the grid

struct AttnParams {   // 128 bytes of kernel arguments
    const uint16_t *q;          // [B][Qmax][Hq][D] bf16
    const uint16_t *k_pages;    // [num_pages][Hkv][P][D] bf16
    const uint16_t *v_pages;
    const int32_t *page_table;  // [B][max_pages]
    const int32_t *ctx_lens;    // [B]
    const int32_t *q_lens;      // [B]
    uint16_t *out;              // [B][Qmax][Hq][D] bf16
    float *ws_o;                // [2W][rows_per_unit][D] fp32 partial outputs
    float *ws_lse;              // [2W][rows_per_unit] fp32 log2-sum-exp
    int *counters;              // arrivals per split unit, unit u at u << cnt_shift (zero between calls)
    int B, Hq, Hkv, D, Qmax, max_pages;
    int G;                      // Hq / Hkv
    int rows_per_unit;          // G * Qmax
    int W;                      // workers (wavefronts)
    int ws_o_bytes;             // bytes of the partial area (set unless kCombineKernel; < 2^31)
    int16_t combine;            // kCombine*: who combines the split partials
    int16_t cnt_shift;          // log2 of the ints between the counters of consecutive units
    float scale_log2;           // scale * log2(e)
};

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// K/V pages are read exactly once per call, so they are loaded with the
// non-temporal hint: on MI355X this raised a plain streaming read from about
// 6.1 to 7.0 TB/s, because the lines are not kept in the caches.
__device__ __forceinline__ u32x4_t ld_stream16(const void *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
}
__device__ __forceinline__ u32x2_t ld_stream8(const void *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
}

// A (page, KV head) block as a buffer resource.  Loads at byte offsets below
// `bytes` read the block; a load at or past `bytes` returns zeros without a
// memory access, so bytes = 0 turns the loads of a page past the segment end
// into no-ops that yield zeros (no branch, no clamped re-read).  Word 3 is the
// raw 32-bit data format of the gfx9 family's buffer descriptors.
typedef __amdgpu_buffer_rsrc_t block_rsrc_t;
constexpr int kBufferWord3 = 0x00020000;
constexpr int kLoadNt = 2;   // cache policy of buffer loads: non-temporal

__device__ __forceinline__ block_rsrc_t block_rsrc(const void *base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, kBufferWord3);
}
__device__ __forceinline__ u32x4_t ld_block16(block_rsrc_t r, int byte_off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kLoadNt);
}
__device__ __forceinline__ u32x2_t ld_block8(block_rsrc_t r, int byte_off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, kLoadNt);
}

// Keeps the instruction scheduler from moving anything across this point, so
// the program order of a prefetch relative to the computation is kept.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two floats -> packed bf16 pair (round to nearest even), lo in bits 0..15.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t b = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ uint16_t to_bf16(float x) {
    return (uint16_t)(pack_bf16x2(x, 0.0f) & 0xffffu);
}

// c + a.lo * b.lo + a.hi * b.hi, with a and b packed bf16 pairs.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                            __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// DPP lane exchanges inside a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, true));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within 8

// Sum over aligned groups of 8 lanes; every lane of the group gets the total.
__device__ __forceinline__ float sum8(float x) {
    x += dpp_f32<kDppXor1>(x);
    x += dpp_f32<kDppXor2>(x);
    x += dpp_f32<kDppHalfMirror>(x);
    return x;
}

__device__ __forceinline__ int first_lane_int(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Split counter of unit (b, g).
__device__ __forceinline__ int *unit_counter(const AttnParams &p, int unit) {
    return p.counters + ((size_t)unit << p.cnt_shift);
}

// Metadata (page table, context and draft lengths) is read-only for the whole
// launch.  Reading it through the constant address space lets wavefront-uniform
// reads become scalar loads, which are counted separately from the vector
// loads of K/V pages; a vector load here would make the wavefront wait for
// every K/V prefetch still in flight before it could compute the next address.
typedef const int32_t __attribute__((address_space(4))) *const_i32_ptr;
__device__ __forceinline__ int32_t ld_meta(const int32_t *p, size_t i) {
    return ((const_i32_ptr)p)[i];
}

// ---------------------------------------------------------------------------
// Work partition (see the header comment).
// ---------------------------------------------------------------------------

// Pages of sequence b that carry work: 0 if q_lens[b] == 0.
__device__ __forceinline__ int seq_pages(const AttnParams &p, int b) {
    int L = ld_meta(p.ctx_lens, b);
    int Q = ld_meta(p.q_lens, b);
    return (Q > 0 && L > 0) ? (L + kPage - 1) / kPage : 0;
}

// Exclusive prefix of seq_pages into s_pre[0..B] (s_pre[B] = total), computed
// by the first wavefront of the block; every thread must call it (it ends in
// a block barrier).  Sequences are taken in batches of 64 * kPrefixRun: lane t
// owns the run of kPrefixRun consecutive sequences starting at t * kPrefixRun.
// All lengths of a batch are loaded before any is used (one memory latency
// for up to 512 sequences), the run totals are scanned across the wavefront
// once, and each lane then writes its run's prefixes.
constexpr int kPrefixRun = 8;

__device__ inline void page_prefix(const AttnParams &p, int *s_pre) {
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        int base = 0;
        for (int b0 = 0; b0 < p.B; b0 += kPrefixRun * kWave) {
            const int first = b0 + lane * kPrefixRun;
            int n[kPrefixRun];
            int run = 0;
#pragma unroll
            for (int k = 0; k < kPrefixRun; k++) {
                // unconditional load at a clamped index, so that every load
                // is issued before the first wait
                const int b = first + k;
                const int v = seq_pages(p, min(b, p.B - 1));
                n[k] = b < p.B ? v : 0;
                run += n[k];
            }
            int incl = run;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const int y = __shfl_up(incl, off, kWave);
                if (lane >= off)
                    incl += y;
            }
            int acc = base + incl - run;
#pragma unroll
            for (int k = 0; k < kPrefixRun; k++) {
                if (first + k < p.B)
                    s_pre[first + k] = acc;
                acc += n[k];
            }
            base += __shfl(incl, kWave - 1, kWave);
        }
        if (lane == 0)
            s_pre[p.B] = base;
    }
    __syncthreads();
}

// Worker of workgroup `block` (of W): the chip deals workgroups to its 8 XCDs
// round-robin (workgroup b runs on XCD b % 8), and each XCD has its own L2.
// Consecutive workers of the partition share units (a unit's pieces, its
// query rows and page-table entries), so they are given consecutive
// workgroups of one XCD: XCD x takes workers base(x) .. base(x + 1) - 1.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_worker(int block, int W) {
    const int x = block % kXcds, s = block / kXcds;
    return x * (W / kXcds) + min(x, W % kXcds) + s;
}

__device__ __forceinline__ int64_t worker_begin(int64_t ptot, int w, int W) {
    return (ptot * (int64_t)w) / (int64_t)W;
}

// Worker whose range holds global page x (0 <= x < ptot).
__device__ __forceinline__ int worker_of(int64_t ptot, int64_t x, int W) {
    return (int)(((x + 1) * (int64_t)W - 1) / ptot);
}

// Sequence holding global page x: the largest b with Hkv * s_pre[b] <= x.
__device__ __forceinline__ int find_seq(const int *s_pre, int B, int64_t x, int Hkv) {
    const int64_t y = x / Hkv;
    int lo = 0, hi = B - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if ((int64_t)s_pre[mid] <= y)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

struct Segment {
    int b, g;          // unit
    int j0, j1;        // logical pages [j0, j1) of the unit
    bool whole;        // the unit is entirely inside this segment
    int np;            // pages of the unit
    int64_t us;        // global index of the unit's first page
    int64_t next;      // global page after the segment
};

__device__ __forceinline__ Segment locate(const AttnParams &p, const int *s_pre, int64_t x,
                                          int64_t range_end) {
    Segment s;
    s.b = first_lane_int(find_seq(s_pre, p.B, x, p.Hkv));
    const int np = s_pre[s.b + 1] - s_pre[s.b];
    const int64_t base = (int64_t)p.Hkv * s_pre[s.b];
    const int64_t off = x - base;
    s.g = first_lane_int((int)(off / np));
    s.j0 = first_lane_int((int)(off % np));
    const int64_t unit_end = base + (int64_t)(s.g + 1) * np;
    const int64_t seg_end = unit_end < range_end ? unit_end : range_end;
    s.j1 = s.j0 + (int)(seg_end - x);
    s.whole = (s.j0 == 0) && (seg_end == unit_end);
    s.np = np;
    s.us = base + (int64_t)s.g * np;
    s.next = seg_end;
    return s;
}

}  // namespace tsattn
