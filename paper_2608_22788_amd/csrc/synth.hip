// synth.hip -- the library's implementation of the seeded input generator:
// a device fill for bf16 N(0,1) values and the host draws of the sweep's
// context lengths and page permutation.  It follows the published
// definitions stated in include/ts_attn.h (SplitMix64, Box-Muller), written
// independently of the test-side generator; tests check the two agree bit for
// bit.  It holds none of the attention arithmetic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint32_t kStreamLenB = 2;   // response-length draws
constexpr uint32_t kStreamPerm = 3;   // page-permutation keys

__host__ __device__ inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__host__ __device__ inline uint64_t stream_key(uint64_t seed, uint32_t stream) {
    return mix64(((seed & ((1ull << 56) - 1)) << 8) + stream);
}

__host__ __device__ inline uint64_t draw(uint64_t key, uint64_t index) {
    return mix64(key + (index + 1) * kGamma);
}

__device__ inline uint16_t normal_bf16(uint64_t z) {
    const double u1 = ((double)(z >> 32) + 1.0) * 0x1p-32;
    const double u2 = (double)(z & 0xffffffffull) * 0x1p-32;
    const double x = sqrt(-2.0 * log(u1)) * cos(u2 * 6.283185307179586);
    const float f = (float)x;
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

__global__ __launch_bounds__(256) void fill_kernel(uint16_t *dst, int64_t n, uint64_t key,
                                                   int64_t offset) {
    const int64_t groups = (n + 7) / 8;
    for (int64_t gi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gi < groups;
         gi += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i0 = gi * 8;
        if (i0 + 8 <= n && ((reinterpret_cast<uintptr_t>(dst + i0) & 15) == 0)) {
            uint32_t w[4];
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const uint16_t a = normal_bf16(draw(key, (uint64_t)(offset + i0 + 2 * k)));
                const uint16_t b = normal_bf16(draw(key, (uint64_t)(offset + i0 + 2 * k + 1)));
                w[k] = (uint32_t)a | ((uint32_t)b << 16);
            }
            *reinterpret_cast<uint4 *>(dst + i0) = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
            for (int64_t i = i0; i < n && i < i0 + 8; i++)
                dst[i] = normal_bf16(draw(key, (uint64_t)(offset + i)));
        }
    }
}

}  // namespace

int synth_fill(void *dst, int64_t n, uint64_t seed, uint32_t stream_id, int64_t offset,
               hipStream_t stream) {
    if (n <= 0)
        return TS_OK;
    const int64_t groups = (n + 7) / 8;
    const int64_t blocks = std::min<int64_t>((groups + 255) / 256, 256 * 64);
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<uint16_t *>(dst), n, stream_key(seed, stream_id), offset);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? TS_OK : hip_fail(e, "synth fill launch");
}

void sweep_lengths(int32_t batch, uint64_t seed, int32_t *ctx_lens) {
    const uint64_t key = stream_key(seed, kStreamLenB);
    for (int32_t b = 0; b < batch; b++) {
        const uint64_t z = draw(key, (uint64_t)b);
        const double u1 = ((double)(z >> 32) + 1.0) * 0x1p-32;
        double resp = std::floor(1024.0 * std::pow(u1, -1.0 / 1.5));
        if (resp > 65536.0)
            resp = 65536.0;
        ctx_lens[b] = 512 + (int32_t)resp;
    }
}

void page_permutation(int64_t total, uint64_t seed, std::vector<int32_t> &perm) {
    const uint64_t key = stream_key(seed, kStreamPerm);
    std::vector<uint64_t> keys((size_t)total);
    for (int64_t i = 0; i < total; i++)
        keys[(size_t)i] = draw(key, (uint64_t)i);
    perm.resize((size_t)total);
    std::iota(perm.begin(), perm.end(), 0);
    std::stable_sort(perm.begin(), perm.end(),
                     [&](int32_t a, int32_t b) { return keys[(size_t)a] < keys[(size_t)b]; });
}

int build_page_table(int32_t batch, const int32_t *ctx_lens, int32_t page_size,
                     int32_t max_pages_per_seq, uint64_t seed, int32_t *page_table) {
    int64_t total = 0;
    for (int32_t b = 0; b < batch; b++) {
        if (ctx_lens[b] < 0)
            return fail(TS_ERR_ARG, "ctx_lens[%d] < 0", b);
        const int64_t np = (ctx_lens[b] + page_size - 1) / page_size;
        if (np > max_pages_per_seq)
            return fail(TS_ERR_ARG, "sequence %d needs %lld pages > max_pages_per_seq %d", b,
                        (long long)np, max_pages_per_seq);
        total += np;
    }
    if (total >= (1LL << 31))
        return fail(TS_ERR_ARG, "more than 2^31 pages");
    std::vector<int32_t> perm;
    page_permutation(total, seed, perm);
    int64_t off = 0;
    for (int32_t b = 0; b < batch; b++) {
        const int64_t np = (ctx_lens[b] + page_size - 1) / page_size;
        int32_t *row = page_table + (size_t)b * max_pages_per_seq;
        for (int64_t j = 0; j < max_pages_per_seq; j++)
            row[j] = j < np ? perm[(size_t)(off + j)] : 0;
        off += np;
    }
    return TS_OK;
}

}  // namespace tsattn

using namespace tsattn;

extern "C" {

int ts_synth_fill_bf16(void *dst, int64_t n, uint64_t seed, uint32_t stream_id,
                       int64_t index_offset, void *stream) {
    clear_error();
    if (!dst)
        return fail(TS_ERR_NULL, "dst is NULL");
    if (n < 0 || index_offset < 0)
        return fail(TS_ERR_ARG, "negative size or offset");
    int st = check_device();
    if (st)
        return st;
    return synth_fill(dst, n, seed, stream_id, index_offset, reinterpret_cast<hipStream_t>(stream));
}

int ts_synth_sweep_lengths(int32_t batch, uint64_t seed, int32_t *ctx_lens) {
    clear_error();
    if (!ctx_lens)
        return fail(TS_ERR_NULL, "ctx_lens is NULL");
    if (batch < 0)
        return fail(TS_ERR_ARG, "batch < 0");
    sweep_lengths(batch, seed, ctx_lens);
    return TS_OK;
}

int ts_synth_page_table(int32_t batch, const int32_t *ctx_lens, int32_t page_size,
                        int32_t max_pages_per_seq, uint64_t seed, int32_t *page_table) {
    clear_error();
    if (!ctx_lens || !page_table)
        return fail(TS_ERR_NULL, "NULL argument");
    if (batch < 0 || page_size < 1 || max_pages_per_seq < 1)
        return fail(TS_ERR_ARG, "invalid batch, page size or table width");
    try {
        return build_page_table(batch, ctx_lens, page_size, max_pages_per_seq, seed, page_table);
    } catch (...) {
        return fail(TS_ERR_ARG, "out of host memory");
    }
}

}  // extern "C"
