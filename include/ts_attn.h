/*
 * ts_attn.h -- C ABI of libtsattn: paged decode and speculative-verify
 * attention for AMD Instinct MI355X (gfx950).
 *
 * The operation.  Rollout replicas spend their decode phase (paper Sec. 2.1)
 * attending each sequence's new query tokens to its whole KV cache.  The bulk
 * pool decodes one token per sequence at high concurrency; the tail pool runs
 * speculative decoding (Sec. 3.4 and Sec. 4.3: multi-token-prediction heads
 * with 3-5 drafts, block drafters with blocks of 4 or more) and verifies the
 * 1 + gamma tokens of each draft block with the target model, so every
 * sequence contributes q_len query rows that attend causally within the
 * block.  The paper observes that long-context generation is bound by
 * KV-cache traffic and attention memory bandwidth (App. F, speculative
 * decoding for long context); these kernels are built to that roofline.
 *
 * Definition computed (fp32 accumulation, bf16 in and out):
 *   for sequence b with L = ctx_lens[b] (L counts the q_len new tokens, whose
 *   keys and values are already in the pages) and Q = q_lens[b]:
 *     row i in [0, Q) sits at absolute position L - Q + i and sees keys
 *     t in [0, L - Q + i]  (causal within the draft block, diagonal included);
 *     query head h reads KV head h / (Hq / Hkv)  (contiguous GQA groups);
 *     K_t = k_pages[page_table[b][t / P]][g][t % P][:], V_t likewise;
 *     out[b][i][h][:] = sum_t softmax_t(scale * <q[b][i][h][:], K_t>) V_t.
 *
 * Memory layouts (row-major, all device memory unless stated):
 *   q, out      bf16  [num_seqs][max_q_len][num_q_heads][head_dim]
 *   k_pages,
 *   v_pages     bf16  [num_pages][num_kv_heads][page_size][head_dim]
 *   page_table  int32 [num_seqs][max_pages_per_seq]; entries at logical
 *               page j >= ceil(L / P) are never read
 *   ctx_lens,
 *   q_lens      int32 [num_seqs]
 *
 * Ownership and errors.  The caller owns every buffer and the stream; the
 * library allocates nothing inside ts_decode_attn, never synchronises it and
 * never reads device data on the host, so a call can be captured into a HIP
 * graph.  Inputs are read-only; out is written only at rows i < q_lens[b]
 * (q_lens[b] = 0 skips sequence b).  The workspace starts with a fixed
 * 1 MiB area of arrival counters (one per (sequence, KV head), up to 4 KiB
 * apart when there are few), then the
 * TS_DEBUG flag word, then split partial results.  It must be zero-filled
 * before its first use (e.g. hipMemset once after allocation); every completed
 * call leaves the counters zero again and never writes anything else over
 * them, so a workspace can be reused by any later call, of any shape, on one
 * stream (the rest of its contents is undefined on return).  Calls that may
 * run concurrently need distinct workspaces.  Every entry point
 * returns TS_OK (0) or a negative ts_status; on error nothing is launched and
 * ts_last_error() describes the cause.  No C++ exception crosses the ABI.
 *
 * Device-side preconditions (1 <= q_lens[b] <= ctx_lens[b] <= max_ctx_len,
 * ctx_lens[b] <= max_pages_per_seq * page_size, q_lens[b] <= max_q_len, page
 * ids in [0, num_pages)) are the caller's to keep on the fast path; with the
 * environment variable TS_DEBUG=1 a checking kernel verifies them (and that
 * the workspace counters are zero) first, the call synchronises and returns
 * TS_ERR_SHAPE (TS_ERR_WORKSPACE for the counters) if any fails.
 */
#ifndef TS_ATTN_H
#define TS_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TS_ATTN_ABI_VERSION 4

typedef enum ts_status {
    TS_OK = 0,
    TS_ERR_NULL = -1,        /* a required pointer is NULL */
    TS_ERR_SHAPE = -2,       /* shape outside the supported set, or a failed TS_DEBUG check */
    TS_ERR_WORKSPACE = -3,   /* workspace smaller than ts_decode_attn_workspace_size() */
    TS_ERR_UNSUPPORTED = -4, /* no device of the supported architecture */
    TS_ERR_HIP = -5,         /* a HIP runtime call failed; see ts_last_error() */
    TS_ERR_ARG = -6          /* an argument other than the shape is invalid */
} ts_status;

/* Host-known description of one call.  Supported: page_size 16; head_dim 64
 * or 128; num_q_heads a multiple of num_kv_heads with group size
 * G = num_q_heads / num_kv_heads in 1..16 and G * max_q_len <= 64;
 * max_q_len in 1..16; num_seqs in 1..4096; num_seqs * num_kv_heads <= 2^18.
 * max_ctx_len is an upper bound on ctx_lens, used for validation and to size
 * the automatic worker count; the launch grid depends on the shape alone.
 * num_workers = 0 lets the library choose how many workers (one wavefront,
 * or a four-wavefront team for verify at head_dim 128) share the KV stream;
 * a positive value fixes it (the result does not depend on it
 * beyond rounding; tests use it to vary the split points).  variant selects
 * the kernel:
 *   TS_VARIANT_AUTO  the matrix-core kernel in which one wavefront holds
 *                    every row block for up to 32 rows per (sequence, KV
 *                    head), the team kernel beyond (head_dim 128);
 *   TS_VARIANT_WAVE  the single-wavefront matrix-core kernel, any shape;
 *   TS_VARIANT_TEAM  head_dim 128 only: four wavefronts share each page
 *                    through LDS;
 *   TS_VARIANT_VALU  max_q_len 1 with a group size of 1, 2, 4 or 8 only: the
 *                    one-token kernel on vector ALUs (dot2), kept for
 *                    comparison; the matrix-core kernel measured faster. */
#define TS_VARIANT_AUTO 0
#define TS_VARIANT_WAVE 1
#define TS_VARIANT_TEAM 2
#define TS_VARIANT_VALU 3

typedef struct ts_attn_shape {
    int32_t num_seqs;
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t page_size;
    int32_t max_q_len;
    int32_t max_pages_per_seq;
    int32_t max_ctx_len;
    int64_t num_pages;
    int32_t num_workers;
    int32_t variant;
} ts_attn_shape;

/* Bytes of device workspace ts_decode_attn needs for this shape (split-KV
 * partial outputs, their log-sum-exp, the per-unit arrival counters and the
 * TS_DEBUG flag word).
 * Host only; returns 0 and sets ts_last_error() for an unsupported shape. */
size_t ts_decode_attn_workspace_size(const ts_attn_shape *shape);

/* Paged decode / verify attention as defined above, enqueued on `stream`
 * (a hipStream_t; NULL is the default stream).  `scale` multiplies the dot
 * products (typically 1/sqrt(head_dim)).  `workspace` is device memory of at
 * least ts_decode_attn_workspace_size(shape) bytes, 256-byte aligned,
 * zero-filled before its first use (see above). */
int ts_decode_attn(const ts_attn_shape *shape, const void *q, const void *k_pages,
                   const void *v_pages, const int32_t *page_table, const int32_t *ctx_lens,
                   const int32_t *q_lens, void *out, float scale, void *workspace,
                   size_t workspace_bytes, void *stream);

/* ts_decode_attn whose main (KV-streaming) kernel is launched with `ev_begin`
 * and `ev_end` attached to its dispatch: they take the kernel's own start and
 * end timestamps, so ts_event_elapsed_ms() gives that kernel's duration alone
 * (with the combination of split results when that launch does it, without
 * the separate merge kernel when one follows).  Events come from
 * ts_event_create(); either may be NULL. */
int ts_decode_attn_events(const ts_attn_shape *shape, const void *q, const void *k_pages,
                          const void *v_pages, const int32_t *page_table,
                          const int32_t *ctx_lens, const int32_t *q_lens, void *out,
                          float scale, void *workspace, size_t workspace_bytes, void *stream,
                          void *ev_begin, void *ev_end);

/* What ts_decode_attn launches for `shape` on the current device, for
 * diagnostics and tests: nothing is launched and no device memory is read.
 * Splits of a unit (sequence, KV head) that several workers share are
 * combined by the last worker to finish a piece of it, by merge wavefronts
 * that follow the workers in the same launch, or by a separate merge kernel;
 * the choice and the worker count depend on the shape and on the compiled
 * kernels' occupancy.  Fills *plan; returns TS_OK or a negative ts_status
 * (as ts_decode_attn would for the same shape). */
#define TS_COMBINE_MERGE_KERNEL 0
#define TS_COMBINE_LAST_ARRIVER 1
#define TS_COMBINE_IN_LAUNCH 2

typedef struct ts_attn_plan {
    int32_t variant;            /* kernel used: TS_VARIANT_WAVE, _TEAM or _VALU */
    int32_t num_workers;        /* workers of the page partition */
    int32_t combine;            /* TS_COMBINE_* */
    int32_t grid;               /* workgroups of the streaming launch (workers, then any
                                   merge workgroups) */
    int32_t threads;            /* threads per workgroup of the streaming launch */
    int32_t merge_blocks;       /* workgroups of the merge kernel (0 if none runs) */
    int64_t lds_bytes;          /* dynamic LDS per workgroup of the streaming launch */
    int64_t workspace_bytes;    /* ts_decode_attn_workspace_size(shape) */
} ts_attn_plan;

int ts_decode_attn_plan(const ts_attn_shape *shape, ts_attn_plan *plan);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * ts_decode_attn with the same arguments but no workspace.  Its split
 * partials, arrival counters and TS_DEBUG flag word live in a static device
 * array of TS_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds
 * until the process ends.  The call allocates nothing, on the host's HIP
 * runtime or elsewhere.  Shapes whose ts_decode_attn_workspace_size exceeds
 * the array are rejected with TS_ERR_WORKSPACE before anything is launched
 * (every shape with num_workers = 0 fits).  Every call on one GPU shares that
 * GPU's array, so calls that may overlap on one GPU (different streams, or
 * graphs replayed concurrently) race and must not be issued.  The array starts
 * zeroed and every call leaves its arrival counters zero, as with a
 * zero-filled workspace. */
#define TS_NOALLOC_SCRATCH_BYTES ((size_t)48 << 20)

int ts_decode_attn_noalloc(const ts_attn_shape *shape, const void *q, const void *k_pages,
                           const void *v_pages, const int32_t *page_table, const int32_t *ctx_lens,
                           const int32_t *q_lens, void *out, float scale, void *stream);

/* ---- concurrency-throughput curve ------------------------------------------
 * The paper's controller consumes a measured decode throughput v(b) versus
 * active batch b, and the per-token time tau(b) = 1 / v(b) (Sec. 2.1;
 * Sec. 3.2 outer loop; App. C.2).  ts_concurrency_sweep measures the
 * attention share of that curve on this GPU: for each batch size it draws
 * context lengths (512 + a Pareto(x_min 1024, alpha 1.5) response capped at
 * 65536, the same SplitMix64 definitions as the test generator), a random
 * page permutation and N(0,1) bf16 values, then times ts_decode_attn with HIP
 * events around groups of back-to-back calls while rotating over enough
 * distinct KV pools to defeat the last-level cache.  Synchronous; allocates
 * its device memory once, at the largest point's size, on the current
 * device, and frees it on return. */
typedef struct ts_sweep_config {
    int32_t num_q_heads;        /* 32 */
    int32_t num_kv_heads;       /* 8 */
    int32_t head_dim;           /* 128 */
    int32_t num_batches;        /* entries used in batches[] */
    int32_t batches[32];        /* e.g. 1, 2, 4, ..., 512 */
    int32_t verify_max_batch;   /* batches <= this use q_len = verify_q_len ... */
    int32_t verify_q_len;       /* ... (4); larger batches use q_len 1 */
    int32_t num_seeds;          /* seeds 0 .. num_seeds-1 per batch size */
    int32_t warmup;             /* untimed calls per point */
    int32_t iters;              /* timed calls per point, back to back in groups of
                                   min(10, iters / 5) calls (at least 1), so at least
                                   five groups; a remainder is not timed */
    int64_t min_rotation_bytes; /* KV bytes cycled through per point (>= 1 GiB) */
    double verify_tokens_per_step; /* tokens a verify step emits per sequence (accepted
                                      drafts + 1); the sweep does not model acceptance,
                                      so the caller states it; <= 0 reads as 1.  A
                                      one-token decode step emits 1. */
} ts_sweep_config;

typedef struct ts_sweep_point {
    int32_t batch;
    int32_t q_len;
    int32_t seed;
    int32_t num_pools;          /* distinct KV pools rotated through */
    int64_t sum_ctx;            /* sum of context lengths */
    int64_t kv_bytes;           /* algorithmic K+V bytes per call */
    double t_median_us;         /* per-call time, whole call (every launch it makes):
                                   median over the timed groups of a group's mean */
    double t_p10_us;            /* 10th and 90th percentiles of the same */
    double t_p90_us;
    double kv_gbps;             /* kv_bytes / t_median */
    double hbm_frac;            /* kv_gbps / 8000 (MI355X HBM3E peak) */
    double tokens_per_s;        /* batch * tokens per step / t_median (tokens per step: 1
                                   at q_len 1, verify_tokens_per_step when verifying) */
    double tau_us;              /* t_median / tokens per step: attention time per emitted
                                   token of one sequence, the attention share of tau(b) */
    double gather_median_us;    /* per-call time of ts_page_gather_read over the same pools
                                   (the read-only floor of the same call), timed alike */
} ts_sweep_point;

/* Runs the sweep; writes up to `cap` points (num_batches * num_seeds needed)
 * and their count to *n_out. */
int ts_concurrency_sweep(const ts_sweep_config *cfg, ts_sweep_point *pts, int32_t cap,
                         int32_t *n_out);

/* ---- the steps around the verify attention ----------------------------------
 * One speculative decoding step (Sec. 3.4: drafts are verified by the target
 * model without changing its output distribution) writes the 1 + gamma new
 * tokens' keys and values into the paged cache, runs ts_decode_attn over
 * them, and after the model's remaining layers decides which drafts to keep.
 * Both entry points are asynchronous on `stream`, allocate nothing and read
 * no device data on the host. */

/* KV append: for every sequence b and row i < q_lens[b] (token position
 * t = ctx_lens[b] - q_lens[b] + i, i.e. ctx_lens already counts the new
 * tokens), every KV head g:
 *   k_pages[page_table[b][t / 16]][g][t % 16][:] = k_new[b][i][g][:]  (v alike)
 * k_new, v_new: bf16 [num_seqs][max_q_len][num_kv_heads][head_dim], 16-byte
 * aligned.  Uses num_seqs, num_kv_heads, head_dim (64 or 128), page_size (16),
 * max_q_len, max_pages_per_seq and num_pages of the shape.  A row whose
 * position or page id falls outside the pool is skipped, not written. */
int ts_kv_append(const ts_attn_shape *shape, const void *k_new, const void *v_new, void *k_pages,
                 void *v_pages, const int32_t *page_table, const int32_t *ctx_lens,
                 const int32_t *q_lens, void *stream);

/* Bytes of device workspace ts_spec_accept needs (256-byte aligned). */
size_t ts_spec_accept_workspace_size(int32_t num_seqs, int32_t vocab);

/* Lossless acceptance (speculative sampling, Leviathan et al. 2023, which
 * the paper follows in Sec. 3.4).  Sequence b proposed gamma_b = num_draft[b]
 * (clamped to 0 .. max_draft) tokens d_i = draft_tokens[b][i] drawn from the
 * drafter's distributions q_draft[b][i][:]; the verify pass gave the target's
 * distributions p_target[b][i][:] for i = 0 .. gamma_b (row gamma_b follows
 * the last draft).  Draft i is accepted while u_accept[b][i] * q <= p (a
 * draft id outside [0, vocab) is rejected); at the first rejection k the next
 * token is drawn from max(0, p_k - q_k) (from p_k if that is all zero), after
 * full acceptance from p_gamma, as the smallest token whose cumulative mass
 * exceeds u_sample[b] times the total.  The rule is evaluated exactly, with no
 * rounding (the test on float64 products of the float32 inputs, the masses as
 * integers in units of 2^-149), so the result does not depend on summation
 * order.  Probabilities are clamped to [0, 1] and uniforms to [0, 1 - 2^-24],
 * NaN read as 0.  Writes num_accepted[b] (0 .. gamma_b) and next_token[b]
 * (-1 if the sampling row has no mass at all).
 *   p_target  fp32 [num_seqs][max_draft + 1][vocab], 16-byte aligned
 *   q_draft   fp32 [num_seqs][max_draft][vocab] (may be NULL if max_draft 0)
 *   draft_tokens, u_accept  [num_seqs][max_draft];  num_draft, u_sample,
 *   num_accepted, next_token  [num_seqs]; uniforms in [0, 1).
 * The caller supplies the random numbers, so results are reproducible.  The
 * workspace (ts_spec_accept_workspace_size bytes, 256-byte aligned, any
 * contents) holds the exact block sums and the per-sequence accepted counts
 * between the call's two launches. */
int ts_spec_accept(int32_t num_seqs, int32_t vocab, int32_t max_draft, const float *p_target,
                   const float *q_draft, const int32_t *draft_tokens, const int32_t *num_draft,
                   const float *u_accept, const float *u_sample, int32_t *num_accepted,
                   int32_t *next_token, void *workspace, size_t workspace_bytes, void *stream);

/* ---- replica completion-time model ------------------------------------------
 * Host-only (no GPU needed).  The paper turns the measured per-token decoding
 * time tau(b) = 1 / v(b) at active batch b (Sec. 2.1) into rollout time under
 * the all-admit model: a replica serving requests of completion lengths L_i
 * decodes position x with b(x) = #{i : L_i >= x} requests active, at cost
 * tau(b(x)).  Its completion time is
 *     T = sum_x tau(b(x)) = sum_j tau(j) (L_j - L_{j+1})   (L sorted descending)
 * (Sec. 2.1; App. D), request i's share of it is sum_{x <= L_i} tau(b(x)) /
 * b(x) (App. D; the shares add up to T), and a rollout step's makespan is the
 * largest T over the replicas (App. D).  `tau` arrays are dense tables with
 * tau[b - 1] = tau(b) for b = 1 .. bmax, in any time unit (results are in the
 * same unit); lengths are tokens (>= 0).  All entry points return TS_OK or a
 * negative ts_status with ts_last_error() set, and write nothing on error. */

/* Dense table tau_dense[b - 1], b = 1 .. bmax, from m measured points
 * (batch[k], tau[k]) with strictly increasing batch sizes >= 1: linear between
 * points, the first value below the first point, linear extrapolation of the
 * last segment past the last point (clamped at 0). */
int ts_tau_table(const int32_t *batch, const double *tau, int32_t m, int32_t bmax, double *tau_dense);

/* Completion time of one replica holding n requests (n <= bmax). */
int ts_replica_time(const double *tau, int32_t bmax, const int64_t *lengths, int32_t n, double *T);

/* Each request's share of its replica's completion time (shares[i] for
 * lengths[i]; equal lengths get equal shares). */
int ts_request_shares(const double *tau, int32_t bmax, const int64_t *lengths, int32_t n,
                      double *shares);

/* Rollout-step makespan of an assignment: request i runs on replica
 * replica[i] in [0, n_replicas); writes each replica's completion time to
 * T_replica[r] and their maximum to *T_step.  Each replica may hold at most
 * bmax requests. */
int ts_step_makespan(const double *tau, int32_t bmax, const int64_t *lengths, const int32_t *replica,
                     int32_t n, int32_t n_replicas, double *T_replica, double *T_step);

/* ---- synthetic inputs (same definitions as the test generator) -------------
 * SplitMix64 (Steele, Lea, Flood 2014) addressed by (seed, stream, index):
 * value n = mix64(mix64((seed << 8) + stream) + (n + 1) * 0x9E3779B97F4A7C15);
 * a bf16 value is the Box-Muller normal sqrt(-2 ln u1) cos(2 pi u2), u1 =
 * (hi32 + 1) / 2^32, u2 = lo32 / 2^32, computed in double, rounded to float
 * then to bf16 (nearest even). */

/* Fill n bf16 values dst[i] = normal(seed, stream_id, index_offset + i) on
 * `stream` (device memory). */
int ts_synth_fill_bf16(void *dst, int64_t n, uint64_t seed, uint32_t stream_id,
                       int64_t index_offset, void *stream);

/* Host: context lengths of the sweep distribution for `batch` sequences. */
int ts_synth_sweep_lengths(int32_t batch, uint64_t seed, int32_t *ctx_lens);

/* Host: physical page ids for sequences of the given lengths, a uniform
 * permutation of [0, total pages) (stable order of SplitMix64 keys), laid out
 * [batch][max_pages_per_seq] with unused entries set to 0. */
int ts_synth_page_table(int32_t batch, const int32_t *ctx_lens, int32_t page_size,
                        int32_t max_pages_per_seq, uint64_t seed, int32_t *page_table);

/* ---- measurement helpers ----------------------------------------------------- */

/* Plain device-to-device copy kernel of `bytes` (multiple of 16, 16-byte
 * aligned pointers); calibrates hardware byte counters against a known
 * transfer. */
int ts_copy_bytes(void *dst, const void *src, size_t bytes, void *stream);

/* Plain streaming read of `bytes` (multiple of 16, 16-byte aligned): every
 * word is loaded once by a grid of 2,048 blocks of 256 threads, each block
 * reading one contiguous stretch, and the XOR of the 32-bit words each thread
 * read is written to `sink` (at least 2 MiB, uint32 per thread; the XOR of
 * the whole sink is the XOR of every word of `src`).  Its bandwidth is the
 * practical sequential HBM read ceiling. */
int ts_stream_read(const void *src, size_t bytes, void *sink, size_t sink_bytes, void *stream);

/* Read-only twin of ts_decode_attn: streams exactly the K and V pages a call
 * with the same shape, pools, page table and lengths would read (the whole
 * 16 x head_dim block of every KV head for pages 0 .. ceil(L/16) - 1 of each
 * sequence with q_lens > 0), in the same worker partition and with the same
 * loads, and computes nothing.  Its bandwidth is the ceiling of the paged
 * (random 4 KiB block) access pattern on this GPU, which the attention kernels
 * are compared with.
 *   shape      as for ts_decode_attn (all its checks apply; num_workers 0
 *              means 1,024 wavefronts, 4 per compute unit);
 *   sink       device, at least workers x 64 x 4 bytes: the XOR of the 32-bit
 *              words each lane read (the XOR of the whole sink is the XOR of
 *              every word of the pages read);
 *   ev_begin, ev_end  optional HIP events (NULL allowed) that take the
 *              kernel's own start and end timestamps.
 * Asynchronous on `stream`; device-value preconditions as for
 * ts_decode_attn. */
int ts_page_gather_read(const ts_attn_shape *shape, const void *k_pages, const void *v_pages,
                        const int32_t *page_table, const int32_t *ctx_lens, const int32_t *q_lens,
                        void *sink, size_t sink_bytes, void *stream, void *ev_begin, void *ev_end);

int ts_event_create(void **ev);
int ts_event_destroy(void *ev);
int ts_event_record(void *ev, void *stream);
/* Waits for `stop` and returns the time from `start` to `stop` in ms. */
int ts_event_elapsed_ms(void *start, void *stop, float *ms);

/* ---- diagnostics ------------------------------------------------------------ */
const char *ts_status_string(int status);
/* Message of the last failing call on this thread ("" if none). */
const char *ts_last_error(void);
int ts_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TS_ATTN_H */
