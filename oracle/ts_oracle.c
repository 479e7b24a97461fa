/*
 * ts_oracle.c -- reference paged decode / speculative-verify attention in
 * float64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * loads this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it, to decide whether the GPU kernels are right and to
 * time a plain CPU implementation beside them.  It shares no code, header,
 * table or helper with the GPU path.
 *
 * What it computes.  The paper studies the decode phase of rollout
 * generation (Sec. 2.1) and verifies speculative drafts with the target
 * model (Sec. 3.4, lossless speculative decoding); each such step runs
 * scaled-dot-product attention of the new query tokens against every cached
 * key/value of the sequence.  The paper writes no formula for it, so this is
 * the textbook definition, instantiated for a paged KV cache:
 *
 *   for sequence b with context length L (which already counts the Q new
 *   tokens) and query row i in [0, Q), query head h, KV head g = h / G:
 *     key t is visible iff 0 <= t <= L - Q + i     (causal in the draft block)
 *     K_t = k_pages[page_table[b][t / P]][g][t % P][:], V_t likewise
 *     s_t = scale * <q[b][i][h][:], K_t>
 *     w_t = exp(s_t - max_t s_t) / sum_t exp(s_t - max_t s_t)
 *     o[b][i][h][:] = sum_t w_t V_t
 *
 * bf16 inputs are widened exactly to double; every sum is a plain
 * left-to-right loop in double.  Rows i >= q_lens[b] are not written.
 *
 * Pins (in the test suite): dense brute force and torch's CPU attention on
 * tiny inputs, closed forms (one key, zero scale, equal keys, constant V),
 * hand-derived golden cases, page-relabel / head / batch permutation
 * invariance, key-shift invariance, linearity in V, the verify-row vs
 * prefix-decode identity, split-and-merge equality, and mutants of this file
 * that each must fail at least one pin.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

static double widen_bf16(uint16_t bits)
{
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Offset of element (page p, kv head g, slot u, dim d) in a page pool laid
 * out [num_pages][Hkv][P][D]. */
static size_t pool_at(int64_t p, int g, int u, int d, int Hkv, int P, int D)
{
    return (((size_t)p * (size_t)Hkv + (size_t)g) * (size_t)P + (size_t)u) * (size_t)D + (size_t)d;
}

/* Offset of element (b, i, h, d) of a [B][Qmax][Hq][D] tensor. */
static size_t row_at(int b, int i, int h, int d, int Qmax, int Hq, int D)
{
    return (((size_t)b * (size_t)Qmax + (size_t)i) * (size_t)Hq + (size_t)h) * (size_t)D + (size_t)d;
}

typedef struct {
    int B, Hq, Hkv, D, P, Qmax, max_pages;
    const uint16_t *q, *kp, *vp;
    const int32_t *page_table, *ctx_lens, *q_lens;
    double scale;
} problem;

/* Attention of one query row over the visible keys t in [t_begin, t_end).
 * Writes the normalised output o[D] and lse = max + log(sum exp(s - max));
 * an empty key range gives o = 0 and lse = -inf.  ``s`` is scratch of at
 * least t_end - t_begin doubles. */
static void attend_row(const problem *pr, int b, int i, int h, int t_begin, int t_end,
                       double *o, double *lse, double *s)
{
    const int L = pr->ctx_lens[b];
    const int Q = pr->q_lens[b];
    const int G = pr->Hq / pr->Hkv;
    const int g = h / G;
    const int last_visible = L - Q + i;          /* inclusive */
    int hi = t_end;
    if (hi > last_visible + 1)
        hi = last_visible + 1;
    int lo = t_begin < 0 ? 0 : t_begin;

    for (int d = 0; d < pr->D; d++)
        o[d] = 0.0;
    if (hi <= lo) {
        *lse = -INFINITY;
        return;
    }

    /* scores */
    double m = -INFINITY;
    for (int t = lo; t < hi; t++) {
        int64_t page = pr->page_table[(size_t)b * pr->max_pages + t / pr->P];
        int slot = t % pr->P;
        double acc = 0.0;
        for (int d = 0; d < pr->D; d++) {
            double qv = widen_bf16(pr->q[row_at(b, i, h, d, pr->Qmax, pr->Hq, pr->D)]);
            double kv = widen_bf16(pr->kp[pool_at(page, g, slot, d, pr->Hkv, pr->P, pr->D)]);
            acc += qv * kv;
        }
        s[t - lo] = pr->scale * acc;
        if (s[t - lo] > m)
            m = s[t - lo];
    }

    /* softmax weights (unnormalised) and their sum */
    double l = 0.0;
    for (int t = lo; t < hi; t++) {
        s[t - lo] = exp(s[t - lo] - m);
        l += s[t - lo];
    }

    /* weighted sum of values */
    for (int t = lo; t < hi; t++) {
        int64_t page = pr->page_table[(size_t)b * pr->max_pages + t / pr->P];
        int slot = t % pr->P;
        for (int d = 0; d < pr->D; d++)
            o[d] += s[t - lo] * widen_bf16(pr->vp[pool_at(page, g, slot, d, pr->Hkv, pr->P, pr->D)]);
    }
    for (int d = 0; d < pr->D; d++)
        o[d] /= l;
    *lse = m + log(l);
}

static int max_ctx(const problem *pr)
{
    int m = 1;
    for (int b = 0; b < pr->B; b++)
        if (pr->ctx_lens[b] > m)
            m = pr->ctx_lens[b];
    return m;
}

/* Attention over the key sub-range [t_begin, t_end) of every row; the full
 * definition is t_begin = 0, t_end >= L.  out: [B][Qmax][Hq][D]; lse (may be
 * NULL): [B][Qmax][Hq].  Rows i >= q_lens[b] are left untouched. */
static void run(const problem *pr, int t_begin, int t_end, double *out, double *lse, int nthreads)
{
    const int scratch = max_ctx(pr);
    const int BH = pr->B * pr->Hq;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
#endif
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)scratch);
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int bh = 0; bh < BH; bh++) {
            int b = bh / pr->Hq, h = bh % pr->Hq;
            for (int i = 0; i < pr->q_lens[b]; i++) {
                double row_lse;
                int hi = t_end < pr->ctx_lens[b] ? t_end : pr->ctx_lens[b];
                attend_row(pr, b, i, h, t_begin, hi, out + row_at(b, i, h, 0, pr->Qmax, pr->Hq, pr->D),
                           &row_lse, s);
                if (lse)
                    lse[((size_t)b * pr->Qmax + i) * pr->Hq + h] = row_lse;
            }
        }
        free(s);
    }
    (void)nthreads;
}

/* Full paged attention: out[b][i][h][:] for i < q_lens[b]. */
void ts_oracle_paged_attention(int B, int Hq, int Hkv, int D, int P, int Qmax, int max_pages,
                               const uint16_t *q, const uint16_t *k_pages, const uint16_t *v_pages,
                               const int32_t *page_table, const int32_t *ctx_lens,
                               const int32_t *q_lens, double scale, double *out, int nthreads)
{
    problem pr = {B, Hq, Hkv, D, P, Qmax, max_pages, q, k_pages, v_pages,
                  page_table, ctx_lens, q_lens, scale};
    run(&pr, 0, 1 << 30, out, NULL, nthreads);
}

/* Attention restricted to keys [t_begin, t_end): normalised partial output
 * and its log-sum-exp (natural log); empty rows give o = 0, lse = -inf. */
void ts_oracle_partial_attention(int B, int Hq, int Hkv, int D, int P, int Qmax, int max_pages,
                                 const uint16_t *q, const uint16_t *k_pages, const uint16_t *v_pages,
                                 const int32_t *page_table, const int32_t *ctx_lens,
                                 const int32_t *q_lens, double scale, int t_begin, int t_end,
                                 double *out, double *lse, int nthreads)
{
    problem pr = {B, Hq, Hkv, D, P, Qmax, max_pages, q, k_pages, v_pages,
                  page_table, ctx_lens, q_lens, scale};
    run(&pr, t_begin, t_end, out, lse, nthreads);
}

/* Combine partial results over disjoint key ranges:
 *   M = max_s lse_s,  w_s = exp(lse_s - M),  o = sum_s w_s o_s / sum_s w_s.
 * o_parts: [nsplit][nrows][D], lse_parts: [nsplit][nrows], out: [nrows][D].
 * A split with lse = -inf has weight 0. */
void ts_oracle_lse_merge(int nsplit, int64_t nrows, int D, const double *o_parts,
                         const double *lse_parts, double *out)
{
    for (int64_t r = 0; r < nrows; r++) {
        double M = -INFINITY;
        for (int s = 0; s < nsplit; s++)
            if (lse_parts[(size_t)s * nrows + r] > M)
                M = lse_parts[(size_t)s * nrows + r];
        double wsum = 0.0;
        for (int d = 0; d < D; d++)
            out[(size_t)r * D + d] = 0.0;
        if (M == -INFINITY)
            continue;
        for (int s = 0; s < nsplit; s++) {
            double lse = lse_parts[(size_t)s * nrows + r];
            if (lse == -INFINITY)
                continue;
            double w = exp(lse - M);
            wsum += w;
            for (int d = 0; d < D; d++)
                out[(size_t)r * D + d] += w * o_parts[((size_t)s * nrows + r) * D + d];
        }
        for (int d = 0; d < D; d++)
            out[(size_t)r * D + d] /= wsum;
    }
}

/* Softmax weights of one row over all L keys of sequence b (0 for keys the
 * row cannot see).  w: [ctx_lens[b]].  Exposes the probabilities so a test
 * can check that they sum to one and reproduce the output. */
void ts_oracle_row_weights(int B, int Hq, int Hkv, int D, int P, int Qmax, int max_pages,
                           const uint16_t *q, const uint16_t *k_pages, const uint16_t *v_pages,
                           const int32_t *page_table, const int32_t *ctx_lens,
                           const int32_t *q_lens, double scale, int b, int i, int h, double *w)
{
    const int L = ctx_lens[b];
    const int G = Hq / Hkv;
    const int g = h / G;
    const int last_visible = L - q_lens[b] + i;
    double m = -INFINITY;
    for (int t = 0; t < L; t++) {
        w[t] = 0.0;
        if (t > last_visible)
            continue;
        int64_t page = page_table[(size_t)b * max_pages + t / P];
        double acc = 0.0;
        for (int d = 0; d < D; d++)
            acc += widen_bf16(q[row_at(b, i, h, d, Qmax, Hq, D)]) *
                   widen_bf16(k_pages[pool_at(page, g, t % P, d, Hkv, P, D)]);
        w[t] = scale * acc;
        if (w[t] > m)
            m = w[t];
    }
    double l = 0.0;
    for (int t = 0; t <= last_visible && t < L; t++) {
        w[t] = exp(w[t] - m);
        l += w[t];
    }
    for (int t = 0; t <= last_visible && t < L; t++)
        w[t] /= l;
    (void)B;
}

int ts_oracle_version(void) { return 1; }
