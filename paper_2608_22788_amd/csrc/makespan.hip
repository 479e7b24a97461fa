// makespan.hip -- the replica completion-time model that turns a measured
// per-token decoding time tau(b) into rollout time (paper Sec. 2.1 and
// App. D).  Host code only: no kernel, no HIP call, so it also runs on a
// machine without a GPU.
//
// Under the all-admit model a replica decodes every assigned request from the
// start; at position x the active batch is b(x) = #{i : L_i >= x} and the
// position costs tau(b(x)).  With the lengths sorted in descending order
// (L_1 >= ... >= L_n, L_{n+1} = 0) exactly j requests are active on the
// positions (L_{j+1}, L_j], so the completion time is
//     T = sum_j tau(j) (L_j - L_{j+1})                      (Sec. 2.1)
// and request k (in that order) owns the share
//     S_k = sum_{j >= k} tau(j) (L_j - L_{j+1}) / j          (App. D)
// of it, because the j requests active on such a position split its time
// evenly.  Sorting makes both O(n log n), where the position-by-position
// definition costs O(n max L).  Ties need no special case: equal lengths give
// empty intervals.  tau between measured batch sizes is taken piecewise
// linear (the paper measures v(b) at chosen batch sizes and gives no rule).
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "ts_attn.h"
#include "ts_internal.h"

namespace tsattn {
namespace {

int check_tau(const double *tau, int32_t bmax) {
    if (!tau)
        return fail(TS_ERR_NULL, "tau is NULL");
    if (bmax < 1)
        return fail(TS_ERR_ARG, "bmax %d < 1", bmax);
    for (int32_t b = 0; b < bmax; b++)
        if (!std::isfinite(tau[b]) || tau[b] < 0.0)
            return fail(TS_ERR_ARG, "tau(%d) = %g is not a finite non-negative time", b + 1, tau[b]);
    return TS_OK;
}

int check_lengths(const int64_t *lengths, int32_t n, int32_t bmax) {
    if (n < 0)
        return fail(TS_ERR_ARG, "n %d < 0", n);
    if (n > 0 && !lengths)
        return fail(TS_ERR_NULL, "lengths is NULL");
    if (n > bmax)
        return fail(TS_ERR_ARG, "%d requests but tau is tabulated only up to b = %d", n, bmax);
    for (int32_t i = 0; i < n; i++)
        if (lengths[i] < 0)
            return fail(TS_ERR_ARG, "lengths[%d] = %lld < 0", i, (long long)lengths[i]);
    return TS_OK;
}

// Indices of `lengths` in descending length order (stable).
std::vector<int32_t> order_desc(const int64_t *lengths, int32_t n) {
    std::vector<int32_t> idx((size_t)n);
    std::iota(idx.begin(), idx.end(), 0);
    std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) { return lengths[a] > lengths[b]; });
    return idx;
}

double replica_time(const double *tau, const int64_t *lengths, const std::vector<int32_t> &idx) {
    const size_t n = idx.size();
    double T = 0.0;
    for (size_t j = 0; j < n; j++) {
        const int64_t Lj = lengths[idx[j]];
        const int64_t Lnext = j + 1 < n ? lengths[idx[j + 1]] : 0;
        T += tau[j] * (double)(Lj - Lnext);   // tau(j + 1): j + 1 requests active
    }
    return T;
}

}  // namespace
}  // namespace tsattn

using namespace tsattn;

extern "C" {

int ts_tau_table(const int32_t *batch, const double *tau, int32_t m, int32_t bmax, double *tau_dense) {
    clear_error();
    if (!batch || !tau || !tau_dense)
        return fail(TS_ERR_NULL, "NULL argument");
    if (m < 1 || bmax < 1)
        return fail(TS_ERR_ARG, "need m >= 1 measured points and bmax >= 1 (m %d, bmax %d)", m, bmax);
    for (int32_t k = 0; k < m; k++) {
        if (batch[k] < 1 || (k > 0 && batch[k] <= batch[k - 1]))
            return fail(TS_ERR_ARG, "measured batch sizes must be >= 1 and strictly increasing (at %d)", k);
        if (!std::isfinite(tau[k]) || tau[k] < 0.0)
            return fail(TS_ERR_ARG, "measured tau[%d] = %g is not a finite non-negative time", k, tau[k]);
    }
    for (int32_t b = 1; b <= bmax; b++) {
        double t;
        if (m == 1 || b <= batch[0]) {
            t = tau[0];   // below the first point: its value
        } else {
            // the segment that holds b, or the last one (linear extrapolation)
            int32_t k = 1;
            while (k < m - 1 && batch[k] < b)
                k++;
            const double b0 = batch[k - 1], b1 = batch[k];
            t = tau[k - 1] + (tau[k] - tau[k - 1]) * ((double)b - b0) / (b1 - b0);
            if (t < 0.0)
                t = 0.0;
        }
        tau_dense[b - 1] = t;
    }
    return TS_OK;
}

int ts_replica_time(const double *tau, int32_t bmax, const int64_t *lengths, int32_t n, double *T) {
    clear_error();
    if (!T)
        return fail(TS_ERR_NULL, "T is NULL");
    int st = check_tau(tau, bmax);
    if (st || (st = check_lengths(lengths, n, bmax)))
        return st;
    try {
        *T = replica_time(tau, lengths, order_desc(lengths, n));
        return TS_OK;
    } catch (...) {
        return fail(TS_ERR_HIP, "out of host memory");
    }
}

int ts_request_shares(const double *tau, int32_t bmax, const int64_t *lengths, int32_t n, double *shares) {
    clear_error();
    if (n > 0 && !shares)
        return fail(TS_ERR_NULL, "shares is NULL");
    int st = check_tau(tau, bmax);
    if (st || (st = check_lengths(lengths, n, bmax)))
        return st;
    try {
        const std::vector<int32_t> idx = order_desc(lengths, n);
        double suffix = 0.0;   // sum over j >= k of tau(j) (L_j - L_{j+1}) / j
        for (int32_t k = n - 1; k >= 0; k--) {
            const int64_t Lk = lengths[idx[(size_t)k]];
            const int64_t Lnext = k + 1 < n ? lengths[idx[(size_t)k + 1]] : 0;
            suffix += tau[k] * (double)(Lk - Lnext) / (double)(k + 1);
            shares[idx[(size_t)k]] = suffix;
        }
        return TS_OK;
    } catch (...) {
        return fail(TS_ERR_HIP, "out of host memory");
    }
}

int ts_step_makespan(const double *tau, int32_t bmax, const int64_t *lengths, const int32_t *replica,
                     int32_t n, int32_t n_replicas, double *T_replica, double *T_step) {
    clear_error();
    if (!T_step || (n_replicas > 0 && !T_replica) || (n > 0 && !replica))
        return fail(TS_ERR_NULL, "NULL argument");
    if (n_replicas < 1)
        return fail(TS_ERR_ARG, "n_replicas %d < 1", n_replicas);
    int st = check_tau(tau, bmax);
    if (st)
        return st;
    if (n < 0 || (n > 0 && !lengths))
        return fail(TS_ERR_ARG, "invalid request count or NULL lengths");
    try {
        std::vector<std::vector<int64_t>> per((size_t)n_replicas);
        for (int32_t i = 0; i < n; i++) {
            if (replica[i] < 0 || replica[i] >= n_replicas)
                return fail(TS_ERR_ARG, "replica[%d] = %d outside [0, %d)", i, replica[i], n_replicas);
            if (lengths[i] < 0)
                return fail(TS_ERR_ARG, "lengths[%d] = %lld < 0", i, (long long)lengths[i]);
            per[(size_t)replica[i]].push_back(lengths[i]);
        }
        double worst = 0.0;
        for (int32_t r = 0; r < n_replicas; r++) {
            const std::vector<int64_t> &L = per[(size_t)r];
            if ((int64_t)L.size() > bmax)
                return fail(TS_ERR_ARG, "replica %d holds %zu requests but tau is tabulated only up to b = %d",
                            r, L.size(), bmax);
            const double t = replica_time(tau, L.data(), order_desc(L.data(), (int32_t)L.size()));
            T_replica[r] = t;
            worst = std::max(worst, t);
        }
        *T_step = worst;
        return TS_OK;
    } catch (...) {
        return fail(TS_ERR_HIP, "out of host memory");
    }
}

}  // extern "C"
