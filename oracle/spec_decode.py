"""The steps on either side of the verify attention in one speculative
decoding step: writing the new tokens' keys and values into the paged cache,
and deciding which drafted tokens the target model accepts.  Plain numpy and
Python integers, for checking only.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark may call
this module; the product library never does, and nothing here is shared with
it.

KV append (the layout of the attention path).  Sequence b holds
L = ctx_lens[b] tokens of which the last Q = q_lens[b] are the step's new
ones, so new row i (i < Q) is token t = L - Q + i and lands in
k_pages[page_table[b][t // P]][g][t % P][:] (same for v), for every KV head g.

Acceptance (paper Sec. 3.4 verifies drafts with the target model and keeps
its output distribution, following the speculative sampling of Leviathan,
Kalman and Matias, 2023).  A sequence proposes gamma draft tokens d_0..d_{g-1}
drawn from the drafter's distributions q_0..q_{g-1}; the verify pass yields the
target's distributions p_0..p_gamma at the same positions (p_gamma follows
the last draft).  Walking i = 0, 1, ...: draft i is accepted when
u_i <= p_i(d_i) / q_i(d_i) for a fresh uniform u_i; the first rejection at
position k ends the walk and the next token is drawn from the leftover mass
max(0, p_k - q_k) renormalised; if every draft is accepted the next token is
drawn from p_gamma.  The emitted tokens are then distributed exactly as the
target model alone would produce them.

The rule is stated over real numbers, and it is evaluated here exactly, with
no rounding anywhere, so that any other exact evaluation gives the same
integers:
  * every probability is first clamped to [0, 1] (NaN read as 0) and every
    uniform to [0, 1 - 2^-24] (NaN read as 0): probabilities are
    float32 values, and these are the only inputs the rule is defined on;
  * the test u <= p/q is u * q <= p over the reals (q(d) = 0 accepts, and
    so does 0 <= 0);
  * a draft token outside the vocabulary is rejected;
  * the next token is the smallest v whose cumulative weight
    C_v = w_0 + ... + w_v exceeds u_sample times the total Z (inverse CDF;
    a boundary C_v = u Z belongs to the next token).  Because u < 1 such a v
    exists and carries weight;
  * if the leftover mass is zero the next token is drawn from p_k itself; a
    sampling row with no mass at all (invalid input) gives token -1.
A float32 value in [0, 1] is an integer multiple of 2^-149 (the smallest
positive subnormal), below 2^150 of them, so the weights and their sums are
held as Python integers in units of 2^-149.
"""
from __future__ import annotations

import bisect
import itertools
from fractions import Fraction

import numpy as np

UNIT_BITS = 149                     # 2^-149: the smallest positive float32
U_MAX = 1.0 - 2.0 ** -24            # the largest float32 below 1


def kv_append(k_pages, v_pages, page_table, ctx_lens, q_lens, k_new, v_new, page_size=16):
    """Copies of the pools with the new rows written.  k_new, v_new:
    [B][Qmax][Hkv][D]; pools [num_pages][Hkv][P][D]; any dtype."""
    k_out, v_out = k_pages.copy(), v_pages.copy()
    for b in range(len(ctx_lens)):
        L, Q = int(ctx_lens[b]), int(q_lens[b])
        for i in range(Q):
            t = L - Q + i
            page = int(page_table[b][t // page_size])
            k_out[page, :, t % page_size, :] = k_new[b, i]
            v_out[page, :, t % page_size, :] = v_new[b, i]
    return k_out, v_out


def clamp_prob(x) -> np.ndarray:
    """float32 probabilities as float64 in [0, 1], NaN read as 0 (exact)."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    return np.clip(np.where(np.isnan(x), 0.0, x), 0.0, 1.0)


def clamp_uniform(u) -> float:
    """A uniform as float in [0, 1 - 2^-24], NaN read as 0."""
    u = float(np.float32(u))
    if not u > 0.0:
        return 0.0
    return min(u, U_MAX)


def to_units(x) -> list:
    """Exact integers x * 2^149 of float32 values already clamped to [0, 1].
    Scaling a float64 by a power of two is exact here (no overflow), and the
    result is an integer-valued float, which int() converts exactly."""
    return [int(v) for v in (np.asarray(x, dtype=np.float64) * 2.0 ** UNIT_BITS).tolist()]


def accept_walk(p_target, q_draft, draft, gamma, u_accept) -> int:
    """Number of leading drafts accepted for one sequence (exact test)."""
    V = p_target.shape[-1]
    for i in range(gamma):
        d = int(draft[i])
        if d < 0 or d >= V:
            return i
        u = Fraction(clamp_uniform(u_accept[i]))
        q = Fraction(float(clamp_prob(q_draft[i, d])))
        p = Fraction(float(clamp_prob(p_target[i, d])))
        if not u * q <= p:
            return i
    return gamma


def sampling_weights(p_row, q_row=None) -> list:
    """Integer weights (units of 2^-149): max(0, p - q), or p if q_row is None."""
    P = to_units(clamp_prob(p_row))
    if q_row is None:
        return P
    Q = to_units(clamp_prob(q_row))
    return [a - b if a > b else 0 for a, b in zip(P, Q)]


def sample_inverse_cdf(weights: list, u: float) -> int:
    """Smallest v with w_0 + ... + w_v > u * sum(w), exactly (weights are
    integers); -1 if the weights sum to zero."""
    C = list(itertools.accumulate(weights))
    Z = C[-1] if C else 0
    if Z == 0:
        return -1
    target = Fraction(clamp_uniform(u)) * Z
    # C_v > target  <=>  C_v > floor(target), as C_v is an integer
    return bisect.bisect_right(C, int(target))


def spec_accept(p_target, q_draft, draft_tokens, num_draft, u_accept, u_sample):
    """Per sequence: (accepted draft count, next token).  p_target
    [B][Gmax+1][V], q_draft [B][Gmax][V] (float32 probabilities),
    draft_tokens [B][Gmax], num_draft [B], u_accept [B][Gmax], u_sample [B].
    num_draft is clamped to [0, Gmax]."""
    p_target = np.asarray(p_target)
    Gmax = p_target.shape[1] - 1
    B = len(num_draft)
    n_acc = np.zeros(B, dtype=np.int32)
    nxt = np.zeros(B, dtype=np.int32)
    for b in range(B):
        g = min(max(int(num_draft[b]), 0), Gmax)
        k = accept_walk(p_target[b], q_draft[b] if g else None, draft_tokens[b] if g else None, g,
                        u_accept[b] if g else None)
        n_acc[b] = k
        if k < g:
            w = sampling_weights(p_target[b, k], q_draft[b, k])
            if sum(w) == 0:
                w = sampling_weights(p_target[b, k])
        else:
            w = sampling_weights(p_target[b, g])
        nxt[b] = sample_inverse_cdf(w, float(u_sample[b]))
    return n_acc, nxt
