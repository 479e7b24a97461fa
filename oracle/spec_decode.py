"""The steps on either side of the verify attention in one speculative
decoding step: writing the new tokens' keys and values into the paged cache,
and deciding which drafted tokens the target model accepts.  Plain numpy,
for checking only.

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

Readings where the description leaves a choice:
  * the test u <= p/q is evaluated as u * q <= p in float32 (the precision of
    the probabilities), so both sides take the same decision; q(d) = 0 with
    p(d) > 0 accepts, 0 <= 0 accepts (a token neither model can produce
    never occurs in practice);
  * a draft token outside the vocabulary is rejected;
  * the next token is drawn by inverse CDF: the smallest token v whose
    cumulative (unnormalised) mass exceeds u_sample times the total;
  * if the leftover mass is zero (p_k == q_k up to rounding) the next token
    is drawn from p_k itself.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


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


def accept_walk(p_target, q_draft, draft, gamma, u_accept) -> int:
    """Number of leading drafts accepted for one sequence."""
    V = p_target.shape[-1]
    for i in range(gamma):
        d = int(draft[i])
        if d < 0 or d >= V:
            return i
        lhs = np.float32(u_accept[i]) * np.float32(q_draft[i, d])
        if not lhs <= np.float32(p_target[i, d]):
            return i
    return gamma


def sample_inverse_cdf(weights: np.ndarray, u: float, tol: float = 1e-5) -> Tuple[int, bool]:
    """Smallest v with cumsum(weights)[v] > u * sum(weights), in float64;
    also whether u * sum lies within tol * sum of a cumulative boundary (then
    a float32 evaluation may pick a neighbour)."""
    w = np.asarray(weights, dtype=np.float64)
    c = np.cumsum(w)
    Z = c[-1]
    target = float(u) * Z
    v = int(np.searchsorted(c, target, side="right"))
    v = min(v, len(w) - 1)
    while w[v] == 0.0 and v > 0:            # never land on a zero-mass token
        v -= 1
    near = bool(np.any(np.abs(c - target) <= tol * Z))
    return v, near


def spec_accept(p_target, q_draft, draft_tokens, num_draft, u_accept, u_sample, tol=1e-5):
    """Per sequence: (accepted draft count, next token, decision near a
    boundary).  p_target [B][Gmax+1][V], q_draft [B][Gmax][V] (float32
    probabilities), draft_tokens [B][Gmax], num_draft [B], u_accept [B][Gmax],
    u_sample [B]."""
    B = len(num_draft)
    n_acc = np.zeros(B, dtype=np.int32)
    nxt = np.zeros(B, dtype=np.int32)
    near = np.zeros(B, dtype=bool)
    for b in range(B):
        g = int(num_draft[b])
        k = accept_walk(p_target[b], q_draft[b], draft_tokens[b], g, u_accept[b])
        n_acc[b] = k
        if k < g:
            w = np.maximum(0.0, p_target[b, k].astype(np.float64) - q_draft[b, k].astype(np.float64))
            if w.sum() <= 0.0:
                w = p_target[b, k].astype(np.float64)
        else:
            w = p_target[b, g].astype(np.float64)
        nxt[b], near[b] = sample_inverse_cdf(w, float(u_sample[b]), tol)
    return n_acc, nxt, near
