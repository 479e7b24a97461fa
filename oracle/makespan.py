"""Replica completion time under the all-admit decoding model, written out
position by position (paper App. D, "Exact Makespan and Tail-Side Proxy";
Sec. 2.1 for tau).

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark may call
this module; the product library never does.  It shares nothing with the
library's implementation (``ts_replica_time`` and friends), which computes the
same quantities from sorted lengths in O(n log n).

Definitions (App. D).  A replica serves a set of requests with completion
lengths L_i (tokens).  At decoding position x = 1, 2, ... the active batch is
b(x) = #{i : L_i >= x}, and decoding that position costs tau(b(x)) of wall
time, tau(b) being the per-token decoding time at active batch b (Sec. 2.1:
tau(b) = 1 / v(b)).  Then
  * the replica's completion time is  T = sum_{x=1}^{max_i L_i} tau(b(x));
  * request i's share of it is  sum_{x=1}^{L_i} tau(b(x)) / b(x), and the
    shares add up to T because exactly b(x) requests are active at x;
  * the rollout step's makespan is the largest T over the replicas.
``tau`` is a table with tau[b - 1] = tau(b) for b = 1 .. len(tau).
Plain loops over positions: meant for checking, not speed.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple


def active_batch(lengths: Sequence[int], x: int) -> int:
    """b(x): requests still decoding at position x (1-based)."""
    return sum(1 for L in lengths if L >= x)


def _tau_at(tau: Sequence[float], b: int) -> float:
    if b < 1 or b > len(tau):
        raise ValueError(f"tau is tabulated for b = 1..{len(tau)}, needed b = {b}")
    return float(tau[b - 1])


def replica_time(tau: Sequence[float], lengths: Sequence[int]) -> float:
    """T = sum over positions x = 1 .. max L of tau(b(x))."""
    lmax = max(lengths, default=0)
    total = 0.0
    for x in range(1, lmax + 1):
        total += _tau_at(tau, active_batch(lengths, x))
    return total


def request_shares(tau: Sequence[float], lengths: Sequence[int]) -> List[float]:
    """Share of request i: sum over x = 1 .. L_i of tau(b(x)) / b(x)."""
    lmax = max(lengths, default=0)
    shares = [0.0] * len(lengths)
    for x in range(1, lmax + 1):
        b = active_batch(lengths, x)
        per = _tau_at(tau, b) / b
        for i, L in enumerate(lengths):
            if L >= x:
                shares[i] += per
    return shares


def step_makespan(tau: Sequence[float], lengths: Sequence[int], replica: Sequence[int],
                  n_replicas: int) -> Tuple[List[float], float]:
    """Completion time of every replica (its assigned requests alone) and
    their maximum, the rollout step's makespan."""
    times = []
    for r in range(n_replicas):
        times.append(replica_time(tau, [L for L, k in zip(lengths, replica) if k == r]))
    return times, max(times, default=0.0)
