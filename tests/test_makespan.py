"""The replica completion-time model (paper Sec. 2.1 and App. D).

First the oracle (``oracle/makespan.py``, position-by-position sums) is pinned
to things the paper and arithmetic fix: a hand-worked example, the two closed
forms printed in Sec. 2.1, special cases with closed forms, the share identity
of App. D, the marginal-cost identity of Sec. 2.1, and planted mistakes that
must fail.  Then the library's O(n log n) implementation is checked against
the oracle, and its tau-table interpolation against numpy.  Host code only.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import makespan as om

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "makespan_example.json")))


def rand_case(rng, n, lmax, zeros=False):
    L = rng.integers(0 if zeros else 1, lmax + 1, size=n)
    if n > 3:
        L[rng.integers(0, n, size=2)] = L[0]           # ties
    tau = np.cumsum(rng.uniform(0.01, 1.0, size=max(n, 1)))  # increasing, as measured curves are
    return tau, L


# ---------------------------------------------------------------------------
# pins of the oracle
# ---------------------------------------------------------------------------

def pin_worked_example(om):
    tau, L = GOLD["tau"], GOLD["lengths"]
    assert om.replica_time(tau, L) == pytest.approx(float(Fraction(*GOLD["T"])), abs=1e-12)
    for got, frac in zip(om.request_shares(tau, L), GOLD["shares"]):
        assert got == pytest.approx(float(Fraction(*frac)), abs=1e-12)
    tr = GOLD["two_replicas"]
    times, T = om.step_makespan(tau, L, tr["replica"], 2)
    assert times == pytest.approx(tr["T_replica"]) and T == pytest.approx(tr["T_step"])


def closed_form_differences(tau, L):
    """Sec. 2.1, first form: sum_j tau(j) (L_j - L_{j+1}), L sorted descending."""
    s = sorted(L, reverse=True) + [0]
    return sum(tau[j] * (s[j] - s[j + 1]) for j in range(len(L)))


def closed_form_levels(tau, L):
    """Sec. 2.1, second form: sum_j L_j (tau(j) - tau(j - 1)), tau(0) = 0."""
    s = sorted(L, reverse=True)
    return sum(s[j] * (tau[j] - (tau[j - 1] if j else 0.0)) for j in range(len(L)))


def pin_closed_forms(om, seed):
    rng = np.random.default_rng(seed)
    tau, L = rand_case(rng, int(rng.integers(1, 40)), 300, zeros=seed % 2 == 1)
    T = om.replica_time(tau, L.tolist())
    assert T == pytest.approx(closed_form_differences(tau, L.tolist()), rel=1e-12)
    assert T == pytest.approx(closed_form_levels(tau, L.tolist()), rel=1e-12)


def pin_special_cases(om):
    # constant per-token time: the replica takes as long as its longest request
    assert om.replica_time([2.5] * 6, [7, 3, 9, 1, 9, 4]) == pytest.approx(2.5 * 9)
    # time proportional to the batch: every token costs the same, T = c * sum L
    c = 0.3
    assert om.replica_time([c * b for b in range(1, 7)], [7, 3, 9, 1, 9, 4]) == pytest.approx(c * 33)
    # equal lengths: b = n throughout, shares equal
    tau = [1.0, 1.7, 2.1, 2.6]
    assert om.replica_time(tau, [5] * 4) == pytest.approx(2.6 * 5)
    assert om.request_shares(tau, [5] * 4) == pytest.approx([2.6 * 5 / 4] * 4)
    # a single request runs alone
    assert om.replica_time(tau, [11]) == pytest.approx(11.0)
    # nothing to decode
    assert om.replica_time(tau, []) == 0.0 and om.request_shares(tau, []) == []
    # zero-length requests never become active
    assert om.replica_time(tau, [0, 4, 0]) == pytest.approx(4.0)
    assert om.request_shares(tau, [0, 4, 0]) == pytest.approx([0.0, 4.0, 0.0])


def pin_shares(om, seed):
    rng = np.random.default_rng(100 + seed)
    tau, L = rand_case(rng, int(rng.integers(1, 30)), 200)
    sh = om.request_shares(tau, L.tolist())
    assert sum(sh) == pytest.approx(om.replica_time(tau, L.tolist()), rel=1e-12)
    # a longer request is active on a superset of positions
    order = np.argsort(L)
    assert all(sh[order[k]] <= sh[order[k + 1]] + 1e-12 for k in range(len(L) - 1))


def pin_marginal_costs(om, seed):
    """Sec. 2.1: a request of length L joining a replica that holds c longer
    requests (and no shorter ones) adds L (tau(c + 1) - tau(c))."""
    rng = np.random.default_rng(200 + seed)
    tau, L = rand_case(rng, int(rng.integers(1, 30)), 200)
    held, total = [], 0.0
    for c, x in enumerate(sorted(L.tolist(), reverse=True)):
        before = om.replica_time(tau, held)
        held.append(x)
        delta = om.replica_time(tau, held) - before
        assert delta == pytest.approx(x * (tau[c] - (tau[c - 1] if c else 0.0)), abs=1e-9)
        total += delta
    assert total == pytest.approx(om.replica_time(tau, L.tolist()), rel=1e-12)


def pin_order_and_step_makespan(om):
    rng = np.random.default_rng(7)
    tau, L = rand_case(rng, 25, 120)
    perm = rng.permutation(len(L))
    assert om.replica_time(tau, L[perm].tolist()) == pytest.approx(om.replica_time(tau, L.tolist()))
    rep = rng.integers(0, 3, size=len(L)).tolist()
    times, T = om.step_makespan(tau, L.tolist(), rep, 3)
    for r in range(3):
        assert times[r] == pytest.approx(om.replica_time(tau, [x for x, k in zip(L, rep) if k == r]))
    assert T == max(times)


MUTANTS = {
    "strict_active_count": ("if L >= x)", "if L > x)"),
    "last_position_dropped": ("for x in range(1, lmax + 1):\n        total", "for x in range(1, lmax):\n        total"),
    "share_not_divided": ("per = _tau_at(tau, b) / b", "per = _tau_at(tau, b)"),
    "tau_index_shifted": ("return float(tau[b - 1])", "return float(tau[min(b, len(tau) - 1)])"),
}


def test_worked_example():
    pin_worked_example(om)


@pytest.mark.parametrize("seed", range(8))
def test_oracle_equals_both_closed_forms(seed):
    pin_closed_forms(om, seed)


def test_special_cases():
    pin_special_cases(om)


@pytest.mark.parametrize("seed", range(6))
def test_shares_add_up_and_follow_length(seed):
    pin_shares(om, seed)


@pytest.mark.parametrize("seed", range(6))
def test_marginal_costs_in_descending_order_add_up(seed):
    pin_marginal_costs(om, seed)


def test_order_and_step_makespan():
    pin_order_and_step_makespan(om)


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistakes_fail_a_pin(name):
    old, new = MUTANTS[name]
    src = open(om.__file__).read()
    assert old in src, name
    ns = {}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)

    class Mutant:
        replica_time = staticmethod(ns["replica_time"])
        request_shares = staticmethod(ns["request_shares"])
        step_makespan = staticmethod(ns["step_makespan"])

    pins = [pin_worked_example, pin_special_cases, lambda m: pin_closed_forms(m, 0),
            lambda m: pin_shares(m, 0), lambda m: pin_marginal_costs(m, 0), pin_order_and_step_makespan]
    caught = []
    for pin in pins:
        try:
            pin(Mutant)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin)
    assert caught, f"mutant {name} passed every pin"


# ---------------------------------------------------------------------------
# the library against the oracle
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def lib():
    from paper_2608_22788_amd import binding
    return binding


@pytest.mark.parametrize("seed", range(10))
def test_library_matches_oracle(lib, seed):
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(1, 48))
    tau, L = rand_case(rng, n, 400, zeros=seed % 3 == 0)
    tau = np.concatenate([tau, tau[-1] + np.cumsum(rng.uniform(0, 1, size=5))])   # bmax > n
    assert lib.replica_time(tau, L) == pytest.approx(om.replica_time(tau, L.tolist()), rel=1e-12)
    np.testing.assert_allclose(lib.request_shares(tau, L), om.request_shares(tau, L.tolist()), rtol=1e-12,
                               atol=1e-12)
    rep = rng.integers(0, 4, size=n)
    times, T = lib.step_makespan(tau, L, rep, 4)
    otimes, oT = om.step_makespan(tau, L.tolist(), rep.tolist(), 4)
    np.testing.assert_allclose(times, otimes, rtol=1e-12)
    assert T == pytest.approx(oT, rel=1e-12)


def test_library_large_replica(lib):
    """512 requests up to 65536 tokens: against Sec. 2.1's closed forms (the
    position-by-position oracle would take minutes here)."""
    rng = np.random.default_rng(9)
    L = np.minimum(512 + np.floor(1024 * (1 + rng.pareto(1.5, size=512))), 65536).astype(np.int64)
    tau = np.cumsum(rng.uniform(1.0, 3.0, size=512))
    T = lib.replica_time(tau, L)
    assert T == pytest.approx(closed_form_differences(tau, L.tolist()), rel=1e-12)
    assert T == pytest.approx(closed_form_levels(tau, L.tolist()), rel=1e-12)
    assert lib.request_shares(tau, L).sum() == pytest.approx(T, rel=1e-12)


def test_tau_table(lib):
    b = [1, 2, 4, 8, 16]
    t = [5.0, 5.5, 6.0, 7.5, 11.0]
    dense = lib.tau_table(b, t, 40)
    x = np.arange(1, 41)
    inside = x <= 16
    np.testing.assert_allclose(dense[inside], np.interp(x[inside], b, t), rtol=1e-15)
    # past the last point: the last segment extended
    np.testing.assert_allclose(dense[~inside], 7.5 + (11.0 - 7.5) * (x[~inside] - 8) / 8.0, rtol=1e-15)
    # below the first point: its value
    assert np.all(lib.tau_table([4, 8], [2.0, 3.0], 3) == 2.0)
    assert np.all(lib.tau_table([3], [2.0], 5) == 2.0)


@pytest.mark.parametrize("bad", ["n_gt_bmax", "negative_length", "nan_tau", "replica_id", "unsorted_batch",
                                 "negative_tau"])
def test_library_rejects_bad_input(lib, bad):
    tau, L = [1.0, 2.0, 3.0], [4, 2, 1]
    with pytest.raises(lib.TsError):
        if bad == "n_gt_bmax":
            lib.replica_time(tau[:2], L)
        elif bad == "negative_length":
            lib.request_shares(tau, [4, -1, 1])
        elif bad == "nan_tau":
            lib.replica_time([1.0, float("nan"), 3.0], L)
        elif bad == "replica_id":
            lib.step_makespan(tau, L, [0, 2, 1], 2)
        elif bad == "unsorted_batch":
            lib.tau_table([1, 4, 2], [1.0, 2.0, 3.0], 8)
        else:
            lib.tau_table([1, 2], [1.0, -2.0], 8)
