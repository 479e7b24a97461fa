"""Pins of the speculative-step oracle (``oracle/spec_decode.py``): the KV
append against the attention definition's page walk, and the acceptance rule
against the property that makes it lossless (paper Sec. 3.4, following
Leviathan et al. 2023): the first emitted token is distributed exactly as the
target's p_0, whatever the drafter proposes; against hand-derived cases in
which a rounded evaluation would give another answer
(``tests/golden/spec_accept_exact.json``); and against float64
``numpy.searchsorted`` where no boundary is near.  Planted mistakes must
fail.  CPU only."""
import json
import os
import numpy as np
import pytest

from oracle import spec_decode as sd


# ---------------------------------------------------------------------------
# KV append
# ---------------------------------------------------------------------------

def small_pool(rng, B=3, Hkv=2, D=8, P=16):
    L = np.array([5, 17, 40])[:B]
    Q = np.array([2, 1, 4])[:B]
    npg = (L + P - 1) // P
    perm = rng.permutation(int(npg.sum()) + 2)
    pt = np.zeros((B, int(npg.max())), dtype=np.int32)
    off = 0
    for b in range(B):
        pt[b, :npg[b]] = perm[off:off + npg[b]]
        off += npg[b]
    NP = len(perm)
    k = rng.standard_normal((NP, Hkv, P, D))
    v = rng.standard_normal((NP, Hkv, P, D))
    kn = rng.standard_normal((B, int(Q.max()), Hkv, D))
    vn = rng.standard_normal((B, int(Q.max()), Hkv, D))
    return k, v, pt, L, Q, kn, vn


def pin_append(sd):
    rng = np.random.default_rng(0)
    k, v, pt, L, Q, kn, vn = small_pool(rng)
    k2, v2 = sd.kv_append(k, v, pt, L, Q, kn, vn)
    changed = np.zeros(k.shape, dtype=bool)
    for b in range(len(L)):
        for i in range(Q[b]):
            t = L[b] - Q[b] + i
            pg, s = pt[b, t // 16], t % 16
            # reading token t back through the page table gives the new rows
            assert np.array_equal(k2[pg, :, s, :], kn[b, i]) and np.array_equal(v2[pg, :, s, :], vn[b, i])
            changed[pg, :, s, :] = True
    # nothing else moved
    assert np.array_equal(k2[~changed], k[~changed]) and np.array_equal(v2[~changed], v[~changed])
    # rows of padded draft positions (i >= Q) are never written
    assert changed.sum() == int(Q.sum()) * k.shape[1] * k.shape[3]


def test_append():
    pin_append(sd)


# ---------------------------------------------------------------------------
# acceptance
# ---------------------------------------------------------------------------

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "spec_accept_exact.json")


def dist(rng, V, conc=1.0):
    x = rng.gamma(conc, size=V)
    return (x / x.sum()).astype(np.float32)


def first_token_law(sd, p0, q0, N=400):
    """Distribution of the first emitted token of a one-draft step, computed
    through spec_accept alone: the draft d is enumerated with weight q0(d);
    the acceptance uniform and the sampling uniform each sweep N midpoints
    (the two draws are independent, so their effects separate)."""
    V = len(p0)
    p = np.stack([p0, p0])[None]          # p_1 (bonus row) unused when gamma = 1 rejects
    q = q0[None, None]
    law = np.zeros(V)
    grid = (np.arange(N) + 0.5) / N
    for d in range(V):
        if q0[d] == 0:
            continue
        acc = sum(int(sd.spec_accept(p, q, [[d]], [1], [[u]], [0.5])[0][0]) for u in grid) / N
        law[d] += q0[d] * acc
        if acc < 1.0:
            # force the rejection branch (a uniform above p/q), sweep the sampler
            ratio = float(p0[d]) / float(q0[d])
            u_rej = min(0.9999999, (1.0 + ratio) / 2)
            nxt = [int(sd.spec_accept(p, q, [[d]], [1], [[u_rej]], [u])[1][0]) for u in grid]
            law += q0[d] * (1.0 - acc) * np.bincount(nxt, minlength=V) / N
    return law


def pin_lossless(sd):
    rng = np.random.default_rng(1)
    for trial in range(3):
        V = 5
        p0, q0 = dist(rng, V), dist(rng, V)
        law = first_token_law(sd, p0, q0)
        np.testing.assert_allclose(law, p0, atol=3.0 / 400)


def test_lossless_first_token():
    pin_lossless(sd)


def golden_cases():
    f = lambda a: np.array([float.fromhex(x) for x in a], dtype=np.float64).astype(np.float32)  # noqa: E731
    for c in json.load(open(GOLDEN))["cases"]:
        p = np.stack([f(r) for r in c["p"]])[None]
        g = len(c["drafts"])
        V = p.shape[-1]
        q = np.stack([f(r) for r in c["q"]])[None] if g else np.zeros((1, 0, V), np.float32)
        d = np.array([c["drafts"]], dtype=np.int32).reshape(1, g)
        ua = f(c["u_accept"]).reshape(1, g)
        us = f([c["u_sample"]])
        yield c, (p, q, d, np.array([g], dtype=np.int32), ua, us)


def pin_golden(sd):
    for c, args in golden_cases():
        n, t = sd.spec_accept(*args)
        assert [int(n[0]), int(t[0])] == c["want"], f'{c["name"]}: {[int(n[0]), int(t[0])]} vs {c["want"]}'


def test_golden_exact_cases():
    pin_golden(sd)


def pin_special_cases(sd):
    rng = np.random.default_rng(2)
    V, g = 50, 3
    p = np.stack([dist(rng, V) for _ in range(g + 1)])[None]
    u = np.array([[0.999, 0.999, 0.999]], dtype=np.float32)
    d = np.array([[3, 7, 11]])
    # drafter equal to the target: everything accepted, next from p_gamma
    n, t = sd.spec_accept(p, p[:, :g], d, [g], u, [0.3])
    assert n[0] == g and t[0] == sd.sample_inverse_cdf(sd.sampling_weights(p[0, g]), 0.3)
    # a draft the target gives zero probability is rejected there
    p2 = p.copy()
    p2[0, 1, 7] = 0.0
    p2[0, 1] /= p2[0, 1].sum()
    q2 = p.copy()[:, :g]
    n, t = sd.spec_accept(p2, q2, d, [g], np.array([[0.5, 0.5, 0.5]], dtype=np.float32), [0.5])
    assert n[0] == 1
    # the leftover mass at a rejection excludes tokens where q >= p
    w = np.maximum(0, p2[0, 1].astype(np.float64) - q2[0, 1].astype(np.float64))
    assert w[t[0]] > 0
    # no drafts: plain sampling from p_0
    n, t = sd.spec_accept(p, p[:, :g], d, [0], u, [0.42])
    c = np.cumsum(p[0, 0].astype(np.float64))
    assert n[0] == 0 and t[0] == int(np.searchsorted(c, np.float32(0.42) * c[-1], side="right"))
    # a draft id outside the vocabulary is rejected
    n, _ = sd.spec_accept(p, p[:, :g], np.array([[3, V + 5, 11]]), [g], u * 0, [0.5])
    assert n[0] == 1


def test_special_cases():
    pin_special_cases(sd)


def units(a):
    return sd.to_units(np.asarray(a, dtype=np.float64))


def pin_inverse_cdf(sd):
    w = sd.to_units(np.array([0.0, 0.0, 0.25, 0.0, 0.5, 0.25, 0.0]))
    assert sd.sample_inverse_cdf(w, 0.0) == 2            # first token with mass
    assert sd.sample_inverse_cdf(w, 0.2499) == 2
    assert sd.sample_inverse_cdf(w, 0.25) == 4           # boundary belongs to the next token
    assert sd.sample_inverse_cdf(w, 0.74) == 4
    assert sd.sample_inverse_cdf(w, 0.75) == 5
    assert sd.sample_inverse_cdf(w, 0.9999) == 5          # last token with mass
    assert sd.sample_inverse_cdf([0, 0], 0.5) == -1


def test_inverse_cdf():
    pin_inverse_cdf(sd)


def pin_float64_library_agreement(sd):
    """Away from any boundary, float64 cumulative sums and numpy's
    searchsorted give the same token as the exact rule."""
    rng = np.random.default_rng(5)
    checked = 0
    for trial in range(40):
        V = int(rng.integers(2, 3000))
        p = dist(rng, V, conc=0.3)
        q = dist(rng, V, conc=0.3) if trial % 2 else None
        u = np.float32(rng.random())
        w = np.asarray(p, dtype=np.float64)
        if q is not None:
            w = np.maximum(0.0, w - np.asarray(q, dtype=np.float64))
        c = np.cumsum(w)
        target = float(u) * c[-1]
        if np.min(np.abs(c - target)) <= 1e-9 * c[-1]:
            continue
        want = int(np.searchsorted(c, target, side="right"))
        got = sd.sample_inverse_cdf(sd.sampling_weights(p, q), float(u))
        assert got == want, (trial, got, want)
        checked += 1
    assert checked >= 30


def test_float64_library_agreement():
    pin_float64_library_agreement(sd)


def test_exact_walk_agrees_with_float64_product():
    """The product of two float32 values is exact in float64, so the
    acceptance decision also equals the float64 comparison on random rows."""
    rng = np.random.default_rng(6)
    for trial in range(200):
        V = 7
        p = dist(rng, V)[None]
        q = dist(rng, V)[None]
        d = [int(rng.integers(0, V))]
        u = np.float32(rng.random())
        want = 1 if float(u) * float(q[0, d[0]]) <= float(p[0, d[0]]) else 0
        assert sd.accept_walk(p, q, d, 1, [u]) == want


def test_returned_token_owns_the_target():
    """The token v satisfies C_{v-1} <= u Z < C_v and carries weight, at a
    152K vocabulary."""
    from fractions import Fraction
    rng = np.random.default_rng(7)
    for trial in range(3):
        V = 151936
        p = dist(rng, V, conc=0.05)
        q = dist(rng, V, conc=0.05)
        u = float(np.float32(rng.random()))
        w = sd.sampling_weights(p, q)
        v = sd.sample_inverse_cdf(w, u)
        Z = sum(w)
        before = sum(w[:v])
        assert w[v] > 0 and before <= Fraction(u) * Z < before + w[v]


MUTANTS = {
    "accept_sign": ("if not u * q <= p:", "if u * q <= p:"),
    "accept_float32_product": ("if not u * q <= p:",
                               "if not np.float32(float(u)) * np.float32(float(q)) <= np.float32(float(p)):"),
    "no_positive_part": ("return [a - b if a > b else 0 for a, b in zip(P, Q)]",
                         "return [abs(a - b) for a, b in zip(P, Q)]"),
    "residual_in_float64": ("    Q = to_units(clamp_prob(q_row))\n    return [a - b if a > b else 0 for a, b in zip(P, Q)]",
                            "    return to_units(np.maximum(0.0, clamp_prob(p_row) - clamp_prob(q_row)))"),
    "cumsum_in_float64": ("    C = list(itertools.accumulate(weights))\n",
                          "    C = [int(x) for x in np.cumsum(np.asarray(weights, dtype=np.float64)).tolist()]\n"),
    "bonus_from_last_draft_row": ("w = sampling_weights(p_target[b, g])", "w = sampling_weights(p_target[b, max(g - 1, 0)])"),
    "append_off_by_one": ("t = L - Q + i\n", "t = L - Q + i + 1\n"),
    "cdf_left_side": ("return bisect.bisect_right(C, int(target))", "return bisect.bisect_left(C, int(target))"),
    "residual_uses_draft_row": ("w = sampling_weights(p_target[b, k], q_draft[b, k])",
                                "w = sampling_weights(p_target[b, k])"),
    "no_probability_clamp": ("return np.clip(np.where(np.isnan(x), 0.0, x), 0.0, 1.0)", "return np.abs(x)"),
    "no_uniform_clamp": ("    return min(u, U_MAX)", "    return u"),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistakes_fail_a_pin(name):
    old, new = MUTANTS[name]
    src = open(sd.__file__).read()
    assert old in src, name
    ns = {"__name__": f"mutant_{name}"}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)

    class Mutant:
        pass

    for fn in ("kv_append", "accept_walk", "sample_inverse_cdf", "spec_accept", "sampling_weights",
               "to_units", "clamp_prob", "clamp_uniform"):
        setattr(Mutant, fn, staticmethod(ns[fn]))

    caught = 0
    for pin in (pin_append, pin_golden, pin_special_cases, pin_inverse_cdf, pin_float64_library_agreement,
                pin_lossless):
        try:
            pin(Mutant)
        except (AssertionError, IndexError, ValueError, TypeError):
            caught += 1
    assert caught, f"mutant {name} passed every pin"
