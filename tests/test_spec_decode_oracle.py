"""Pins of the speculative-step oracle (``oracle/spec_decode.py``): the KV
append against the attention definition's page walk, and the acceptance rule
against the property that makes it lossless (paper Sec. 3.4, following
Leviathan et al. 2023): the first emitted token is distributed exactly as the
target's p_0, whatever the drafter proposes.  Planted mistakes must fail.
CPU only."""
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


def pin_special_cases(sd):
    rng = np.random.default_rng(2)
    V, g = 50, 3
    p = np.stack([dist(rng, V) for _ in range(g + 1)])[None]
    u = np.array([[0.999, 0.999, 0.999]], dtype=np.float32)
    d = np.array([[3, 7, 11]])
    # drafter equal to the target: everything accepted, next from p_gamma
    n, t, _ = sd.spec_accept(p, p[:, :g], d, [g], u, [0.3])
    assert n[0] == g and t[0] == sd.sample_inverse_cdf(p[0, g], 0.3)[0]
    # a draft the target gives zero probability is rejected there
    p2 = p.copy()
    p2[0, 1, 7] = 0.0
    p2[0, 1] /= p2[0, 1].sum()
    q2 = p.copy()[:, :g]
    n, t, _ = sd.spec_accept(p2, q2, d, [g], np.array([[0.5, 0.5, 0.5]], dtype=np.float32), [0.5])
    assert n[0] == 1
    # the leftover mass at a rejection excludes tokens where q >= p
    w = np.maximum(0, p2[0, 1].astype(np.float64) - q2[0, 1].astype(np.float64))
    assert w[t[0]] > 0
    # no drafts: plain sampling from p_0
    n, t, _ = sd.spec_accept(p, p[:, :g], d, [0], u, [0.42])
    c = np.cumsum(p[0, 0].astype(np.float64))
    assert n[0] == 0 and t[0] == int(np.searchsorted(c, 0.42 * c[-1], side="right"))
    # a draft id outside the vocabulary is rejected
    n, _, _ = sd.spec_accept(p, p[:, :g], np.array([[3, V + 5, 11]]), [g], u * 0, [0.5])
    assert n[0] == 1


def test_special_cases():
    pin_special_cases(sd)


def pin_inverse_cdf(sd):
    w = np.array([0.0, 0.0, 0.25, 0.0, 0.5, 0.25, 0.0])
    assert sd.sample_inverse_cdf(w, 0.0)[0] == 2            # first token with mass
    assert sd.sample_inverse_cdf(w, 0.2499)[0] == 2
    assert sd.sample_inverse_cdf(w, 0.25)[0] == 4           # boundary belongs to the next token
    assert sd.sample_inverse_cdf(w, 0.74)[0] == 4
    assert sd.sample_inverse_cdf(w, 0.9999)[0] == 5          # last token with mass
    assert sd.sample_inverse_cdf(w, 0.25)[1] and not sd.sample_inverse_cdf(w, 0.4)[1]


def test_inverse_cdf():
    pin_inverse_cdf(sd)


MUTANTS = {
    "accept_sign": ("if not lhs <= np.float32(p_target[i, d]):", "if lhs <= np.float32(p_target[i, d]):"),
    "no_positive_part": ("w = np.maximum(0.0, p_target[b, k].astype(np.float64) - q_draft[b, k].astype(np.float64))",
                         "w = np.abs(p_target[b, k].astype(np.float64) - q_draft[b, k].astype(np.float64))"),
    "bonus_from_last_draft_row": ("w = p_target[b, g].astype(np.float64)", "w = p_target[b, max(g - 1, 0)].astype(np.float64)"),
    "append_off_by_one": ("t = L - Q + i\n", "t = L - Q + i + 1\n"),
    "cdf_left_side": ('v = int(np.searchsorted(c, target, side="right"))', 'v = int(np.searchsorted(c, target, side="left"))'),
    "residual_uses_draft_row": ("w = np.maximum(0.0, p_target[b, k].astype(np.float64) - q_draft[b, k].astype(np.float64))",
                                "w = np.maximum(0.0, p_target[b, k].astype(np.float64) - 0.0 * q_draft[b, k].astype(np.float64))"),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistakes_fail_a_pin(name):
    old, new = MUTANTS[name]
    src = open(sd.__file__).read()
    assert old in src, name
    ns = {"__name__": f"mutant_{name}"}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)

    class Mutant:
        kv_append = staticmethod(ns["kv_append"])
        accept_walk = staticmethod(ns["accept_walk"])
        sample_inverse_cdf = staticmethod(ns["sample_inverse_cdf"])
        spec_accept = staticmethod(ns["spec_accept"])

    caught = 0
    for pin in (pin_append, pin_special_cases, pin_inverse_cdf, pin_lossless):
        try:
            pin(Mutant)
        except (AssertionError, IndexError, ValueError):
            caught += 1
    assert caught, f"mutant {name} passed every pin"
