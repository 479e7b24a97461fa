"""Pins of the float64 oracle against facts that do not come from the oracle.

Each ``pin_*`` takes an oracle handle and raises AssertionError when the
oracle disagrees with: a dense brute force on tiny inputs, torch's CPU
attention routine, a closed form, a hand-derived golden case, or an
invariant of the attention definition (page relabelling, head/batch
permutation, key shift, linearity in V, verify row == prefix decode,
split-and-merge == unsplit).  ``run_all`` is also executed against mutated
copies of the oracle source, each of which must fail at least one pin.
"""
from __future__ import annotations

import json
import math
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_22788_amd import synth  # noqa: E402

P = 16


def bf16(x) -> np.ndarray:
    return synth.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def widen(h) -> np.ndarray:
    return synth.bf16_bits_to_f32(h).astype(np.float64)


def small_problem(seed, B, Hq, Hkv, D, lens, qlens, scale=None, spare=0):
    cfg = dict(B=B, Hq=Hq, Hkv=Hkv, D=D, q_len=1, lengths=("uniform", 1, 1),
               scale=1.0 / math.sqrt(D) if scale is None else scale)
    wl = synth.make_workload("pin", seed=seed, cfg=cfg, ctx_lens=lens, q_lens=qlens,
                             spare_pages=spare)
    return dict(q=wl.q_values(), kp=wl.k_pages(), vp=wl.v_pages(), pt=wl.page_table,
                cl=wl.ctx_lens, ql=wl.q_lens, scale=wl.scale)


def call(orc, pr, **over):
    d = dict(pr)
    d.update(over)
    return orc.attention(d["q"], d["kp"], d["vp"], d["pt"], d["cl"], d["ql"], d["scale"])


def dense_reference(pr):
    """Brute force: gather pages into dense K, V; full score matrix with an
    explicit boolean causal mask; KV heads repeated per query-head group."""
    q, kp, vp, pt, cl, ql = (pr[k] for k in ("q", "kp", "vp", "pt", "cl", "ql"))
    B, Qmax, Hq, D = q.shape
    Hkv = kp.shape[1]
    G = Hq // Hkv
    out = np.full(q.shape, np.nan)
    for b in range(B):
        L, Q = int(cl[b]), int(ql[b])
        t = np.arange(L)
        phys = pt[b, t // P]
        K = widen(kp[phys, :, t % P, :])            # [L, Hkv, D]
        V = widen(vp[phys, :, t % P, :])
        Kh = np.repeat(K, G, axis=1)                 # [L, Hq, D]
        Vh = np.repeat(V, G, axis=1)
        qq = widen(q[b, :Q])                         # [Q, Hq, D]
        S = np.einsum("ihd,thd->iht", qq, Kh) * pr["scale"]
        mask = t[None, :] <= (L - Q + np.arange(Q))[:, None]   # [Q, L]
        S = np.where(mask[:, None, :], S, -np.inf)
        S = S - S.max(axis=2, keepdims=True)
        W = np.exp(S)
        W /= W.sum(axis=2, keepdims=True)
        out[b, :Q] = np.einsum("iht,thd->ihd", W, Vh)
    return out


def valid_close(a, b, tol):
    m = ~np.isnan(b)
    assert np.array_equal(m, ~np.isnan(a)), "row coverage differs"
    err = np.abs(a[m] - b[m]).max() if m.any() else 0.0
    assert err <= tol, f"max abs err {err:g} > {tol:g}"


# ---------------------------------------------------------------------------

def pin_bruteforce(orc):
    rng = np.random.default_rng(1)
    for (B, Hq, Hkv, D, Q) in [(1, 1, 1, 16, 1), (3, 4, 2, 16, 2), (2, 8, 2, 64, 4),
                               (3, 4, 1, 32, 16), (2, 8, 8, 16, 3), (1, 4, 4, 128, 5)]:
        lens = [int(x) for x in rng.integers(Q, 70, size=B)]
        lens[0] = max(Q, 32)                     # multiple of the page size
        if B > 1:
            lens[1] = max(Q, 33)                 # one token into a new page
        if B > 2:
            lens[2] = max(Q, 47)                 # one short of a page
        pr = small_problem(int(rng.integers(1 << 30)), B, Hq, Hkv, D, lens, [Q] * B)
        valid_close(call(orc, pr), dense_reference(pr), 1e-12)


def pin_torch_sdpa(orc):
    import torch
    import torch.nn.functional as F
    for (B, Hq, Hkv, D, Q, seed) in [(2, 8, 2, 64, 1, 3), (2, 4, 2, 32, 4, 4), (1, 4, 1, 16, 7, 5)]:
        lens = [Q + 20 + 13 * b for b in range(B)]
        pr = small_problem(seed, B, Hq, Hkv, D, lens, [Q] * B, scale=0.37)
        got = call(orc, pr)
        for b in range(B):
            L = lens[b]
            t = np.arange(L)
            phys = pr["pt"][b, t // P]
            K = torch.from_numpy(widen(pr["kp"][phys, :, t % P, :])).permute(1, 0, 2)
            V = torch.from_numpy(widen(pr["vp"][phys, :, t % P, :])).permute(1, 0, 2)
            K = K.repeat_interleave(Hq // Hkv, dim=0)
            V = V.repeat_interleave(Hq // Hkv, dim=0)
            qq = torch.from_numpy(widen(pr["q"][b, :Q])).permute(1, 0, 2)
            mask = torch.from_numpy(t[None, :] <= (L - Q + np.arange(Q))[:, None])
            ref = F.scaled_dot_product_attention(qq[None], K[None].contiguous(), V[None].contiguous(),
                                                 attn_mask=mask, scale=0.37)[0]
            err = np.abs(ref.permute(1, 0, 2).numpy() - got[b, :Q]).max()
            assert err < 1e-12, f"sdpa mismatch {err:g}"


def pin_one_key(orc):
    pr = small_problem(7, 3, 8, 2, 64, [1, 1, 1], [1, 1, 1])
    got = call(orc, pr)
    G = 4
    for b in range(3):
        for h in range(8):
            v0 = widen(pr["vp"][pr["pt"][b, 0], h // G, 0, :])
            assert np.array_equal(got[b, 0, h], v0), "one key must return its value row"


def pin_zero_scale(orc):
    lens, qs = [40, 17, 16], [4, 1, 16]
    pr = small_problem(8, 3, 4, 2, 16, lens, qs, scale=0.0)
    got = call(orc, pr)
    for b in range(3):
        L, Q = lens[b], qs[b]
        t = np.arange(L)
        V = widen(pr["vp"][pr["pt"][b, t // P], :, t % P, :])   # [L, Hkv, D]
        for i in range(Q):
            n = L - Q + i + 1
            mean = V[:n].mean(axis=0)
            for h in range(4):
                assert np.abs(got[b, i, h] - mean[h // 2]).max() < 1e-12, "zero scale is a mean"


def pin_const_v(orc):
    pr = small_problem(9, 2, 4, 2, 32, [50, 3], [2, 3])
    pr["vp"] = np.full_like(pr["vp"], bf16([1.5])[0])
    got = call(orc, pr)
    m = ~np.isnan(got)
    assert np.abs(got[m] - 1.5).max() < 1e-14


def pin_equal_keys(orc):
    pr = small_problem(10, 2, 4, 2, 16, [37, 20], [3, 1])
    kp = pr["kp"].copy()
    kp[:] = kp[0, 0, 0, :]          # every key row identical
    got = call(orc, pr, kp=kp)
    zero = call(orc, pr, kp=kp, scale=0.0)
    valid_close(got, zero, 1e-12)


def pin_key_shift(orc):
    rng = np.random.default_rng(11)
    pr = small_problem(11, 2, 4, 2, 16, [35, 21], [2, 4])
    kint = rng.integers(-4, 5, size=pr["kp"].shape).astype(np.float32)
    qint = rng.integers(-3, 4, size=pr["q"].shape).astype(np.float32)
    shift = rng.integers(-3, 4, size=(pr["kp"].shape[1], pr["kp"].shape[3])).astype(np.float32)
    a = call(orc, pr, kp=bf16(kint), q=bf16(qint), scale=0.25)
    b = call(orc, pr, kp=bf16(kint + shift[None, :, None, :]), q=bf16(qint), scale=0.25)
    valid_close(a, b, 1e-12)


def pin_linearity_v(orc):
    rng = np.random.default_rng(12)
    pr = small_problem(12, 2, 4, 1, 16, [29, 40], [3, 2])
    v1 = rng.integers(-8, 9, size=pr["vp"].shape).astype(np.float32)
    v2 = rng.integers(-8, 9, size=pr["vp"].shape).astype(np.float32)
    a = call(orc, pr, vp=bf16(v1))
    b = call(orc, pr, vp=bf16(v2))
    c = call(orc, pr, vp=bf16(v1 + v2))
    d = call(orc, pr, vp=bf16(3 * v1))
    valid_close(c, a + b, 1e-12)
    valid_close(d, 3 * a, 1e-12)


def pin_page_relabel(orc):
    pr = small_problem(13, 3, 4, 2, 16, [45, 16, 70], [2, 1, 5], spare=3)
    base = call(orc, pr)
    n = pr["kp"].shape[0]
    perm = np.random.default_rng(13).permutation(n)        # new id of old page p
    kp2 = np.empty_like(pr["kp"])
    vp2 = np.empty_like(pr["vp"])
    kp2[perm] = pr["kp"]
    vp2[perm] = pr["vp"]
    pt2 = perm[pr["pt"]].astype(np.int32)
    got = call(orc, pr, kp=kp2, vp=vp2, pt=pt2)
    assert np.array_equal(np.isnan(got), np.isnan(base))
    m = ~np.isnan(base)
    assert np.array_equal(got[m], base[m]), "relabelled pages must give identical output"


def pin_verify_prefix(orc):
    L, Q = 53, 6
    pr = small_problem(14, 1, 4, 2, 32, [L], [Q])
    full = call(orc, pr)
    for i in range(Q):
        qi = np.zeros_like(pr["q"])
        qi[0, 0] = pr["q"][0, i]
        one = call(orc, pr, q=qi, cl=np.array([L - Q + i + 1], np.int32),
                   ql=np.array([1], np.int32))
        assert np.array_equal(one[0, 0], full[0, i]), f"verify row {i} != prefix decode"


def pin_split_merge(orc):
    lens, qs = [61, 33, 16], [5, 1, 16]
    pr = small_problem(15, 3, 4, 2, 16, lens, qs)
    full = call(orc, pr)
    args = [pr[k] for k in ("q", "kp", "vp", "pt", "cl", "ql")]
    for cuts in ([0, 1, 1, 17, 40, 200], [0, 32, 200], [0, 60, 61, 200], [0, 5, 9, 100]):
        parts, lses = [], []
        for a, b in zip(cuts[:-1], cuts[1:]):
            o, l = orc.partial(*args, pr["scale"], a, b)
            parts.append(o)
            lses.append(l)
        for b in range(3):
            for i in range(qs[b]):
                op = np.stack([p[b, i] for p in parts])      # [S, Hq, D]
                lp = np.stack([l[b, i] for l in lses])      # [S, Hq]
                merged = orc.lse_merge(op, lp)
                assert np.abs(merged - full[b, i]).max() < 1e-13, "split + merge != unsplit"


def pin_weights(orc):
    pr = small_problem(16, 2, 4, 2, 16, [44, 19], [4, 2])
    full = call(orc, pr)
    args = [pr[k] for k in ("q", "kp", "vp", "pt", "cl", "ql")]
    for (b, i, h) in [(0, 0, 0), (0, 3, 3), (1, 1, 2), (1, 0, 1)]:
        w = orc.row_weights(*args, pr["scale"], b, i, h)
        L, Q = int(pr["cl"][b]), int(pr["ql"][b])
        assert abs(w.sum() - 1.0) < 1e-12 and (w >= 0).all()
        assert (w[L - Q + i + 1:] == 0).all() and (w[:L - Q + i + 1] > 0).all()
        t = np.arange(L)
        V = widen(pr["vp"][pr["pt"][b, t // P], h // 2, t % P, :])
        assert np.abs(w @ V - full[b, i, h]).max() < 1e-12


def pin_permutations(orc):
    pr = small_problem(17, 3, 8, 2, 16, [30, 50, 18], [2, 3, 1])
    base = call(orc, pr)
    # batch order
    order = [2, 0, 1]
    got = call(orc, pr, q=pr["q"][order], pt=pr["pt"][order], cl=pr["cl"][order], ql=pr["ql"][order])
    valid_close(got, base[order], 0.0)
    # query heads within a group (KV head 0 owns heads 0..3)
    hp = [2, 0, 3, 1, 4, 5, 6, 7]
    got = call(orc, pr, q=pr["q"][:, :, hp])
    valid_close(got, base[:, :, hp], 0.0)
    # swap KV heads together with their query-head groups
    hp = [4, 5, 6, 7, 0, 1, 2, 3]
    got = call(orc, pr, q=pr["q"][:, :, hp], kp=pr["kp"][:, ::-1].copy(), vp=pr["vp"][:, ::-1].copy())
    valid_close(got, base[:, :, hp], 0.0)


def load_golden():
    with open(os.path.join(HERE, "golden", "closed_forms.json")) as f:
        return json.load(f)["cases"]


def pin_golden(orc):
    env = {"e": math.e}
    for case in load_golden():
        Hq, Hkv, D, L, Q = case["Hq"], case["Hkv"], case["D"], case["L"], case["Q"]
        pages = case["pages"]
        kp = np.zeros((len(pages), Hkv, P, D), np.float32)
        vp = np.zeros_like(kp)
        for t in range(L):
            kp[pages[t // P], :, t % P, :] = np.asarray(case["k"][t], np.float32)
            vp[pages[t // P], :, t % P, :] = np.asarray(case["v"][t], np.float32)
        q = np.asarray(case["q"], np.float32)[None]
        got = orc.attention(bf16(q), bf16(kp), bf16(vp), np.asarray([pages], np.int32),
                            np.asarray([L], np.int32), np.asarray([Q], np.int32), case["scale"])
        want = np.asarray([[[eval(x, {}, env) for x in hrow] for hrow in irow]
                           for irow in case["expect"]], np.float64)
        err = np.abs(got[0] - want).max()
        assert err < 1e-14, f"golden {case['name']}: err {err:g}"


PINS = [pin_bruteforce, pin_torch_sdpa, pin_one_key, pin_zero_scale, pin_const_v,
        pin_equal_keys, pin_key_shift, pin_linearity_v, pin_page_relabel, pin_verify_prefix,
        pin_split_merge, pin_weights, pin_permutations, pin_golden]


def run_all(orc) -> list:
    """Names of the pins that fail (an exception counts as a failure)."""
    failed = []
    for pin in PINS:
        try:
            pin(orc)
        except Exception as e:  # noqa: BLE001
            failed.append(f"{pin.__name__}: {type(e).__name__}: {e}")
    return failed


if __name__ == "__main__":
    # usage: python oracle_pins.py <path to a compiled oracle .so>
    sys.path.insert(0, ROOT)
    import oracle
    bad = run_all(oracle.load(sys.argv[1]))
    print(json.dumps(bad))
    sys.exit(1 if bad else 0)
