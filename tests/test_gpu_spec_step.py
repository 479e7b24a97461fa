"""The steps around the verify attention on the GPU, through the C ABI,
against the oracle (``oracle/spec_decode.py``): the KV append bit for bit,
and the acceptance decision and next token exactly.  With a 152K-token
vocabulary many inverse-CDF boundaries lie within fp32 rounding of the
target; a token that differs from the float64 oracle's must then own the
target within that rounding (4e-6 of the total mass) and carry mass."""
import numpy as np
import pytest

from oracle import spec_decode as sd
from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("D,Hkv", [(128, 8), (64, 2)])
def test_kv_append_matches_oracle(D, Hkv):
    import torch
    from paper_2608_22788_amd import binding
    rng = np.random.default_rng(D + Hkv)
    ctx = [37, 16, 1, 300, 129, 64]
    ql = [4, 1, 1, 16, 0, 3]
    Qmax = 16
    P = 16
    npg = [(L + P - 1) // P for L in ctx]
    NP = sum(npg) + 3
    perm = rng.permutation(NP)
    pt = np.zeros((len(ctx), max(npg)), dtype=np.int32)
    off = 0
    for b, n in enumerate(npg):
        pt[b, :n] = perm[off:off + n]
        off += n
    k = rng.integers(0, 1 << 16, size=(NP, Hkv, P, D), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=(NP, Hkv, P, D), dtype=np.uint16)
    kn = rng.integers(0, 1 << 16, size=(len(ctx), Qmax, Hkv, D), dtype=np.uint16)
    vn = rng.integers(0, 1 << 16, size=(len(ctx), Qmax, Hkv, D), dtype=np.uint16)
    k_ref, v_ref = sd.kv_append(k, v, pt, ctx, ql, kn, vn)
    dev = lambda a: torch.from_numpy(a.view(np.int16)).cuda()  # noqa: E731
    tk, tv = dev(k), dev(v)
    i32 = lambda a: torch.tensor(a, dtype=torch.int32, device="cuda")  # noqa: E731
    say(f"kv append D={D} Hkv={Hkv} lens={ctx} q={ql}")
    binding.kv_append(dev(kn), dev(vn), tk, tv, torch.from_numpy(pt).cuda(), i32(ctx), i32(ql))
    torch.cuda.synchronize()
    assert np.array_equal(tk.cpu().numpy().view(np.uint16), k_ref)
    assert np.array_equal(tv.cpu().numpy().view(np.uint16), v_ref)


def probs(rng, B, R, V, scale, base=None, noise=0.0):
    logits = rng.standard_normal((B, R, V)) * scale if base is None else base + noise * rng.standard_normal(base.shape)
    e = np.exp(logits - logits.max(-1, keepdims=True))
    return (e / e.sum(-1, keepdims=True)).astype(np.float32), logits


def run_accept(p, q, d, nd, ua, us):
    import torch
    from paper_2608_22788_amd import binding
    B = p.shape[0]
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dtype=dt, device="cuda")  # noqa: E731
    na = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    nt = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    binding.spec_accept(t(p, torch.float32), t(q, torch.float32) if q is not None else None,
                        t(d, torch.int32) if d is not None else None, t(nd, torch.int32),
                        t(ua, torch.float32) if ua is not None else None, t(us, torch.float32), na, nt)
    torch.cuda.synchronize()
    return na.cpu().numpy(), nt.cpu().numpy()


def check_against_oracle(p, q, d, nd, ua, us, tag):
    n_ref, t_ref, near = sd.spec_accept(p, q, d, nd, ua, us, tol=5e-5)
    n, t = run_accept(p, q, d, nd, ua, us)
    assert np.array_equal(n, n_ref), f"{tag}: accepted {n} vs {n_ref}"
    for b in range(len(nd)):
        if t[b] == t_ref[b]:
            continue
        assert near[b], f"{tag} seq {b}: token {t[b]} vs {t_ref[b]} away from any boundary"
        k = int(n_ref[b])
        w = (np.maximum(0.0, p[b, k].astype(np.float64) - q[b, k].astype(np.float64))
             if k < nd[b] else p[b, nd[b]].astype(np.float64))
        # fp32 block sums, runs and scans keep the cumulative mass within a
        # few 1e-6 of the total: the GPU's token must own the target up to that
        c = np.cumsum(w)
        target = float(us[b]) * c[-1]
        eps = 4e-6 * c[-1]
        lo = c[t[b] - 1] if t[b] > 0 else 0.0
        assert w[t[b]] > 0 and lo - eps <= target < c[t[b]] + eps, \
            f"{tag} seq {b}: token {t[b]} owns [{lo}, {c[t[b]]}), target {target}"
    say(f"  {tag}: accepted {list(n)}; tokens equal {int((t == t_ref).sum())}/{len(t)}")


@pytest.mark.parametrize("V,G,B", [(151936, 4, 16), (1001, 3, 9), (50, 15, 4)])
def test_accept_matches_oracle(V, G, B):
    rng = np.random.default_rng(V + G)
    p, logits = probs(rng, B, G + 1, V, 2.0)
    q, _ = probs(rng, B, G, V, 0, base=logits[:, :G], noise=0.7)
    d = np.zeros((B, G), dtype=np.int32)
    for b in range(B):
        for i in range(G):
            qq = q[b, i].astype(np.float64)
            d[b, i] = rng.choice(V, p=qq / qq.sum())
    nd = rng.integers(0, G + 1, size=B).astype(np.int32)
    ua = rng.random((B, G)).astype(np.float32)
    us = rng.random(B).astype(np.float32)
    say(f"accept V={V} G={G} B={B} drafts={list(nd)}")
    check_against_oracle(p, q, d, nd, ua, us, f"V{V}")


def test_accept_special_cases():
    rng = np.random.default_rng(3)
    V, G, B = 4096, 3, 6
    p, logits = probs(rng, B, G + 1, V, 1.0)
    q = p[:, :G].copy()
    d = rng.integers(0, V, size=(B, G)).astype(np.int32)
    nd = np.full(B, G, dtype=np.int32)
    ua = np.full((B, G), 0.999, dtype=np.float32)
    us = rng.random(B).astype(np.float32)
    d[1, 1] = V + 7                         # out of the vocabulary: rejected at 1
    p[2, 0, d[2, 0]] = 0.0                   # target gives the first draft no mass
    p[2, 0] /= p[2, 0].sum()
    nd[3] = 0                                # no drafts: plain sampling
    q[4, 2] = p[4, 2]                        # leftover mass exactly zero at a rejection
    d[4, 2] = int(np.argmax(p[4, 2]))
    ua[4, 2] = 1.0 - 1e-7
    p4 = p[4, 2].copy()
    q[4, 2, d[4, 2]] = p4[d[4, 2]] * 2       # rejects; leftover max(0, p - q) is all zero there
    n, t = run_accept(p, q, d, nd, ua, us)
    n_ref, t_ref, _ = sd.spec_accept(p, q, d, nd, ua, us)
    assert list(n) == list(n_ref)
    assert n[0] == G and n[1] == 1 and n[2] == 0 and n[3] == 0 and n[4] == 2
    assert np.array_equal(t, t_ref)
