"""The steps around the verify attention on the GPU, through the C ABI,
against the oracle (``oracle/spec_decode.py``): the KV append bit for bit,
and the accepted draft count and next token exactly.  Both sides evaluate the
acceptance rule without rounding (paper Sec. 3.4), so every index must be
equal, including at a 152K-token vocabulary where many inverse-CDF
boundaries lie within float32 or float64 rounding of the target."""
import json
import os

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
    n_ref, t_ref = sd.spec_accept(p, q, d, nd, ua, us)
    n, t = run_accept(p, q, d, nd, ua, us)
    say(f"  {tag}: accepted {list(n)}; tokens equal {int((t == t_ref).sum())}/{len(t)}")
    assert np.array_equal(n, n_ref), f"{tag}: accepted {n} vs {n_ref}"
    assert np.array_equal(t, t_ref), f"{tag}: tokens differ at {np.nonzero(t != t_ref)[0]}"


# 300,007 tokens: 1,172 block sums, 19 per lane of the pick kernel (more than
# the 16 it keeps in registers, so it re-loads them), and a row length that
# is not a multiple of 4 (the scalar tail of the row loads)
@pytest.mark.parametrize("V,G,B", [(151936, 4, 16), (300007, 3, 6), (1001, 3, 9), (50, 15, 4)])
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
    p[5, 0] = 0.0                            # no drafts accepted... and a row without mass
    d[5, 0] = V + 1
    q[5, 0] = 0.0
    n, t = run_accept(p, q, d, nd, ua, us)
    n_ref, t_ref = sd.spec_accept(p, q, d, nd, ua, us)
    assert list(n) == list(n_ref)
    assert n[0] == G and n[1] == 1 and n[2] == 0 and n[3] == 0 and n[4] == 2 and n[5] == 0
    assert t[5] == -1
    assert np.array_equal(t, t_ref)


def test_accept_many_sequences_full_vocabulary():
    """64 sequences at a 152K vocabulary with 0 to 15 drafts each, drafters
    close to and far from the target, so that acceptance stops at every depth
    and the sampling row is the leftover mass or a bonus row."""
    rng = np.random.default_rng(64)
    V, G, B = 151936, 15, 64
    p, logits = probs(rng, B, G + 1, V, 3.0)
    noise = np.where(np.arange(B) % 2 == 0, 0.2, 1.5)[:, None, None]
    q, _ = probs(rng, B, G, V, 0, base=logits[:, :G], noise=noise)
    d = np.zeros((B, G), dtype=np.int32)
    for b in range(B):
        for i in range(G):
            qq = q[b, i].astype(np.float64)
            d[b, i] = rng.choice(V, p=qq / qq.sum())
    nd = (np.arange(B) % (G + 1)).astype(np.int32)
    ua = rng.random((B, G)).astype(np.float32)
    us = rng.random(B).astype(np.float32)
    say(f"accept V={V} G={G} B={B} (every gamma 0..15)")
    check_against_oracle(p, q, d, nd, ua, us, "V151936xB64")


def test_accept_golden_cases():
    """The hand-derived cases of the oracle's pins (each separates the exact
    rule from a rounded evaluation), run as one batch on the GPU."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "spec_accept_exact.json")
    cases = json.load(open(path))["cases"]
    f = lambda a: np.array([float.fromhex(x) for x in a], dtype=np.float64).astype(np.float32)  # noqa: E731
    V = max(len(c["p"][0]) for c in cases)
    G = max(len(c["drafts"]) for c in cases)
    B = len(cases)
    p = np.zeros((B, G + 1, V), np.float32)
    q = np.zeros((B, G, V), np.float32)
    d = np.zeros((B, G), np.int32)
    ua = np.zeros((B, G), np.float32)
    us = np.zeros(B, np.float32)
    nd = np.zeros(B, np.int32)
    want = []
    for b, c in enumerate(cases):
        # pad each case's vocabulary with zero-probability tokens; an
        # out-of-vocabulary draft keeps its meaning by moving past the padding
        for i, r in enumerate(c["p"]):
            p[b, i, :len(r)] = f(r)
        for i, r in enumerate(c["q"]):
            q[b, i, :len(r)] = f(r)
        Vc = len(c["p"][0])
        for i, x in enumerate(c["drafts"]):
            d[b, i] = x if x < Vc else V + x
        ua[b, :len(c["u_accept"])] = f(c["u_accept"])
        us[b] = f([c["u_sample"]])[0]
        nd[b] = len(c["drafts"])
        want.append(c["want"])
    n, t = run_accept(p, q, d, nd, ua, us)
    for b, c in enumerate(cases):
        assert [int(n[b]), int(t[b])] == c["want"], f'{c["name"]}: {[int(n[b]), int(t[b])]} vs {c["want"]}'


def test_accept_one_workspace_for_many_calls():
    """One workspace, never cleared, serves calls of different batch sizes
    and vocabularies in turn: every result equals the oracle's (the
    workspace's contents on entry do not matter)."""
    import torch
    from paper_2608_22788_amd import binding
    big = int(binding.lib.ts_spec_accept_workspace_size(64, 151936))
    ws = torch.full((big,), 0x5A, dtype=torch.uint8, device="cuda")
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dtype=dt, device="cuda")  # noqa: E731
    for n, (V, G, B) in enumerate([(151936, 4, 8), (1001, 3, 9), (151936, 15, 64), (50, 2, 3), (32000, 6, 17)]):
        rng = np.random.default_rng(500 + n)
        p, logits = probs(rng, B, G + 1, V, 2.0)
        q, _ = probs(rng, B, G, V, 0, base=logits[:, :G], noise=0.5)
        d = np.stack([[rng.choice(V, p=q[b, i].astype(np.float64) / q[b, i].astype(np.float64).sum())
                       for i in range(G)] for b in range(B)]).astype(np.int32)
        nd = rng.integers(0, G + 1, size=B).astype(np.int32)
        ua = rng.random((B, G)).astype(np.float32)
        us = rng.random(B).astype(np.float32)
        say(f"accept reuse {n}: V={V} G={G} B={B}")
        na = torch.full((B,), -1, dtype=torch.int32, device="cuda")
        nt = torch.full((B,), -1, dtype=torch.int32, device="cuda")
        binding.spec_accept(t(p, torch.float32), t(q, torch.float32), t(d, torch.int32), t(nd, torch.int32),
                            t(ua, torch.float32), t(us, torch.float32), na, nt, workspace=ws)
        torch.cuda.synchronize()
        n_ref, t_ref = sd.spec_accept(p, q, d, nd, ua, us)
        assert np.array_equal(na.cpu().numpy(), n_ref) and np.array_equal(nt.cpu().numpy(), t_ref), f"call {n}"
