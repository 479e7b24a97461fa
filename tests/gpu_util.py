"""Helpers for the GPU parity tests: tolerance checks against the oracle and
workload runners.  The oracle always sees inputs from the host generator;
the GPU sees either copies of them or the library's device fill of the same
definition."""
from __future__ import annotations

import sys

import numpy as np

from paper_2608_22788_amd import synth

# Parity bar on bf16 outputs with N(0,1) inputs: max-abs and mean-abs error
# over valid output elements, plus relative L2 (outputs shrink like
# sqrt(e / L) at long context, where the absolute bars alone get weak).
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
REL_L2 = 1e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_out(orc, wl: synth.Workload, nthreads: int = 0) -> np.ndarray:
    return orc.attention(wl.q_values(), wl.k_pages(), wl.v_pages(), wl.page_table, wl.ctx_lens,
                         wl.q_lens, wl.scale, nthreads=nthreads)


def errors(got: np.ndarray, ref: np.ndarray):
    m = ~np.isnan(ref)
    d = got[m] - ref[m]
    if d.size == 0:
        return 0.0, 0.0, 0.0
    rel = float(np.linalg.norm(d) / max(np.linalg.norm(ref[m]), 1e-30))
    return float(np.abs(d).max()), float(np.abs(d).mean()), rel


def assert_parity(got: np.ndarray, ref: np.ndarray, tag: str):
    assert np.isfinite(got[~np.isnan(ref)]).all(), f"{tag}: non-finite output"
    mx, mean, rel = errors(got, ref)
    say(f"  {tag}: max_abs={mx:.3g} mean_abs={mean:.3g} rel_l2={rel:.3g}")
    assert mx <= MAX_ABS and mean <= MEAN_ABS and rel <= REL_L2, \
        f"{tag}: max_abs={mx:g} mean_abs={mean:g} rel_l2={rel:g}"


def canary_ok(t, wl: synth.Workload) -> None:
    """Guard bands and rows i >= q_lens[b] still hold the canary."""
    from paper_2608_22788_amd import device
    full = t["out_full"].cpu().numpy().view(np.uint16)
    g = device.GUARD
    assert (full[:g] == device.CANARY).all() and (full[-g:] == device.CANARY).all(), "guard band written"
    out = full[g:-g].reshape(wl.B, wl.Qmax, wl.Hq, wl.D)
    for b in range(wl.B):
        q = int(wl.q_lens[b])
        assert (out[b, q:] == device.CANARY).all(), f"padded rows of sequence {b} written"


def sample_seqs(wl: synth.Workload, k: int, seed: int = 0):
    """The longest and shortest sequences plus k - 2 random others."""
    rng = np.random.default_rng(seed)
    picks = {int(np.argmax(wl.ctx_lens)), int(np.argmin(wl.ctx_lens))}
    others = [b for b in range(wl.B) if b not in picks]
    rng.shuffle(others)
    picks.update(others[:max(0, k - len(picks))])
    return sorted(picks)
