"""The completion-time model fed with a curve measured on this GPU: the
concurrency sweep's per-token attention time tau(b) becomes a dense table, and
the library's replica time and request shares for the bulk workload's lengths
match the position-by-position oracle (paper Sec. 2.1, App. D)."""
import numpy as np
import pytest

from oracle import makespan as om
from paper_2608_22788_amd import synth

from gpu_util import say

pytestmark = pytest.mark.gpu


def test_measured_curve_drives_the_model():
    from paper_2608_22788_amd import binding
    batches = (1, 2, 4, 8, 16, 32, 64, 128, 256)
    pts = binding.concurrency_sweep(batches=batches, seeds=1, warmup=3, iters=10)
    b = [p["batch"] for p in pts]
    tau_pts = [p["tau_us"] for p in pts]
    say("tau(b) us:", dict(zip(b, np.round(tau_pts, 2))))
    assert all(t > 0 for t in tau_pts)
    tau = binding.tau_table(b, tau_pts, 256)
    assert tau[0] == pytest.approx(tau_pts[0]) and tau[255] == pytest.approx(tau_pts[-1])
    L = synth.make_workload("bulk", seed=0).ctx_lens.astype(np.int64)
    T = binding.replica_time(tau, L)
    T_ref = om.replica_time(tau.tolist(), L.tolist())
    say(f"bulk lengths on one replica: T = {T / 1e6:.4f} s (attention share)")
    assert T == pytest.approx(T_ref, rel=1e-12)
    sh = binding.request_shares(tau, L)
    np.testing.assert_allclose(sh, om.request_shares(tau.tolist(), L.tolist()), rtol=1e-10)
    assert sh.sum() == pytest.approx(T, rel=1e-12)
