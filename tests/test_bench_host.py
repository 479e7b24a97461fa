"""Host-side logic of bench.py (no GPU): the single-GPU guard, the sweep
aggregation over seeds, the makespan block built from one-token points only,
the parity figures, and the rule that a committed traffic figure counts only
for the kernel sources it was measured on."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_sweep_summary_aggregates_over_seeds(bench):
    pts = [dict(batch=b, q_len=4 if b <= 8 else 1, seed=s, kv_gbps=100.0 * b + s,
                hbm_frac=(100.0 * b + s) / 8000, tokens_per_s=10.0 * s, tau_us=1.0 + s, t_median_us=2.0 + s)
           for b in (8, 16) for s in range(5)]
    out = bench.sweep_summary(pts)
    assert [r["batch"] for r in out] == [8, 16]
    r = out[0]
    assert r["seeds"] == 5 and r["q_len"] == 4
    assert r["kv_gbps"] == 802.0 and r["kv_gbps_min"] == 800.0 and r["kv_gbps_max"] == 804.0
    assert r["tau_us"] == 3.0 and r["tau_us_min"] == 1.0 and r["tau_us_max"] == 5.0
    assert r["call_us"] == 4.0 and r["call_us_min"] == 2.0 and r["call_us_max"] == 6.0
    assert r["regime"].startswith("verify") and out[1]["regime"].startswith("decode")


def test_traffic_counts_only_for_matching_sources(bench, tmp_path, monkeypatch):
    h = bench.kernel_hash("dflash")
    f = tmp_path / "t.md"
    f.write_text(f"traffic dflash kernel_hash={h} bytes_per_launch=123\n"
                 f"traffic mtp kernel_hash=0000000000000000 bytes_per_launch=456\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.measured_traffic("dflash") == 123
    assert bench.measured_traffic("mtp") is None        # stale: sources changed since
    assert bench.measured_traffic("bulk") is None       # never measured
    assert len(h) == 16 and h != bench.kernel_hash("bulk")


def test_makespan_model_block(bench):
    """The bench's model block: the replica time of the bulk lengths under a
    tau curve equals the position-by-position oracle on the same table."""
    import numpy as np
    from oracle import makespan as om
    from paper_2608_22788_amd import binding, synth
    wl = synth.make_workload("bulk", seed=0)
    pts = [(1, 4.6), (2, 5.0), (4, 5.6), (8, 7.1), (16, 53.0), (32, 88.0), (64, 153.0), (128, 288.0),
           (256, 554.0), (512, 1066.0)]
    sweep = [dict(batch=b, q_len=1, tau_us=t) for b, t in pts]
    # verify-regime points at the same batch sizes must not enter the table
    sweep += [dict(batch=b, q_len=4, tau_us=1e6) for b, _ in pts[:4]]
    out = bench.makespan_model(sweep, wl)
    tau = binding.tau_table([b for b, _ in pts], [t for _, t in pts], 512)
    L = wl.ctx_lens.astype(np.int64)
    s = sorted(L.tolist(), reverse=True) + [0]
    closed = sum(tau[j] * (s[j] - s[j + 1]) for j in range(len(L)))
    assert out["bulk_replica_attention_s"] == round(closed / 1e6, 6)
    assert out["bulk_requests"] == 256 and 0.05 < out["longest_5pct_share"] < 1.0
    # the shares of a few requests, position by position
    small = L[:12].tolist()
    np.testing.assert_allclose(binding.request_shares(tau, small), om.request_shares(tau.tolist(), small),
                               rtol=1e-12)


def test_sweep_summary_reports_the_gather_floor(bench):
    pts = [dict(batch=1, q_len=4, seed=s, kv_gbps=500.0, hbm_frac=0.0625, tokens_per_s=1.0, tau_us=20.0,
                kv_bytes=10_000_000, t_median_us=20.0, gather_median_us=10.0 + s) for s in range(2)]
    r = bench.sweep_summary(pts)[0]
    assert r["gather_gbps"] == round((1e7 / 10e-6 + 1e7 / 11e-6) / 2 / 1e9, 1)
    assert r["call_frac_of_gather"] == round((10.0 / 20.0 + 11.0 / 20.0) / 2, 4)


def test_tp2_share_halves_the_heads_only(bench):
    from paper_2608_22788_amd import synth
    for name in ("bulk", "dflash"):
        cfg, base = bench.tp2_share(name), synth.CONFIGS[name]
        assert (cfg["Hq"], cfg["Hkv"]) == (base["Hq"] // 2, base["Hkv"] // 2) == (16, 4)
        assert {k: v for k, v in cfg.items() if k not in ("Hq", "Hkv")} == \
               {k: v for k, v in base.items() if k not in ("Hq", "Hkv")}


def test_ceiling_summary(bench):
    r = dict(gather_gbps=6700.0, kernel_frac_of_gather=0.96, stream_read=dict(gbps=6980.0, bytes=123))
    out = bench.ceiling_summary(r)
    assert out["page_gather_gbps"] == 6700.0 and out["kernel_frac_of_page_gather"] == 0.96
    assert out["stream_read_gbps"] == 6980.0 and out["page_gather_frac_of_peak"] == round(6700 / 8000, 4)
    assert bench.ceiling_summary(dict(ceiling_error="x")) == {"error": "x"}
    assert bench.ceiling_summary({}) is None


def test_parity_errors_over_valid_rows(bench):
    import numpy as np
    ref = np.full((2, 2, 1, 4), np.nan)
    ref[0, 0] = [1.0, -2.0, 0.5, 0.0]
    ref[1] = 0.25
    got = np.zeros_like(ref)
    got[0, 0] = [1.0, -2.0, 0.5, 0.1]
    got[1] = 0.25
    got[0, 1] = 123.0                       # a padded row: not compared
    p = bench.parity_errors(got, ref)
    assert p["elements"] == 12 and p["finite"]
    assert abs(p["max_abs"] - 0.1) < 1e-15 and abs(p["mean_abs"] - 0.1 / 12) < 1e-15
    norm = np.sqrt(1 + 4 + 0.25 + 8 * 0.0625)
    assert abs(p["rel_l2"] - 0.1 / norm) < 1e-15


def test_plan_summary_names_the_launch():
    import bench
    got = bench.plan_summary(dict(variant=2, num_workers=512, combine=2, grid=1024, threads=256,
                                  merge_blocks=0, lds_bytes=66560, workspace_bytes=1 << 20))
    assert got == dict(kernel="team of four wavefronts", workers=512, combine="merge wavefronts in the launch",
                       grid=1024)
    assert bench.plan_summary(dict(variant=1, num_workers=1024, combine=1, grid=1024))["combine"] == \
        "last arriver in the launch"
