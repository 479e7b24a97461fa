"""The C ABI without a GPU: the library loads, exports every function that
include/ts_attn.h declares, rejects bad shapes and arguments before any HIP
call, and its host-side generators agree with the test generator."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_22788_amd import binding as b
from paper_2608_22788_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "ts_attn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ts_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(b.lib, n), f"{n} not exported"
    assert sorted(b.EXPORTS) == names


def test_version_and_status_strings():
    assert b.lib.ts_version() == b.ABI_VERSION == 4
    for st in (0, -1, -2, -3, -4, -5, -6):
        assert b.lib.ts_status_string(st)
    assert b.lib.ts_status_string(-99) == b"unknown status"


def base_shape(**kw):
    d = dict(num_seqs=4, num_q_heads=8, num_kv_heads=2, head_dim=64, max_q_len=1,
             max_pages_per_seq=16, max_ctx_len=256, num_pages=64)
    d.update(kw)
    return b.make_shape(**d)


@pytest.mark.parametrize("kw", [
    dict(num_seqs=0), dict(num_seqs=5000), dict(num_q_heads=6, num_kv_heads=4),
    dict(num_kv_heads=0), dict(head_dim=96), dict(head_dim=256), dict(max_q_len=0),
    dict(max_q_len=17), dict(num_q_heads=32, num_kv_heads=1, max_q_len=4),
    dict(max_pages_per_seq=0), dict(max_ctx_len=257), dict(max_ctx_len=0), dict(num_pages=0),
    dict(num_workers=-1), dict(num_seqs=4096, num_q_heads=128, num_kv_heads=128)])
def test_bad_shapes_rejected(kw):
    s = base_shape(**kw)
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) == 0
    assert b.lib.ts_last_error()
    st = b.lib.ts_decode_attn(ctypes.byref(s), 16, 16, 16, 16, 16, 16, 16, ctypes.c_float(1.0),
                              256, 1 << 30, None)
    assert st == -2
    assert b.lib.ts_decode_attn_plan(ctypes.byref(s), ctypes.byref(b.AttnPlan())) == -2


def test_plan_needs_an_output():
    assert b.lib.ts_decode_attn_plan(ctypes.byref(base_shape()), None) == -1
    assert b"plan" in b.lib.ts_last_error()


def test_variant_checks():
    s = base_shape(max_q_len=4)
    s.variant = 3
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) == 0
    s.variant = b.VARIANT_TEAM          # team kernel needs head_dim 128
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) == 0
    s.head_dim = 128
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) > 0
    s.variant = b.VARIANT_WAVE
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) > 0
    s.variant = b.VARIANT_VALU          # the VALU kernel is one-token only
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) == 0
    s.max_q_len = 1
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) > 0
    s.variant = 4
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) == 0


def test_page_size_must_be_16():
    s = base_shape()
    s.page_size = 32
    assert b.lib.ts_decode_attn_workspace_size(ctypes.byref(s)) == 0


def test_null_and_workspace_errors_before_device_use():
    s = base_shape()
    need = b.workspace_size(s)
    assert need > 0 and need % 256 == 0
    f = ctypes.c_float(0.125)
    assert b.lib.ts_decode_attn(None, 16, 16, 16, 16, 16, 16, 16, f, 256, need, None) == -1
    assert b.lib.ts_decode_attn(ctypes.byref(s), None, 16, 16, 16, 16, 16, 16, f, 256, need, None) == -1
    assert b.lib.ts_decode_attn(ctypes.byref(s), 16, 16, 16, 16, 16, 16, 16, f, None, need, None) == -1
    assert b.lib.ts_decode_attn(ctypes.byref(s), 16, 16, 16, 16, 16, 16, 16, f, 256, need - 1, None) == -3
    assert b.lib.ts_decode_attn(ctypes.byref(s), 16, 16, 16, 16, 16, 16, 16, f, 128, need, None) == -6
    assert b.lib.ts_decode_attn(ctypes.byref(s), 8, 16, 16, 16, 16, 16, 16, f, 256, need, None) == -6
    nan = ctypes.c_float(float("nan"))
    assert b.lib.ts_decode_attn(ctypes.byref(s), 16, 16, 16, 16, 16, 16, 16, nan, 256, need, None) == -6


def test_workspace_grows_with_workers_and_rows():
    w1 = b.workspace_size(base_shape(num_workers=10))
    w2 = b.workspace_size(base_shape(num_workers=20))
    assert w2 > w1
    big = b.make_shape(4, 32, 8, 128, 16, 7000, 98304, 30000)
    small = b.make_shape(4, 32, 8, 128, 4, 7000, 98304, 30000)
    assert b.workspace_size(big) > b.workspace_size(small)


def test_sweep_config_rejected_without_running():
    cfg = b.SweepConfig()
    cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim = 32, 8, 128
    cfg.num_batches, cfg.num_seeds, cfg.iters = 0, 1, 1
    pts = (b.SweepPoint * 4)()
    n = ctypes.c_int32()
    assert b.lib.ts_concurrency_sweep(ctypes.byref(cfg), pts, 4, ctypes.byref(n)) == -6
    cfg.num_batches = 2
    cfg.batches[0], cfg.batches[1] = 1, 2
    cfg.verify_q_len = 4
    assert b.lib.ts_concurrency_sweep(ctypes.byref(cfg), pts, 1, ctypes.byref(n)) == -6


@pytest.mark.parametrize("seed", [0, 1, 4])
def test_library_sweep_lengths_match_generator(seed):
    for B in (1, 2, 8, 64, 512):
        assert np.array_equal(b.sweep_lengths(B, seed), synth.lengths_sweep(seed, B).astype(np.int32))


def test_library_page_table_matches_generator():
    for seed, name in [(0, "sweep_b64"), (2, "sweep_b8"), (0, "tiny")]:
        wl = synth.make_workload(name, seed=seed)
        pt = b.page_table(wl.ctx_lens, wl.max_pages, seed)
        assert np.array_equal(pt, wl.page_table)


def test_host_generator_c_matches_numpy():
    if synth._host_lib() is None:
        synth.build_host()
    for seed, stream, start, n in [(0, 5, 0, 1 << 20), (7, 6, 123456789, 100003), (3, 4, 2 ** 40, 5000)]:
        a = synth.normal_bf16_range(seed, stream, start, n)
        c = synth.normal_bf16_range_numpy(seed, stream, start, n)
        assert np.array_equal(a, c)
