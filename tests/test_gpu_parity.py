"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Every test compares every output element of the call it makes: the small
and random cases, and the full-size workloads (bulk, MTP verify, block-draft
verify and every seed-0 point of the concurrency sweep) in the launch
configuration the benchmark times.  The oracle sees the host generator's
values; the GPU sees the library's device fill of the same definition,
checked bit for bit against the host side.  Properties that hold at any
size are checked too (finite outputs, untouched canaries).  A few side
cases (group sizes, TP2 shares, the ragged mixed batch) compare sampled
sequences."""
import numpy as np
import pytest

from paper_2608_22788_amd import synth

from gpu_util import assert_parity, canary_ok, oracle_out, sample_seqs, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_22788_amd import binding, device
    return binding, device


def small_cfg(Hq, Hkv, D):
    return dict(B=1, Hq=Hq, Hkv=Hkv, D=D, q_len=1, lengths=("uniform", 1, 1), scale=1.0 / np.sqrt(D))


def test_device_fill_matches_host_generator(dev):
    import torch
    binding, _ = dev
    for seed, stream, off, n in [(0, synth.S_K, 0, 1 << 22), (5, synth.S_V, 987654321, 1 << 20 | 7),
                                 (2, synth.S_Q, 3, 1001)]:
        say(f"fill seed={seed} stream={stream} off={off} n={n}")
        t = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        binding.synth_fill(t, seed, stream, off)
        got = t.view(torch.int16).cpu().numpy().view(np.uint16)
        want = synth.normal_bf16_range(seed, stream, off, n)
        assert np.array_equal(got, want)


def variants_for(wl):
    """Kernel variants to check for a workload: the automatic choice, the
    single-wavefront matrix-core kernel, at head_dim 128 the team kernel, and
    for one-token decode with a group size of 1, 2, 4 or 8 the VALU kernel."""
    v = [0, 1] + ([2] if wl.D == 128 else [])
    if wl.Qmax == 1 and wl.Hq // wl.Hkv in (1, 2, 4, 8):
        v.append(3)
    return tuple(v)


def run_case(dev, orc, wl, workers=(0,), values="host"):
    _, device = dev
    ref = oracle_out(orc, wl)
    t = device.upload(wl, values=values)
    for var in variants_for(wl):
        for w in workers:
            say(f"case {wl.name} B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Qmax={wl.Qmax} "
                f"lens={list(wl.ctx_lens)[:8]} q={list(wl.q_lens)[:8]} workers={w} variant={var}")
            t["out_full"].fill_(device.CANARY)
            device.run(wl, t, num_workers=w, variant=var)
            got = device.out_as_f64(t)
            assert_parity(got, ref, f"{wl.name}/w{w}/v{var}")
            canary_ok(t, wl)
    return t, ref


def test_tiny_config(dev, orc):
    wl = synth.make_workload("tiny", seed=0, poison=True, spare_pages=3)
    run_case(dev, orc, wl, workers=(0, 1, 2, 7, 64))


GRID = [
    # (Hq, Hkv, D, q_lens, ctx_lens)
    (8, 2, 64, [1, 1, 1], [16, 17, 300]),
    (32, 8, 128, [1] * 5, [1, 15, 16, 33, 1000]),
    (8, 8, 128, [1, 1], [47, 2048]),
    (16, 2, 128, [1, 1, 1], [64, 65, 511]),
    (4, 4, 64, [2, 2], [2, 80]),
    (32, 8, 128, [4] * 3, [4, 31, 777]),
    (32, 8, 128, [3, 3], [19, 260]),
    (32, 8, 128, [5, 6], [100, 6]),
    (32, 8, 128, [16, 16], [16, 1500]),
    (32, 8, 64, [16, 7], [40, 333]),
    (16, 1, 128, [4, 4], [48, 129]),
    (32, 8, 128, [4, 1, 0, 4], [64, 50, 30, 97]),     # ragged, one sequence skipped
    (8, 2, 128, [1, 0, 1], [20, 5, 700]),
]


@pytest.mark.parametrize("case", range(len(GRID)))
def test_small_grid(dev, orc, case):
    Hq, Hkv, D, ql, cl = GRID[case]
    wl = synth.make_workload(f"grid{case}", seed=100 + case, cfg=small_cfg(Hq, Hkv, D), ctx_lens=cl,
                             q_lens=ql, poison=True, spare_pages=2)
    run_case(dev, orc, wl, workers=(0, 1, 3, 40))


def random_shape(seed):
    """A seeded shape: KV heads, group size, head_dim, draft depth, and
    ragged lengths that favour page boundaries (16 k - 1, 16 k, 16 k + 1)
    and short contexts equal to q_len."""
    rng = np.random.default_rng(1000 + seed)
    D = int(rng.choice([64, 128]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    while True:
        G = int(rng.choice([1, 2, 3, 4, 6, 8, 16]))
        Qmax = int(rng.choice([1, 2, 3, 4, 5, 6, 8, 16]))
        if G * Qmax <= 64:
            break
    B = int(rng.integers(1, 24))
    ql = rng.integers(0, Qmax + 1, size=B)
    ql[rng.integers(0, B)] = Qmax                      # at least one full draft block
    ctx = []
    for q in ql:
        kind = rng.integers(0, 4)
        if kind == 0:
            L = max(int(q), 1)                         # nothing but the draft block
        elif kind == 1:
            L = 16 * int(rng.integers(1, 40)) + int(rng.integers(-1, 2))
        else:
            L = int(rng.integers(1, 2500))
        ctx.append(max(L, int(q), 1))
    return dict(Hq=G * Hkv, Hkv=Hkv, D=D, q_lens=[int(x) for x in ql], ctx_lens=ctx, Qmax=Qmax)


@pytest.mark.parametrize("seed", range(24))
def test_random_shapes(dev, orc, seed):
    sh = random_shape(seed)
    wl = synth.make_workload(f"rand{seed}", seed=seed, cfg=small_cfg(sh["Hq"], sh["Hkv"], sh["D"]),
                             ctx_lens=sh["ctx_lens"], q_lens=sh["q_lens"], Qmax=sh["Qmax"], poison=True,
                             spare_pages=1)
    run_case(dev, orc, wl, workers=(0, 5, 333))


@pytest.mark.parametrize("B,Qmax", [(513, 1), (1100, 4), (4096, 1)])
def test_many_sequences(dev, orc, B, Qmax):
    """Past the 512 sequences whose lengths the partition loads in one batch,
    up to the largest supported batch (4096), with ragged lengths and some
    sequences skipped (q_len 0)."""
    rng = np.random.default_rng(B)
    ctx = rng.integers(1, 90, size=B)
    ctx[rng.integers(0, B, size=8)] = 700
    q = np.minimum(rng.integers(0, Qmax + 1, size=B) if Qmax > 1 else np.ones(B, np.int64), ctx)
    q[rng.integers(0, B, size=5)] = 0
    wl = synth.make_workload(f"many{B}", seed=B, cfg=small_cfg(8, 2, 64), ctx_lens=ctx.tolist(),
                             q_lens=q.tolist(), Qmax=Qmax, poison=True, spare_pages=1)
    run_case(dev, orc, wl, workers=(0, 5, 2000))


def test_random_worker_counts_every_combine_mode(dev, orc):
    """Random shapes (a third of them a few long sequences, so units hold many
    pieces) at the automatic and at a random worker count, every variant,
    one workspace for all calls: every output element against the oracle,
    the canaries untouched, the counter area zero after each call, and each
    of the three ways of combining splits taken at least once."""
    import torch
    binding, device = dev
    ws = binding.new_workspace(640 << 20)
    seen = set()
    for seed in range(36):
        rng = np.random.default_rng(7000 + seed)
        sh = random_shape(seed + 5000)
        if seed % 3 == 0:
            Hkv = int(rng.choice([1, 2, 8]))
            Qmax = int(rng.choice([1, 2, 4, 8, 16]))
            G = int(rng.choice([g for g in (1, 2, 4, 8) if g * Qmax <= 64]))
            ql = [int(x) for x in rng.integers(1, Qmax + 1, size=int(rng.integers(1, 4)))]
            ql[0] = Qmax
            sh = dict(Hq=G * Hkv, Hkv=Hkv, D=int(rng.choice([64, 128])), Qmax=Qmax, q_lens=ql,
                      ctx_lens=[int(max(q, rng.integers(1000, 30000))) for q in ql])
        wl = synth.make_workload(f"modes{seed}", seed=seed, cfg=small_cfg(sh["Hq"], sh["Hkv"], sh["D"]),
                                 ctx_lens=sh["ctx_lens"], q_lens=sh["q_lens"], Qmax=sh["Qmax"], poison=True,
                                 spare_pages=1)
        ref = oracle_out(orc, wl, nthreads=8)
        t = device.upload(wl)
        for var in variants_for(wl):
            for w in (0, int(rng.choice([1, 7, 64, 333, 1024, 2048, 4096]))):
                plan = binding.decode_attn_plan(binding.shape_of(t["q"], t["k_pages"], t["page_table"],
                                                                 max(1, wl.max_ctx_len), num_workers=w,
                                                                 variant=var))
                seen.add(plan["combine"])
                say(f"modes seed={seed} B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Qmax={wl.Qmax} "
                    f"variant={var} workers={w} combine={plan['combine']}")
                t["out_full"].fill_(device.CANARY)
                device.run(wl, t, num_workers=w, variant=var, workspace=ws)
                assert_parity(device.out_as_f64(t), ref, f"modes{seed} v{var} w{w}")
                canary_ok(t, wl)
                torch.cuda.synchronize()
                assert int(ws[:1 << 20].count_nonzero()) == 0, f"counters left set: seed {seed} v{var} w{w}"
    assert seen == {binding.COMBINE_MERGE_KERNEL, binding.COMBINE_LAST_ARRIVER, binding.COMBINE_IN_LAUNCH}, seen


def test_workspace_reused_across_calls_and_shapes(dev, orc):
    """One zero-filled workspace serves a run of calls of different shapes and
    worker counts; each result matches the oracle, and after every call the
    per-unit arrival counters (the first B * Hkv int32 of the workspace) are
    zero again."""
    import torch
    from paper_2608_22788_amd import binding
    _, device = dev
    ws = binding.new_workspace(64 << 20)
    cases = [(32, 8, 128, [1] * 5, [1, 15, 16, 33, 1000], 0), (8, 2, 64, [1] * 3, [16, 17, 300], 3),
             (32, 8, 128, [4, 4], [500, 77], 0), (32, 8, 128, [1] * 40, [130] * 40, 300),
             (16, 2, 128, [1, 1, 1], [64, 65, 511], 1), (32, 8, 128, [1] * 256, [40] * 256, 0)]
    for n, (Hq, Hkv, D, ql, cl, w) in enumerate(cases):
        wl = synth.make_workload(f"reuse{n}", seed=40 + n, cfg=small_cfg(Hq, Hkv, D), ctx_lens=cl, q_lens=ql)
        ref = oracle_out(orc, wl)
        t = device.upload(wl)
        say(f"reuse case {n}: B={wl.B} Hq={Hq} Hkv={Hkv} D={D} workers={w}")
        device.run(wl, t, num_workers=w, workspace=ws)
        assert_parity(device.out_as_f64(t), ref, f"reuse{n}")
        torch.cuda.synchronize()
        assert int(ws[:1 << 20].count_nonzero()) == 0, f"counters left set after case {n}"


@pytest.mark.parametrize("Qmax", [1, 4])
def test_in_kernel_combine_with_many_pieces(dev, orc, Qmax):
    """Skewed lengths so that units are plentiful (in-kernel combining is on:
    units >= 2 x workers) while one long sequence's units are each split over
    ~40 workers, more pieces than one combine batch holds."""
    binding, device = dev
    ctx = [50000] + [16 + (7 * b) % 40 for b in range(99)]
    q = [Qmax] * 100
    wl = synth.make_workload("manypieces", seed=21, cfg=small_cfg(32, 8, 128), ctx_lens=ctx, q_lens=q,
                             poison=True, spare_pages=1)
    ref = oracle_out(orc, wl)
    t = device.upload(wl)
    for var in (0, 1, 3) if Qmax == 1 else (0, 1):
        for w in (300, 397):
            say(f"many pieces Qmax={Qmax} variant={var} workers={w}")
            plan = binding.decode_attn_plan(binding.shape_of(t["q"], t["k_pages"], t["page_table"],
                                                             wl.max_ctx_len, num_workers=w, variant=var))
            assert plan["combine"] == binding.COMBINE_LAST_ARRIVER and plan["grid"] == w, plan
            t["out_full"].fill_(device.CANARY)
            device.run(wl, t, num_workers=w, variant=var)
            got = device.out_as_f64(t)
            canary_ok(t, wl)
            assert_parity(got, ref, f"manypieces v{var} w{w}")


# Few units with many pieces each (workers >= 8 x units) and at most 512
# merge workgroups: merge wavefronts that follow the workers in the grid
# combine the splits.  (name, Hq, Hkv, D, q_lens, ctx_lens); with the
# automatic worker count: 16 units for 768 workers (256 merge wavefronts),
# 32 units for 1,024 (128), 16 units for 512 teams (256 workgroups).
IN_LAUNCH = [
    ("verify_q4", 32, 8, 128, [4, 3], [20000, 3001]),              # one draft shorter than max_q_len
    ("decode_q1", 32, 8, 128, [1, 1, 1, 0], [9000, 40, 17000, 500]),  # a unit whole in one worker, a skipped sequence
    ("team_q16", 32, 8, 128, [16, 5], [30000, 7000]),              # 64 rows: the team kernel
    ("d64_g8", 64, 8, 64, [2, 2], [12000, 16]),
]
# variants whose plan is not the in-launch merge: 64 rows on one wavefront
# need 16 units x 64 merge wavefronts, more than the launch takes
NOT_IN_LAUNCH = {("team_q16", 1)}


@pytest.mark.parametrize("case", IN_LAUNCH, ids=[c[0] for c in IN_LAUNCH])
def test_merge_in_the_launch(dev, orc, case):
    """Every variant, with the automatic worker count and with 4,096 workers
    (more than one resident round, so merge workgroups start only after
    several rounds of workers); every output element against the oracle, the
    canaries untouched, and the workspace's counter area zero after each
    call."""
    import torch
    from paper_2608_22788_amd import binding
    _, device = dev
    name, Hq, Hkv, D, ql, cl = case
    wl = synth.make_workload(f"inlaunch_{name}", seed=31, cfg=small_cfg(Hq, Hkv, D), ctx_lens=cl, q_lens=ql,
                             poison=True, spare_pages=1)
    ref = oracle_out(orc, wl)
    t = device.upload(wl, values="device")
    ws = binding.new_workspace(640 << 20)
    for var in variants_for(wl):
        for w in (0, 4096):
            say(f"in-launch merge {name} variant={var} workers={w}")
            plan = binding.decode_attn_plan(binding.shape_of(t["q"], t["k_pages"], t["page_table"],
                                                             max(1, wl.max_ctx_len), num_workers=w, variant=var))
            want = binding.COMBINE_MERGE_KERNEL if (name, var) in NOT_IN_LAUNCH else binding.COMBINE_IN_LAUNCH
            assert plan["combine"] == want, plan
            if want == binding.COMBINE_IN_LAUNCH:
                assert plan["grid"] > plan["num_workers"] and plan["merge_blocks"] == 0, plan
            t["out_full"].fill_(device.CANARY)
            device.run(wl, t, num_workers=w, variant=var, workspace=ws)
            got = device.out_as_f64(t)
            assert_parity(got, ref, f"inlaunch {name} v{var} w{w}")
            canary_ok(t, wl)
            torch.cuda.synchronize()
            assert int(ws[:1 << 20].count_nonzero()) == 0, f"counters left set: {name} v{var} w{w}"


def test_no_work_at_all():
    """Every sequence skipped (q_lens all 0): no pages carry work, every
    variant returns without touching the output."""
    from paper_2608_22788_amd import device
    import torch
    wl = synth.make_workload("empty", seed=11, cfg=small_cfg(32, 8, 128), ctx_lens=[40, 900, 17],
                             q_lens=[0, 0, 0], Qmax=4)
    t = device.upload(wl)
    for var in (0, 1, 2):
        for w in (0, 1, 50):
            t["out_full"].fill_(device.CANARY)
            device.run(wl, t, num_workers=w, variant=var)
            torch.cuda.synchronize()
            canary_ok(t, wl)


def test_one_key_returns_value_row_bitwise(dev, orc):
    _, device = dev
    for Qmax, var in ((1, 0), (1, 3), (2, 1), (2, 2)):
        wl = synth.make_workload("onekey", seed=9, cfg=small_cfg(32, 8, 128), ctx_lens=[1, 1, 1],
                                 q_lens=[1, 1, 1], Qmax=Qmax)
        t = device.upload(wl)
        device.run(wl, t, variant=var)
        out = t["out"].view(__import__("torch").int16).cpu().numpy().view(np.uint16)
        vp = wl.v_pages()
        for b in range(3):
            for h in range(32):
                assert np.array_equal(out[b, 0, h], vp[wl.page_table[b, 0], h // 4, 0]), (Qmax, b, h)


def test_constant_values_give_exactly_that_value(dev):
    import torch
    _, device = dev
    for q, var in ((1, 0), (1, 3), (4, 1), (4, 2), (16, 1), (16, 2)):
        wl = synth.make_workload("constv", seed=4, cfg=small_cfg(32, 8, 128), ctx_lens=[q + 40, 3000],
                                 q_lens=[q, q])
        t = device.upload(wl, values="device")
        t["v_pages"].fill_(1.0)
        device.run(wl, t, variant=var)
        got = device.out_as_f64(t)
        assert (got[:, :q] == 1.0).all(), (q, var)


def test_page_relabel_is_bitwise_invariant(dev):
    import torch
    _, device = dev
    wl = synth.make_workload("relabel", seed=5, cfg=small_cfg(32, 8, 128), ctx_lens=[100, 3001, 64],
                             q_lens=[4, 4, 2])
    t = device.upload(wl)
    device.run(wl, t)
    base = t["out"].clone()
    perm = torch.from_numpy(np.random.default_rng(0).permutation(wl.num_pages)).cuda()
    k2 = torch.empty_like(t["k_pages"])
    v2 = torch.empty_like(t["v_pages"])
    k2[perm] = t["k_pages"]
    v2[perm] = t["v_pages"]
    t["k_pages"], t["v_pages"] = k2, v2
    t["page_table"] = perm[t["page_table"].long()].int().contiguous()
    device.run(wl, t)
    assert torch.equal(t["out"].view(torch.int16), base.view(torch.int16))


def test_run_to_run_bitwise_deterministic(dev):
    import torch
    _, device = dev
    for name in ("tiny", "mtp"):
        wl = synth.make_workload(name, seed=1)
        t = device.upload(wl, values="device")
        device.run(wl, t)
        first = t["out"].clone()
        for _ in range(2):
            device.run(wl, t)
            assert torch.equal(t["out"].view(torch.int16), first.view(torch.int16)), name


def test_verify_rows_equal_prefix_decodes(dev, orc):
    import torch
    _, device = dev
    L, Q = 2000, 6
    wl = synth.make_workload("vp", seed=6, cfg=small_cfg(32, 8, 128), ctx_lens=[L], q_lens=[Q])
    t = device.upload(wl)
    device.run(wl, t)
    full = device.out_as_f64(t)
    for i in range(Q):
        one = synth.make_workload("vp1", seed=6, cfg=small_cfg(32, 8, 128), ctx_lens=[L - Q + i + 1],
                                  q_lens=[1])
        t1 = device.upload(one)
        t1["k_pages"], t1["v_pages"] = t["k_pages"], t["v_pages"]
        t1["page_table"] = t["page_table"]
        t1["q"] = t["q"][:, i:i + 1].contiguous()
        device.run(one, t1, workspace=None)
        got = device.out_as_f64(t1)
        assert_parity(got[0, 0][None, None], full[0, i][None, None], f"row{i}")


def test_split_points_do_not_change_the_result(dev):
    import torch
    _, device = dev
    wl = synth.make_workload("split", seed=2, cfg=synth.CONFIGS["dflash"], ctx_lens=[20000, 333],
                             q_lens=[16, 16])
    t = device.upload(wl, values="device")
    outs = []
    for var in (1, 2):
        for w in (1, 2, 7, 0, 300):
            device.run(wl, t, num_workers=w, variant=var)
            outs.append(device.out_as_f64(t))
    for o in outs[1:]:
        assert_parity(o, outs[0], "split")


# ---------------------------------------------------------------------------
# full-size workloads against the oracle
# ---------------------------------------------------------------------------

FULL = {"bulk": 6, "mtp": 3, "dflash": 2}


@pytest.mark.parametrize("name", list(FULL))
def test_full_size_config(dev, orc, name):
    """The benchmarked workloads in full: every sequence, row and head of the
    call against the oracle, for the automatic launch (the one the benchmark
    times) and every other kernel variant."""
    _, device = dev
    wl = synth.make_workload(name, seed=0)
    say(f"full {name}: B={wl.B} sum_ctx={int(wl.ctx_lens.sum())} max={wl.max_ctx_len} "
        f"KV={wl.kv_bytes() / 1e9:.2f} GB")
    t = device.upload(wl, values="device")
    say(f"  oracle over the whole call (host inputs)")
    ref = oracle_out(orc, wl)
    for var in variants_for(wl):
        t["out_full"].fill_(device.CANARY)
        device.run(wl, t, variant=var)      # variant 0 / auto is the benchmarked launch
        got = device.out_as_f64(t)
        canary_ok(t, wl)
        assert np.isfinite(got[~np.isnan(ref)]).all()
        assert_parity(got, ref, f"{name} all {wl.B} seqs variant {var}")
        # and no sequence is far off while the whole stays inside the bar
        worst = max(float(np.nanmax(np.abs(got[b] - ref[b]))) for b in range(wl.B))
        assert worst <= 2e-2, f"{name} variant {var}: a sequence has max_abs {worst:g}"


@pytest.mark.parametrize("name", ["bulk", "dflash"])
def test_full_size_tp2_share(dev, orc, name):
    """One GPU's share of a two-way tensor-parallel replica: the same
    sequences with half the heads (16 query / 4 KV), sampled against the
    oracle.  At 1,024 units for 1,024 workers the bulk share takes the merge
    kernel instead of combining its splits in the kernel."""
    _, device = dev
    cfg = dict(synth.CONFIGS[name], Hq=16, Hkv=4)
    wl = synth.make_workload(name + "_tp2", seed=0, cfg=cfg)
    say(f"tp2 share {name}: B={wl.B} heads 16/4 sum_ctx={int(wl.ctx_lens.sum())}")
    t = device.upload(wl, values="device")
    seqs = sample_seqs(wl, FULL[name])
    ref = oracle_out(orc, wl.subset(seqs))
    for var in variants_for(wl):
        t["out_full"].fill_(device.CANARY)
        device.run(wl, t, variant=var)
        got = device.out_as_f64(t)
        canary_ok(t, wl)
        assert np.isfinite(got).all()
        assert_parity(got[seqs], ref, f"{name} tp2 seqs {seqs} variant {var}")


@pytest.mark.parametrize("Hq,Hkv,ql", [(32, 4, 1), (64, 4, 1), (32, 4, 4)])
def test_full_size_group_sizes(dev, orc, Hq, Hkv, ql):
    """The bulk sequences at GQA group sizes 8 and 16 (the benchmark's
    group_sizes field), sampled against the oracle."""
    _, device = dev
    cfg = dict(synth.CONFIGS["bulk"], Hq=Hq, Hkv=Hkv, q_len=ql)
    wl = synth.make_workload(f"bulk_g{Hq // Hkv}_q{ql}", seed=0, cfg=cfg)
    say(f"group size {Hq // Hkv}, q_len {ql}: B={wl.B} sum_ctx={int(wl.ctx_lens.sum())}")
    t = device.upload(wl, values="device")
    seqs = sample_seqs(wl, 3)
    ref = oracle_out(orc, wl.subset(seqs))
    for var in variants_for(wl):
        t["out_full"].fill_(device.CANARY)
        device.run(wl, t, variant=var)
        got = device.out_as_f64(t)
        canary_ok(t, wl)
        assert np.isfinite(got).all()
        assert_parity(got[seqs], ref, f"G{Hq // Hkv} q{ql} seqs {seqs} variant {var}")


def test_full_size_ragged_mixed_batch(dev, orc):
    """One launch over the bulk workload in which the 8 longest sequences
    verify 4 drafted tokens and the other 248 decode one (ragged q_lens under
    max_q_len 4), the benchmark's mixed-batch case; rows of both kinds
    against the oracle (every sequence), padded rows untouched."""
    _, device = dev
    base = synth.make_workload("bulk", seed=0)
    tail = np.argsort(base.ctx_lens)[::-1][:8]
    ql = np.ones(base.B, dtype=np.int64)
    ql[tail] = 4
    wl = synth.make_workload("bulk", seed=0, q_lens=ql.tolist(), Qmax=4)
    t = device.upload(wl, values="device")
    ref = oracle_out(orc, wl)
    for var in variants_for(wl):
        t["out_full"].fill_(device.CANARY)
        device.run(wl, t, variant=var)
        got = device.out_as_f64(t)
        canary_ok(t, wl)
        assert_parity(got, ref, f"mixed all seqs variant {var}")


SWEEP_CASES = [(b, 0) for b in synth.SWEEP_BATCHES] + \
              [(b, s) for b in synth.SWEEP_BATCHES if b <= 64 for s in range(1, 5)]


@pytest.mark.parametrize("batch,seed", SWEEP_CASES)
def test_sweep_workload(dev, orc, batch, seed):
    """Every sweep point of seed 0, and of seeds 1-4 up to 64 sequences, in
    full against the oracle."""
    _, device = dev
    wl = synth.make_workload(f"sweep_b{batch}", seed=seed)
    say(f"sweep b={batch} seed={seed}: q_len={wl.Qmax} sum_ctx={int(wl.ctx_lens.sum())}")
    t = device.upload(wl, values="device")
    device.run(wl, t)
    got = device.out_as_f64(t)
    canary_ok(t, wl)
    assert np.isfinite(got).all()
    ref = oracle_out(orc, wl)
    assert_parity(got, ref, f"sweep b{batch} s{seed} all seqs")


def test_concurrency_sweep_entry_point(dev):
    binding, _ = dev
    pts = binding.concurrency_sweep(batches=(1, 16, 128), seeds=2, warmup=2, iters=10,
                                    min_rotation_bytes=1 << 30)
    assert len(pts) == 6
    for p in pts:
        say(f"  sweep point {p}")
        assert p["q_len"] == (4 if p["batch"] <= 8 else 1)
        lens = synth.lengths_sweep(p["seed"], p["batch"])
        assert p["sum_ctx"] == int(lens.sum())
        assert p["kv_bytes"] == int(lens.sum()) * 8 * 128 * 4
        assert p["num_pools"] * p["kv_bytes"] >= (1 << 30)
        assert 0 < p["t_p10_us"] <= p["t_median_us"] <= p["t_p90_us"]
        assert p["kv_gbps"] > 0 and p["hbm_frac"] < 1.2
        # the read-only twin over the same pools: positive, and no slower than
        # the whole attention call by more than timing noise
        assert 0 < p["gather_median_us"] < 1.2 * p["t_median_us"]
