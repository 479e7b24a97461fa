#!/usr/bin/env python3
"""Benchmark of the decode / verify attention hot path on one MI355X.

One step = one ts_decode_attn call (plan + launch, split-KV streaming
kernel, log-sum-exp merge) over one batch of the bulk-pool workload: 256
sequences, one query token each, 32 query / 8 KV heads, head_dim 128,
context = prompt U{256..1024} + response min(lognormal(median 2048,
sigma 0.8), 16384), page size 16, bf16 N(0,1) values, seed 0.  Inputs are
resident in HBM before timing; calls rotate over distinct KV pools (like the
layers of a model) so the 256 MB last-level cache cannot serve a pool twice
in a row.

Printed: one JSON line with the bulk KV GB/s as ``value``, the roofline of
the streaming kernel (its average duration from HIP events recorded around
it on its own stream), the float64 oracle timed on this host's cores, the
two tail-pool verify workloads and the concurrency curve (mean, min and max
over 5 seeds per batch size).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time
import traceback

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_GBPS = 8000.0          # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_counters.md")
# Files whose content decides the streaming kernel of each workload and its
# launch; a traffic figure counts only while their hash matches the one it was
# measured on.
TRAFFIC_SOURCES = {
    "bulk": ["csrc/attn_common.h", "csrc/attn_split.h", "csrc/attn_verify.hip", "csrc/api.hip", "build.py"],
    "mtp": ["csrc/attn_common.h", "csrc/attn_split.h", "csrc/attn_verify.hip", "csrc/api.hip", "build.py"],
    "dflash": ["csrc/attn_common.h", "csrc/attn_split.h", "csrc/attn_verify_team.hip", "csrc/api.hip", "build.py"],
}
KERNELS = {"bulk": "verify_kernel<128,1>", "mtp": "verify_kernel<128,1>",
           "dflash": "verify_team_kernel<4>"}

WORKLOADS = {
    "bulk": "bulk pool decode: 256 seqs, q_len 1, 32 q / 8 kv heads, d128, page 16, "
            "ctx = U{256..1024} + min(lognormal(median 2048, sigma 0.8), 16384), bf16 N(0,1), seed 0",
    "mtp": "tail pool MTP verify: 8 seqs, q_len 4 causal, 32/8 heads, d128, ctx U{16384..65536}",
    "dflash": "tail pool block-draft verify: 4 seqs, q_len 16 causal, 32/8 heads, d128, "
              "ctx U{32768..98304}",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _code_only(text: str) -> str:
    """Source text without comments and blank-space differences, so that an
    edit of comments alone does not count as a kernel change."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    text = re.sub(r"#[^\n]*$", lambda m: m.group(0), text, flags=re.M)
    return " ".join(text.split())


def kernel_hash(name: str) -> str:
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES.get(name, []):
        with open(os.path.join(ROOT, "paper_2608_22788_amd", f), encoding="utf-8") as fh:
            text = fh.read()
        if not f.endswith(".py"):
            text = _code_only(text)
        h.update(text.encode())
    return h.hexdigest()[:16]


def measured_traffic(name: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    they were taken on the current kernel sources (else None)."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(rf"^traffic {name} kernel_hash=(\w+) bytes_per_launch=(\d+)$", text, re.M)
    if not m or m.group(1) != kernel_hash(name):
        return None
    return int(m.group(2))


def make_pools(wl, n_pools):
    """n_pools copies of the KV pool, carved out of one allocation (as a
    serving engine holds its KV cache in one preallocated arena): pool 0 holds
    the workload's values, pool p the next values of the same streams."""
    import torch
    from paper_2608_22788_amd import binding, device, synth
    shp = (wl.num_pages, wl.Hkv, wl.P, wl.D)
    arena = torch.empty((n_pools, 2) + shp, dtype=torch.bfloat16, device="cuda")
    elems = int(np.prod(shp))
    pools = []
    for p in range(n_pools):
        k, v = arena[p, 0], arena[p, 1]
        binding.synth_fill(k, wl.seed, synth.S_K, p * elems)
        binding.synth_fill(v, wl.seed, synth.S_V, p * elems)
        pools.append((k, v))
    t = device.upload(wl, values="device")
    t["k_pages"], t["v_pages"] = pools[0]
    t["arena"] = arena
    return t, pools


# The GPU needs tens of milliseconds of this load before its clocks settle
# (the first ~100 block-draft calls run up to 15 % slower), so the tail
# workloads get at least this much untimed warm-up; the bulk step gets exactly
# --warmup calls (100 by default, about 50 ms).
MIN_WARMUP_MS = 60.0

# Kernel durations come from HIP events attached to the streaming kernel's
# dispatch.  A dispatch that carries them measured about 4.6 us longer per
# call back to back (bulk: 490.1 against 485.5 us per call, kernel 484.6 us
# in both), so inside the timed region only every EVENT_EVERY-th call carries
# events; the kernel average is taken over those calls.
EVENT_EVERY = 10


def stream_read_gbps(buf, calls=10):
    """Sequential read ceiling: the library's streaming read over `buf`
    (median of `calls` timed reads after 3 untimed ones)."""
    import torch
    from paper_2608_22788_amd import binding
    flat = buf.view(-1).view(torch.uint8)
    sink = torch.empty(2 << 20, dtype=torch.uint8, device="cuda")
    for _ in range(3):
        binding.stream_read(flat, sink)
    ev = [(binding.Event(), binding.Event()) for _ in range(calls)]
    for a, b in ev:
        a.record()
        binding.stream_read(flat, sink)
        b.record()
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_ms(b) for a, b in ev]))
    return dict(bytes=flat.numel(), ms=round(ms, 4), gbps=round(flat.numel() / (ms * 1e-3) / 1e9, 1))


def tp2_share(name):
    """The per-GPU share of a two-way tensor-parallel replica of a workload:
    half the query and KV heads, the same sequences and lengths."""
    from paper_2608_22788_amd import synth
    cfg = dict(synth.CONFIGS[name])
    cfg["Hq"], cfg["Hkv"] = cfg["Hq"] // 2, cfg["Hkv"] // 2
    return cfg


def time_workload(name, steps, warmup, min_warmup_ms=0.0, min_rotation=4 << 30, ceiling=True,
                  stream_ceiling=False, cfg=None):
    import torch
    from paper_2608_22788_amd import binding, synth
    wl = synth.make_workload(name, seed=0, cfg=cfg)
    kv = wl.kv_bytes()
    n_pools = max(2, -(-min_rotation // kv))
    log(f"[bench] {name}: B={wl.B} q_len={wl.Qmax} sum_ctx={int(wl.ctx_lens.sum())} "
        f"KV={kv / 1e9:.3f} GB pools={n_pools}")
    t, pools = make_pools(wl, n_pools)
    shape = binding.shape_of(t["q"], t["k_pages"], t["page_table"], wl.max_ctx_len)
    ws = binding.new_workspace(binding.workspace_size(shape))
    plan = binding.decode_attn_plan(shape)
    ev = [(binding.Event(), binding.Event()) for _ in range(steps)]
    sampled = range(0, steps, EVENT_EVERY)   # timed calls that carry kernel events

    def call(i, events=None):
        k, v = pools[i % n_pools]
        binding.decode_attn(t["q"], k, v, t["page_table"], t["ctx_lens"], t["q_lens"], t["out"],
                            wl.scale, workspace=ws, max_ctx_len=wl.max_ctx_len, events=events)

    torch.cuda.synchronize()
    w0 = time.perf_counter()
    i = 0
    while i < warmup or (time.perf_counter() - w0) * 1e3 < min_warmup_ms:
        call(i)
        i += 1
        if i % 16 == 0:
            torch.cuda.synchronize()
    warmup = i
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        call(warmup + i, ev[i] if i % EVENT_EVERY == 0 else None)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / steps
    kern_ms = np.array([ev[i][0].elapsed_ms(ev[i][1]) for i in sampled])
    alg = wl.algorithmic_bytes()
    extra = {}
    if ceiling:
        # the same pages, the same partition and loads, no arithmetic: the
        # ceiling of this access pattern, timed on the same rotation of pools
        # (a failure here is reported, the attention timing is kept)
        try:
            sink = torch.empty(1024 * 64, dtype=torch.int32, device="cuda")

            def gather(i, events=None):
                k, v = pools[i % n_pools]
                binding.page_gather_read(k, v, t["page_table"], t["ctx_lens"], t["q_lens"], sink,
                                         max_ctx_len=wl.max_ctx_len, events=events)

            for i in range(10):
                gather(i)
            for i in range(steps):
                gather(10 + i, ev[i])
            torch.cuda.synchronize()
            g_ms = float(np.mean([a.elapsed_ms(b) for a, b in ev]))
            extra = dict(gather_ms_mean=g_ms, gather_gbps=alg / (g_ms * 1e-3) / 1e9,
                         kernel_frac_of_gather=g_ms / float(kern_ms.mean()))
            if stream_ceiling:
                extra["stream_read"] = stream_read_gbps(t["arena"])
        except Exception as e:   # noqa: BLE001
            log(f"[bench] {name}: ceiling measurement failed: {e!r}")
            extra = dict(ceiling_error=repr(e))
    # the output of one more call on pool 0 (the workload's own values) for
    # the parity check against the oracle
    k, v = pools[0]
    binding.decode_attn(t["q"], k, v, t["page_table"], t["ctx_lens"], t["q_lens"], t["out"],
                        wl.scale, workspace=ws, max_ctx_len=wl.max_ctx_len)
    torch.cuda.synchronize()
    from paper_2608_22788_amd import device
    out_f64 = device.out_as_f64(t)
    # the memory stays in torch's cache for the next workload: memory obtained
    # from the driver again after a free streams up to 5 % slower here
    del pools, t, ws
    qtok = int(wl.q_lens.sum())
    return dict(workload=name, warmup_calls=warmup, kv_bytes=kv, alg_bytes=alg, ms_per_step=ms_step,
                kernel_ms_mean=float(kern_ms.mean()), kernel_ms_median=float(np.median(kern_ms)),
                kernel_ms_p10=float(np.percentile(kern_ms, 10)), kernel_ms_p90=float(np.percentile(kern_ms, 90)),
                kv_gbps=kv / (ms_step * 1e-3) / 1e9,
                kernel_gbps=alg / (kern_ms.mean() * 1e-3) / 1e9,
                query_tokens_per_s=qtok / (ms_step * 1e-3), tokens_per_s=wl.B / (ms_step * 1e-3),
                n_pools=n_pools, plan=plan_summary(plan), wl=wl, out_f64=out_f64, **extra)


PLAN_KERNEL = {1: "single-wavefront matrix-core", 2: "team of four wavefronts", 3: "VALU"}
PLAN_COMBINE = {0: "merge kernel after the launch", 1: "last arriver in the launch",
                2: "merge wavefronts in the launch"}


def plan_summary(plan):
    """What the timed call launched (ts_decode_attn_plan): kernel, workers,
    how its splits were combined, workgroups of the streaming launch."""
    return dict(kernel=PLAN_KERNEL.get(plan["variant"], str(plan["variant"])), workers=plan["num_workers"],
                combine=PLAN_COMBINE.get(plan["combine"], str(plan["combine"])), grid=plan["grid"])


def parity_errors(got, ref):
    """Max-abs, mean-abs and relative L2 error over the valid output rows
    (the oracle marks rows i >= q_lens[b] with NaN)."""
    m = ~np.isnan(ref)
    d = got[m] - ref[m]
    return dict(max_abs=float(np.abs(d).max()), mean_abs=float(np.abs(d).mean()),
                rel_l2=float(np.linalg.norm(d) / np.linalg.norm(ref[m])), elements=int(m.sum()),
                finite=bool(np.isfinite(got[m]).all()))


# Parity bar on bf16 outputs with N(0,1) inputs (max-abs, mean-abs), plus the
# relative L2 bar that keeps the check meaningful at long context.
PARITY_BAR = dict(max_abs=2e-2, mean_abs=2e-3, rel_l2=1e-2)


def oracle_leg(r, threads, min_seconds=0.0, max_runs=50):
    """The float64 oracle on this host's cores over the whole call of a timed
    workload: its time per call (repeated for about min_seconds, bounded by
    max_runs) and the parity of the GPU output of the same call."""
    import oracle
    orc = oracle.load()
    wl = r["wl"]
    log(f"[bench] oracle {r['workload']}: generating host inputs")
    q, k, v = wl.q_values(), wl.k_pages(), wl.v_pages()
    log(f"[bench] oracle {r['workload']}: {threads} threads")
    runs, ref, t0 = 0, None, time.perf_counter()
    while runs < max_runs:
        o = orc.attention(q, k, v, wl.page_table, wl.ctx_lens, wl.q_lens, wl.scale, nthreads=threads)
        ref = o if ref is None else ref
        runs += 1
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = (time.perf_counter() - t0) / runs
    del q, k, v
    par = parity_errors(r["out_f64"], ref)
    par["within_bar"] = par["finite"] and all(par[key] <= bar for key, bar in PARITY_BAR.items())
    par = {key: (float(f"{val:.4g}") if isinstance(val, float) else val) for key, val in par.items()}
    par["oracle_s"] = round(dt, 4)
    return dt, runs, par


def cpu_baseline(bulk, tails, min_seconds=10.0, max_runs=50):
    """The float64 oracle on this host's cores over the whole bulk call,
    repeated until about min_seconds of work (bounded by max_runs), then once
    over each tail workload's whole call; every GPU output of those calls is
    compared with it element by element."""
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    wl = bulk["wl"]
    dt, runs, par_bulk = oracle_leg(bulk, threads, min_seconds, max_runs)
    parity = {"bulk": par_bulk}
    for name, r in tails.items():
        if r is not None and "wl" in r:
            parity[name] = oracle_leg(r, threads)[2]
    return dict(value=wl.kv_bytes() / dt / 1e9, unit="GB/s", cores=threads, kind="oracle",
                sample=f"whole bulk call ({wl.B} seqs, {int(wl.ctx_lens.sum())} context tokens), "
                       f"float64, {runs} runs, {dt:.3f} s each",
                seconds_per_call=round(dt, 4), os_cpu_count=os.cpu_count(),
                omp_num_threads=os.environ.get("OMP_NUM_THREADS"),
                parity=parity, parity_bar=PARITY_BAR,
                parity_note="GPU output of one timed-configuration call per workload against the "
                            "oracle over every sequence, row and head of that call")


def makespan_model(decode_rows, wl):
    """The measured curve fed into the completion-time model (Sec. 2.1,
    App. D) for the bulk pool, which decodes one token per step: tau(b) =
    mean attention time per step over the seeds at q_len 1, tabulated for
    b = 1..512, then the bulk workload's lengths decoded on one replica: its
    completion time and the share of the longest 5 % of requests.  Only
    q_len 1 points enter (verify points describe another regime)."""
    from paper_2608_22788_amd import binding
    rows = sorted((r for r in decode_rows if r["q_len"] == 1), key=lambda r: r["batch"])
    b = [r["batch"] for r in rows]
    tau = binding.tau_table(b, [r["tau_us"] for r in rows], max(b))
    L = wl.ctx_lens.astype(np.int64)
    T = binding.replica_time(tau, L)
    sh = binding.request_shares(tau, L)
    top = np.argsort(L)[::-1][:max(1, len(L) // 20)]
    return dict(tau_source="mean call time per batch size at q_len 1 (sweep points with q_len 1, "
                           "plus a q_len 1 run of the sweep at the batch sizes it verifies at)",
                batches=b, bmax=max(b), bulk_requests=len(L), bulk_replica_attention_s=round(T / 1e6, 6),
                longest_5pct_share=round(float(sh[top].sum() / T), 4))


def depth_sweep(depths=(1, 2, 3, 4, 5, 6), seed_count=1):
    """Route-specialised speculative decoding (Sec. 3.4, Sec. 4.3): the same
    concurrency sweep with every batch size verifying q_len = 1 + gamma
    tokens per sequence; the median call time per step.  How many tokens a
    step emits depends on acceptance, which is not modelled here."""
    from paper_2608_22788_amd import binding
    rows = []
    for q in depths:
        pts = binding.concurrency_sweep(seeds=seed_count, warmup=10, iters=20,
                                        verify_max_batch=4096 if q > 1 else 0, verify_q_len=max(q, 1))
        for r in sweep_summary(pts):
            rows.append(dict(q_len=q, batch=r["batch"], kv_gbps=r["kv_gbps"], call_us=r["call_us"]))
    return rows


def mixed_and_graph(steps=50):
    """Ragged mixed batches and graph capture (the engine-side problem the
    paper cites for variable draft lengths, Sec. 3.4).  The bulk workload's
    256 sequences where the 8 longest verify 4 tokens (MTP-3) and the rest
    decode 1, timed as one launch (max_q_len 4, ragged q_lens) against the
    same work as two launches (248 x q_len 1, 8 x q_len 4).  Then a small
    ragged step (8 sequences of the sweep's lengths, q_lens 4,4,1,...)
    captured once into a HIP graph and replayed, against eager calls from
    Python."""
    import torch
    from paper_2608_22788_amd import binding, device, synth
    base = synth.make_workload("bulk", seed=0)
    tail = np.argsort(base.ctx_lens)[::-1][:8]
    ql = np.ones(base.B, dtype=np.int64)
    ql[tail] = 4
    wl = synth.make_workload("bulk", seed=0, q_lens=ql.tolist(), Qmax=4)
    t, pools = make_pools(wl, 2)
    bulk_idx = torch.from_numpy(np.setdiff1d(np.arange(wl.B), tail)).cuda()
    tail_idx = torch.from_numpy(np.sort(tail).copy()).cuda()
    parts = []
    for idx, q in ((bulk_idx, 1), (tail_idx, 4)):
        parts.append(dict(q=t["q"][idx, :q].contiguous(), page_table=t["page_table"][idx].contiguous(),
                          ctx_lens=t["ctx_lens"][idx].contiguous(), q_lens=t["q_lens"][idx].contiguous(),
                          out=torch.empty_like(t["q"][idx, :q]).contiguous()))
    ws = binding.new_workspace(256 << 20)

    def one(i):
        k, v = pools[i % 2]
        binding.decode_attn(t["q"], k, v, t["page_table"], t["ctx_lens"], t["q_lens"], t["out"], wl.scale,
                            workspace=ws, max_ctx_len=wl.max_ctx_len)

    def two(i):
        k, v = pools[i % 2]
        for pt in parts:
            binding.decode_attn(pt["q"], k, v, pt["page_table"], pt["ctx_lens"], pt["q_lens"], pt["out"],
                                wl.scale, workspace=ws, max_ctx_len=wl.max_ctx_len)

    def timed(fn):
        for i in range(100):
            fn(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            fn(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps * 1e6

    res = dict(workload="bulk lengths, 8 longest verify q_len 4, 248 decode q_len 1",
               kv_bytes=wl.kv_bytes(), one_launch_us=round(timed(one), 2), two_launches_us=round(timed(two), 2))
    res["one_launch_kv_gbps"] = round(wl.kv_bytes() / res["one_launch_us"] / 1e3, 1)
    del pools, t, parts

    # a small ragged step in a graph
    sw = synth.make_workload("sweep_b8", seed=0, q_lens=[4, 4, 1, 1, 4, 1, 1, 1], Qmax=4)
    n_pools = max(2, -(-(1 << 30) // sw.kv_bytes()))
    t, pools = make_pools(sw, n_pools)
    ws2 = binding.new_workspace(binding.workspace_size(
        binding.shape_of(t["q"], t["k_pages"], t["page_table"], sw.max_ctx_len)))

    def small(i):
        k, v = pools[i % n_pools]
        binding.decode_attn(t["q"], k, v, t["page_table"], t["ctx_lens"], t["q_lens"], t["out"], sw.scale,
                            workspace=ws2, max_ctx_len=sw.max_ctx_len)

    eager = timed(small)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(n_pools):
                small(i)
    torch.cuda.current_stream().wait_stream(s)
    reps = max(1, 200 // n_pools)
    g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        g.replay()
    torch.cuda.synchronize()
    graph = (time.perf_counter() - t0) / (reps * n_pools) * 1e6
    res.update(graph_workload="8 sequences (sweep lengths), q_lens 4,4,1,1,4,1,1,1",
               eager_python_us=round(eager, 2), graph_replay_us=round(graph, 2))
    del pools, t, g
    return res


def spec_step(steps=50, vocab=151936):
    """One speculative verify step on the MTP and block-draft workloads
    (Sec. 3.4): the KV append of the 1 + gamma new tokens, the verify
    attention, and the lossless acceptance over a 151,936-token vocabulary
    (synthetic fp32 distributions; the drafter's are the target's logits
    plus noise, which accepts about half of the drafts).  Times each kernel
    group alone and the three back to back."""
    import torch
    from paper_2608_22788_amd import binding, synth
    out = {}
    for name in ("mtp", "dflash"):
        wl = synth.make_workload(name, seed=0)
        t, pools = make_pools(wl, 2)
        B, Q, G = wl.B, wl.Qmax, wl.Qmax - 1
        gen = torch.Generator(device="cuda").manual_seed(1)
        logits = torch.randn((B, Q, vocab), device="cuda", generator=gen) * 2.0
        p = torch.softmax(logits, -1).contiguous()
        q = torch.softmax(logits[:, :G] + 0.7 * torch.randn((B, G, vocab), device="cuda", generator=gen),
                          -1).contiguous()
        d = torch.multinomial(q.reshape(-1, vocab), 1, generator=gen).reshape(B, G).to(torch.int32)
        nd = torch.full((B,), G, dtype=torch.int32, device="cuda")
        ua = torch.rand((B, G), device="cuda", generator=gen)
        us = torch.rand((B,), device="cuda", generator=gen)
        na = torch.empty(B, dtype=torch.int32, device="cuda")
        nt = torch.empty(B, dtype=torch.int32, device="cuda")
        kn = torch.randn((B, Q, wl.Hkv, wl.D), device="cuda", generator=gen).to(torch.bfloat16)
        vn = torch.randn((B, Q, wl.Hkv, wl.D), device="cuda", generator=gen).to(torch.bfloat16)
        ws = binding.new_workspace(256 << 20)
        aws = torch.empty(binding.lib.ts_spec_accept_workspace_size(B, vocab), dtype=torch.uint8, device="cuda")

        def append(i):
            k, v = pools[i % 2]
            binding.kv_append(kn, vn, k, v, t["page_table"], t["ctx_lens"], t["q_lens"])

        def attend(i):
            k, v = pools[i % 2]
            binding.decode_attn(t["q"], k, v, t["page_table"], t["ctx_lens"], t["q_lens"], t["out"], wl.scale,
                                workspace=ws, max_ctx_len=wl.max_ctx_len)

        def accept(i):
            binding.spec_accept(p, q, d, nd, ua, us, na, nt, workspace=aws)

        def step(i):
            append(i)
            attend(i)
            accept(i)

        def timed(fn):
            for i in range(50):
                fn(i)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(steps):
                fn(i)
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) / steps * 1e6

        r = {k: round(timed(fn), 2) for k, fn in (("append_us", append), ("attention_us", attend),
                                                    ("accept_us", accept), ("step_us", step))}
        acc = na.cpu().numpy()
        rejected = int((acc < G).sum())
        accept_bytes = (B + rejected) * vocab * 4
        r.update(batch=B, q_len=Q, vocab=vocab, mean_accepted=round(float(acc.mean()), 2),
                 accept_read_bytes=accept_bytes, accept_gbps=round(accept_bytes / r["accept_us"] / 1e3, 1))
        out[name] = r
        del pools, t, p, q, logits
    return out


def sweep_summary(points):
    """Per batch size: mean, min and max over seeds of the sweep figures.
    call_us is the median time of one step; tokens_per_s and tau_us count one
    emitted token per sequence and step (a verify step's accepted drafts are
    not credited), so at q_len > 1 they are a floor."""
    out = []
    for b in sorted({p["batch"] for p in points}):
        ps = [p for p in points if p["batch"] == b]
        q = ps[0]["q_len"]
        row = dict(batch=b, q_len=q, seeds=len(ps),
                   regime="decode (one query token per sequence)" if q == 1 else
                   f"verify ({q} query tokens per sequence, one emitted token per step credited)")
        calls = np.array([p["t_median_us"] for p in ps])
        row["call_us"] = round(float(calls.mean()), 2)
        row["call_us_min"] = round(float(calls.min()), 2)
        row["call_us_max"] = round(float(calls.max()), 2)
        for f, nd in (("kv_gbps", 1), ("hbm_frac", 4), ("tokens_per_s", 0), ("tau_us", 2)):
            xs = np.array([p[f] for p in ps])
            row[f] = round(float(xs.mean()), nd)
            row[f + "_min"] = round(float(xs.min()), nd)
            row[f + "_max"] = round(float(xs.max()), nd)
        if all("gather_median_us" in p for p in ps):
            # the read-only twin over the same pools: the latency floor of the call
            g = np.array([p["kv_bytes"] / (p["gather_median_us"] * 1e-6) / 1e9 for p in ps])
            row["gather_gbps"] = round(float(g.mean()), 1)
            row["call_frac_of_gather"] = round(float(np.mean([p["gather_median_us"] / p["t_median_us"]
                                                               for p in ps])), 4)
        out.append(row)
    return out


def ceiling_summary(r):
    """Measured read ceilings beside the bulk kernel: a sequential stream read
    and the page gather (the kernel's own pages and partition, no arithmetic)."""
    if "ceiling_error" in r:
        return {"error": r["ceiling_error"]}
    if "gather_gbps" not in r:
        return None
    out = {"page_gather_gbps": round(r["gather_gbps"], 1),
           "page_gather_frac_of_peak": round(r["gather_gbps"] / PEAK_GBPS, 4),
           "kernel_frac_of_page_gather": round(r["kernel_frac_of_gather"], 4),
           "note": "GB/s on the kernel's algorithmic bytes; the gather reads the same whole pages "
                   "with the same partition and loads and computes nothing"}
    if "stream_read" in r:
        out["stream_read_gbps"] = r["stream_read"]["gbps"]
        out["stream_read_bytes"] = r["stream_read"]["bytes"]
    return out


def small_batch_trace(iters=100):
    """The library's concurrency sweep (ts_concurrency_sweep, seed 0) at 1, 2,
    4 and 8 sequences, first with 4-token verify and then with one-token
    decode: per point 20 untimed and `iters` timed attention calls back to
    back, then the page-gather twin the same way.  Meant to run under a
    kernel trace (rocprofv3 --kernel-trace), which gives every dispatch's
    start and end; the returned points name what ran, in order, with what
    each call launches (ts_decode_attn_plan) and the sweep's own times."""
    import torch
    from paper_2608_22788_amd import binding, synth
    out = []
    for vmax in (8, 0):
        pts = binding.concurrency_sweep(batches=(1, 2, 4, 8), seeds=1, warmup=20, iters=iters,
                                        verify_max_batch=vmax)
        for pt in pts:
            cfg = dict(synth.sweep_config(pt["batch"]))
            cfg["q_len"] = pt["q_len"]
            wl = synth.make_workload(f"sweep_b{pt['batch']}", seed=0, cfg=cfg)
            maxp = wl.page_table.shape[1]
            plan = binding.decode_attn_plan(binding.make_shape(wl.B, wl.Hq, wl.Hkv, wl.D, wl.Qmax, maxp,
                                                               wl.max_ctx_len, wl.num_pages))
            out.append(dict(batch=pt["batch"], q_len=pt["q_len"], warmup=20, iters=iters,
                            call_us=round(pt["t_median_us"], 2), gather_us=round(pt["gather_median_us"], 2),
                            kv_bytes=pt["kv_bytes"], plan=plan_summary(plan),
                            merge_kernel=plan["merge_blocks"] > 0))
            log(f"[bench] small-batch trace: b={pt['batch']} q_len={pt['q_len']} call {pt['t_median_us']:.2f} us")
    torch.cuda.synchronize()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-tail", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--sweep-seeds", type=int, default=5)
    ap.add_argument("--no-depth-sweep", action="store_true")
    ap.add_argument("--no-mixed", action="store_true")
    ap.add_argument("--no-spec-step", action="store_true")
    ap.add_argument("--no-groups", action="store_true",
                    help="skip the bulk sequences at GQA group sizes 8 and 16")
    ap.add_argument("--no-shards", action="store_true",
                    help="skip the per-GPU shares of two-way tensor-parallel replicas")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the read-only ceiling kernels timed beside each workload")
    ap.add_argument("--only", choices=list(WORKLOADS), help="time one workload only (profiling)")
    ap.add_argument("--small-trace", action="store_true",
                    help="run the concurrency sweep at 1-8 sequences (4-token verify, then one-token "
                         "decode) for a kernel trace, and print what ran; --steps sets its timed calls")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="with --only: first copy BYTES with the library's plain copy kernel, "
                         "so hardware byte counters can be scaled against a known transfer")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the attention path has no cross-GPU step; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_22788_amd import binding
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    if args.small_trace:
        print(json.dumps({"small_batch_trace": small_batch_trace(args.steps)}), flush=True)
        return

    if args.only:
        if args.calibrate_copy:
            n = args.calibrate_copy // 16 * 16
            src = torch.empty(n, dtype=torch.uint8, device="cuda")
            dst = torch.empty(n, dtype=torch.uint8, device="cuda")
            binding.copy_bytes(dst, src)
            torch.cuda.synchronize()
            del src, dst
        r = time_workload(args.only, args.steps, args.warmup, MIN_WARMUP_MS, ceiling=not args.no_ceiling)
        r.pop("wl"), r.pop("out_f64")
        print(json.dumps(r), flush=True)
        return

    bulk = time_workload("bulk", args.steps, args.warmup, ceiling=not args.no_ceiling, stream_ceiling=True)

    def guarded(what, fn):
        # A failing side measurement is reported in its field; the headline
        # line is still printed.
        try:
            return fn()
        except Exception as e:   # noqa: BLE001
            log(f"[bench] {what} failed: {e!r}")
            traceback.print_exc(file=sys.stderr)
            return {"error": repr(e)}

    tail_runs = {}

    def tail_one(name):
        r = time_workload(name, args.steps, args.warmup, MIN_WARMUP_MS, ceiling=not args.no_ceiling)
        tail_runs[name] = r
        out = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()
               if k not in ("wl", "out_f64")}
        out["hbm_frac"] = round(r["kv_gbps"] / PEAK_GBPS, 4)
        out["kernel"] = KERNELS[name]
        out["kernel_frac"] = round(r["kernel_gbps"] / PEAK_GBPS, 4)
        out["traffic"] = measured_traffic(name)
        return out

    tail = {}
    if not args.no_tail:
        for name in ("mtp", "dflash"):
            tail[name] = guarded(name, lambda: tail_one(name))
    groups = None
    if not args.no_groups:
        # the bulk sequences at larger GQA group sizes (more query rows per KV
        # byte: G flop per byte at q_len 1), and G = 8 verifying 4 tokens
        groups = {}
        for Hq, Hkv, ql in ((32, 4, 1), (64, 4, 1), (32, 4, 4)):
            key = f"bulk_g{Hq // Hkv}_q{ql}"

            def group_one(Hq=Hq, Hkv=Hkv, ql=ql, key=key):
                from paper_2608_22788_amd import synth
                cfg = dict(synth.CONFIGS["bulk"], Hq=Hq, Hkv=Hkv, q_len=ql)
                r = time_workload(key, args.steps, args.warmup, MIN_WARMUP_MS, ceiling=not args.no_ceiling,
                                  cfg=cfg)
                r.pop("wl"), r.pop("out_f64")
                out = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()}
                out["heads"] = f"{Hq} q / {Hkv} kv"
                out["q_len"] = ql
                out["hbm_frac"] = round(r["kv_gbps"] / PEAK_GBPS, 4)
                out["kernel_frac"] = round(r["kernel_gbps"] / PEAK_GBPS, 4)
                return out
            groups[key] = guarded(key, group_one)
    shards = None
    if not args.no_shards:
        # one GPU's share of a TP2 replica (KV heads split 8 -> 4 per GPU;
        # attention needs no exchange, so this is the whole per-GPU step)
        shards = {}
        for parent in ("bulk", "dflash"):
            def shard_one(parent=parent):
                r = time_workload(parent + "_tp2", args.steps, args.warmup, MIN_WARMUP_MS,
                                  ceiling=not args.no_ceiling, cfg=tp2_share(parent))
                r.pop("wl"), r.pop("out_f64")
                out = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()}
                out["heads"] = "16 q / 4 kv"
                out["hbm_frac"] = round(r["kv_gbps"] / PEAK_GBPS, 4)
                out["kernel"] = KERNELS[parent]
                out["kernel_frac"] = round(r["kernel_gbps"] / PEAK_GBPS, 4)
                return out
            shards[parent + "_tp2"] = guarded(parent + " tp2 share", shard_one)
    sweep = []
    decode_small = None
    model = None
    if not args.no_sweep:
        log(f"[bench] concurrency sweep ({args.sweep_seeds} seeds)")
        sweep = guarded("sweep", lambda: sweep_summary(
            binding.concurrency_sweep(seeds=args.sweep_seeds, warmup=20, iters=100)))
        # the batch sizes the sweep verifies at, decoding one token instead:
        # with the sweep's q_len 1 points this is the bulk pool's tau(b)
        decode_small = guarded("decode sweep", lambda: sweep_summary(
            binding.concurrency_sweep(batches=(1, 2, 4, 8), seeds=args.sweep_seeds, warmup=20, iters=100,
                                      verify_max_batch=0)))
        if isinstance(sweep, list) and isinstance(decode_small, list):
            model = guarded("makespan model", lambda: makespan_model(sweep + decode_small, bulk["wl"]))
    mixed = None
    if not args.no_mixed:
        log("[bench] ragged mixed batch and graph replay")
        mixed = guarded("mixed batch", mixed_and_graph)
    spec = None
    if not args.no_spec_step:
        log("[bench] speculative verify step: KV append, attention, acceptance")
        spec = guarded("spec step", spec_step)
    depth = None
    if not args.no_depth_sweep:
        log("[bench] draft-depth sweep (q_len 1..6 at every batch size, seed 0)")
        depth = guarded("depth sweep", depth_sweep)
    cpu = None if args.no_cpu_baseline else guarded("cpu baseline", lambda: cpu_baseline(bulk, tail_runs))

    achieved = bulk["kernel_gbps"]
    if cpu and "value" in cpu:
        cpu["gpu_speedup"] = round(bulk["kv_gbps"] / cpu["value"], 1)
    traffic = measured_traffic("bulk")
    line = {
        "metric": "decode-attn KV GB/s (% of HBM peak) and tokens/s vs concurrency, bulk+tail",
        "value": round(bulk["kv_gbps"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(bulk["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOADS["bulk"], "global_batch": 256, "q_len": 1,
                   "kv_bytes_per_step": bulk["kv_bytes"], "kv_pools_rotated": bulk["n_pools"],
                   "parallelism": "single GPU"},
        "hbm_frac": round(bulk["kv_gbps"] / PEAK_GBPS, 4),
        "tokens_per_s": round(bulk["tokens_per_s"]),
        "parity": cpu.get("parity") if isinstance(cpu, dict) else None,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_GBPS, 4), "traffic": traffic,
                     "kernel": KERNELS["bulk"],
                     "kernel_ms_mean": round(bulk["kernel_ms_mean"], 5),
                     "kernel_ms_median": round(bulk["kernel_ms_median"], 5),
                     "kernel_ms_p10": round(bulk["kernel_ms_p10"], 5),
                     "kernel_ms_p90": round(bulk["kernel_ms_p90"], 5),
                     "alg_bytes_per_launch": bulk["alg_bytes"], "plan": bulk["plan"]},
        "cpu_baseline": cpu,
        "ceiling": ceiling_summary(bulk),
        "paper_context": {"routing_only_speedup_max": 1.67, "routing_plus_speculation_speedup_max": 2.59,
                          "hardware": "one node of 8x NVIDIA H100, vLLM (paper Sec. 4.2, App. A.1)",
                          "note": "end-to-end rollout speedups over uniform group routing; context only, "
                                  "not this path's metric and not a target"},
        "tail": tail,
        "tp2_shares": shards,
        "group_sizes": groups,
        "sweep": sweep,
        "sweep_decode_small_batches": decode_small if not args.no_sweep else None,
        "makespan_model": model,
        "mixed_batch": mixed,
        "spec_step": spec,
        "depth_sweep": depth,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
