"""Runtime contracts of the C ABI on the GPU: a call can be captured into a
HIP graph and replayed, and TS_DEBUG=1 turns violated device-side
preconditions into TS_ERR_SHAPE (a workspace whose counters are not zero
into TS_ERR_WORKSPACE) before any attention kernel runs."""
import os
import subprocess
import sys
import textwrap

import numpy as np
import pytest

from paper_2608_22788_amd import synth

from gpu_util import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def small_cfg(Hq, Hkv, D):
    return dict(B=1, Hq=Hq, Hkv=Hkv, D=D, q_len=1, lengths=("uniform", 1, 1), scale=1.0 / np.sqrt(D))


@pytest.mark.parametrize("q_lens,ctx", [([1] * 6, [17, 300, 1000, 64, 2048, 5]),
                                         ([4, 4, 1], [100, 3000, 40]),
                                         ([16, 16], [5000, 40])])
def test_graph_capture_replays_match_eager(q_lens, ctx):
    import torch
    from paper_2608_22788_amd import binding, device
    wl = synth.make_workload("graph", seed=3, cfg=small_cfg(32, 8, 128), ctx_lens=ctx, q_lens=q_lens)
    t = device.upload(wl)
    shape = binding.shape_of(t["q"], t["k_pages"], t["page_table"], wl.max_ctx_len)
    ws = binding.new_workspace(binding.workspace_size(shape))
    device.run(wl, t, workspace=ws)                    # eager reference (and device check)
    torch.cuda.synchronize()
    ref = t["out"].clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            device.run(wl, t, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(4):
        say(f"graph replay {rep} q_lens={q_lens}")
        t["out_full"].fill_(device.CANARY)               # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(t["out"].view(torch.int16), ref.view(torch.int16)), f"replay {rep}"


DEBUG_SCRIPT = textwrap.dedent("""
    import sys, numpy as np
    sys.path.insert(0, {root!r})
    import torch
    from paper_2608_22788_amd import binding, device, synth
    cfg = dict(B=1, Hq=8, Hkv=2, D=64, q_len=1, lengths=("uniform", 1, 1), scale=0.125)
    wl = synth.make_workload("dbg", seed=1, cfg=cfg, ctx_lens=[40, 70], q_lens=[1, 1])
    t = device.upload(wl)
    device.run(wl, t)                          # valid call passes the check
    torch.cuda.synchronize()
    results = []
    bad = t["page_table"].clone(); bad[1, 2] = wl.num_pages + 5   # page id out of range
    t2 = dict(t); t2["page_table"] = bad
    try:
        device.run(wl, t2); results.append("no error")
    except binding.TsError as e:
        results.append(str(e.status) + ":" + str(e))
    lens = t["ctx_lens"].clone(); lens[0] = 0      # q_len 1 > ctx_len 0
    t3 = dict(t); t3["ctx_lens"] = lens
    try:
        device.run(wl, t3); results.append("no error")
    except binding.TsError as e:
        results.append(str(e.status) + ":" + str(e))
    # a reused workspace passes the check after every call (its counters are
    # left zero); one that was never zero-filled is reported
    ws = binding.new_workspace(8 << 20)
    for _ in range(3):
        device.run(wl, t, num_workers=7, workspace=ws)
    torch.cuda.synchronize()
    dirty = torch.full((8 << 20,), 1, dtype=torch.uint8, device="cuda")
    try:
        device.run(wl, t, workspace=dirty); results.append("no error")
    except binding.TsError as e:
        results.append(str(e.status) + ":" + str(e))
    print("RESULTS", results)
""")


def test_debug_mode_reports_bad_device_inputs():
    env = dict(os.environ, TS_DEBUG="1")
    r = subprocess.run([sys.executable, "-c", DEBUG_SCRIPT.format(root=ROOT)], capture_output=True,
                       text=True, timeout=240, env=env)
    say(r.stdout[-2000:], r.stderr[-2000:])
    assert r.returncode == 0
    line = [ln for ln in r.stdout.splitlines() if ln.startswith("RESULTS")][0]
    assert "-2:" in line.split("'")[1] and "page id" in line
    assert line.count("-2:") == 2 and "q_lens" in line
    assert line.count("-3:") == 1 and "zero-fill" in line
