"""ts_decode_attn_noalloc, the entry point for callers that cannot allocate,
through the C ABI: two calls in a row (the second with a smaller input) give
bit for bit what ts_decode_attn gives with its own workspace, and both are
within the parity bar of the float64 oracle; a shape beyond the static
scratch is rejected before anything is launched."""
import numpy as np
import pytest

from paper_2608_22788_amd import synth

from gpu_util import assert_parity, canary_ok, oracle_out, say

pytestmark = pytest.mark.gpu


def cfg(Hq, Hkv, D, q_len):
    return dict(B=1, Hq=Hq, Hkv=Hkv, D=D, q_len=q_len, lengths=("uniform", 1, 1), scale=1.0 / np.sqrt(D))


def check_call(wl, orc):
    import torch
    from paper_2608_22788_amd import binding, device
    t = device.upload(wl, values="host")
    ref = oracle_out(orc, wl)
    say(f"no-alloc {wl.name}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Qmax={wl.Qmax}")
    device.run(wl, t)                                   # ts_decode_attn, own workspace
    torch.cuda.synchronize()
    want = t["out"].clone()
    t["out_full"].fill_(device.CANARY)
    torch.cuda.synchronize()
    binding.decode_attn_noalloc(t["q"], t["k_pages"], t["v_pages"], t["page_table"], t["ctx_lens"],
                                t["q_lens"], t["out"], wl.scale, max_ctx_len=wl.max_ctx_len)
    torch.cuda.synchronize()
    canary_ok(t, wl)
    assert torch.equal(t["out"].view(torch.int16), want.view(torch.int16)), f"{wl.name}: differs"
    assert_parity(device.out_as_f64(t), ref, f"no-alloc {wl.name}")


def test_noalloc_matches_the_workspace_entry_point(orc):
    rng = np.random.default_rng(17)
    # 300 x 8 units: splits combined in the streaming kernel (counters in use)
    big = synth.make_workload("noalloc_big", seed=17, cfg=cfg(32, 8, 128, 1),
                              ctx_lens=rng.integers(40, 1500, size=300).tolist(), q_lens=[1] * 300,
                              poison=True, spare_pages=1)
    # then a smaller call: long verify contexts, splits combined by the merge kernel
    small = synth.make_workload("noalloc_small", seed=18, cfg=cfg(32, 8, 128, 4),
                                ctx_lens=[9000, 70, 2500], q_lens=[4, 2, 4], poison=True, spare_pages=1)
    check_call(big, orc)
    check_call(small, orc)


def test_noalloc_rejects_a_shape_beyond_its_scratch():
    import torch
    from paper_2608_22788_amd import binding, device
    wl = synth.make_workload("noalloc_huge", seed=19, cfg=cfg(64, 4, 128, 1), ctx_lens=[100, 200], q_lens=[1, 1])
    t = device.upload(wl)
    # 4,096 workers x 2 slots x 16 rows x 128 dims x 4 bytes = 64 MiB of partials
    shape = binding.shape_of(t["q"], t["k_pages"], t["page_table"], wl.max_ctx_len, 4096, 0)
    assert binding.workspace_size(shape) > (48 << 20)
    t["out_full"].fill_(device.CANARY)
    torch.cuda.synchronize()
    with pytest.raises(binding.TsError) as err:
        binding.decode_attn_noalloc(t["q"], t["k_pages"], t["v_pages"], t["page_table"], t["ctx_lens"],
                                    t["q_lens"], t["out"], wl.scale, max_ctx_len=wl.max_ctx_len,
                                    num_workers=4096)
    assert err.value.status == -3 and "scratch" in str(err.value)
    torch.cuda.synchronize()
    canary_ok(t, wl)
    assert (t["out_full"].cpu().numpy() == device.CANARY).all()     # nothing was launched
