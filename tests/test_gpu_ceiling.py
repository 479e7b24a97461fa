"""The two read-only ceiling kernels on the GPU, through the C ABI.  Each lane
writes the XOR of the 32-bit words it loaded, so the XOR of the whole sink
must equal the XOR of exactly the words the kernel is meant to read: every
word of the buffer (stream read), or every word of the K and V blocks of the
pages an attention call over the same arguments streams (page gather).  A
page read twice or skipped changes the XOR (barring a block whose own XOR is
zero, which random values make vanishingly unlikely).  Bit-exact."""
import numpy as np
import pytest

from paper_2608_22788_amd import synth
from gpu_util import say

pytestmark = pytest.mark.gpu


def xor_all(words: np.ndarray) -> int:
    return int(np.bitwise_xor.reduce(words.reshape(-1).view(np.uint32))) if words.size else 0


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (64 << 20) + 272])
def test_stream_read_reads_every_word_once(nbytes):
    import torch
    from paper_2608_22788_amd import binding
    g = torch.Generator(device="cpu").manual_seed(nbytes)
    host = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, generator=g)
    src = host.cuda()
    sink = torch.zeros((2 << 20) // 4, dtype=torch.int32, device="cuda")
    say(f"stream read {nbytes} B")
    binding.stream_read(src, sink)
    torch.cuda.synchronize()
    assert xor_all(sink.cpu().numpy()) == xor_all(host.numpy())


def expected_gather_xor(wl, k, v) -> int:
    acc = 0
    for b in range(wl.B):
        if wl.q_lens[b] == 0 or wl.ctx_lens[b] == 0:
            continue
        n = (int(wl.ctx_lens[b]) + 15) // 16
        pages = wl.page_table[b, :n]
        acc ^= xor_all(np.ascontiguousarray(k[pages])) ^ xor_all(np.ascontiguousarray(v[pages]))
    return acc


@pytest.mark.parametrize("D,Hkv,ctx,ql,workers", [
    (128, 8, [37, 16, 1, 300, 129, 64, 5000], [1, 4, 1, 16, 0, 3, 1], 0),
    (128, 8, [37, 16, 1, 300, 129, 64, 5000], [1, 4, 1, 16, 0, 3, 1], 7),
    (64, 2, [17, 2048, 33], [1, 1, 2], 0),
    (64, 2, [17, 2048, 33], [1, 1, 2], 5000),        # more workers than pages
])
def test_page_gather_reads_each_referenced_page_once(D, Hkv, ctx, ql, workers):
    import torch
    from paper_2608_22788_amd import binding, device
    cfg = dict(B=len(ctx), Hq=Hkv, Hkv=Hkv, D=D, q_len=1, lengths=("uniform", 1, 1), scale=1.0)
    wl = synth.make_workload("gather", seed=D + Hkv, cfg=cfg, ctx_lens=ctx, q_lens=ql, spare_pages=3)
    t = device.upload(wl, values="device")
    W = workers or 1024
    sink = torch.zeros(W * 64, dtype=torch.int32, device="cuda")
    say(f"page gather D={D} Hkv={Hkv} lens={ctx} q={ql} workers={workers}")
    binding.page_gather_read(t["k_pages"], t["v_pages"], t["page_table"], t["ctx_lens"], t["q_lens"], sink,
                             max_ctx_len=wl.max_ctx_len, num_workers=workers)
    torch.cuda.synchronize()
    k = t["k_pages"].view(torch.int16).cpu().numpy()
    v = t["v_pages"].view(torch.int16).cpu().numpy()
    assert xor_all(sink.cpu().numpy()) == expected_gather_xor(wl, k, v)


def test_page_gather_rejects_a_small_sink():
    import torch
    from paper_2608_22788_amd import binding, device
    cfg = dict(B=1, Hq=2, Hkv=2, D=64, q_len=1, lengths=("uniform", 1, 1), scale=1.0)
    wl = synth.make_workload("gather", seed=0, cfg=cfg, ctx_lens=[40], q_lens=[1])
    t = device.upload(wl, values="device")
    sink = torch.zeros(64 * 10, dtype=torch.int32, device="cuda")
    with pytest.raises(binding.TsError, match="sink"):
        binding.page_gather_read(t["k_pages"], t["v_pages"], t["page_table"], t["ctx_lens"], t["q_lens"], sink,
                                 num_workers=11)
