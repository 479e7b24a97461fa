"""Device-resident inputs for libtsattn calls (test and benchmark plumbing).

Uploads a ``synth.Workload`` into torch CUDA tensors.  Values come either
from the host generator (exact copies of what the oracle sees) or from the
library's device fill, which implements the same SplitMix64 / Box-Muller
definition on the GPU and is checked bit for bit against the host side.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import synth

CANARY = 0x5A5A          # bf16 bit pattern written around and into unused outputs
GUARD = 64               # guard elements before and after `out`


def _bf16(t_u16: np.ndarray, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(t_u16).view(np.int16)).to(device).view(torch.bfloat16)


def upload(wl: synth.Workload, values: str = "host", device: str = "cuda") -> Dict[str, object]:
    """Tensors q, k_pages, v_pages, page_table, ctx_lens, q_lens, out (with
    canary-filled guard bands in ``out_full``) for workload ``wl``."""
    import torch
    from . import binding
    B, Qmax, Hq, D = wl.B, wl.Qmax, wl.Hq, wl.D
    shp_q = (B, Qmax, Hq, D)
    shp_kv = (wl.num_pages, wl.Hkv, wl.P, D)
    if values == "host":
        q = _bf16(wl.q_values(), device)
        k = _bf16(wl.k_pages(), device)
        v = _bf16(wl.v_pages(), device)
    elif values == "device":
        if not (np.array_equal(wl.value_page, np.arange(wl.num_pages)) and
                np.array_equal(wl.q_seq, np.arange(B))):
            raise ValueError("device fill needs a workload with its own page and q numbering")
        q = torch.empty(shp_q, dtype=torch.bfloat16, device=device)
        k = torch.empty(shp_kv, dtype=torch.bfloat16, device=device)
        v = torch.empty(shp_kv, dtype=torch.bfloat16, device=device)
        binding.synth_fill(q, wl.seed, synth.S_Q)
        binding.synth_fill(k, wl.seed, synth.S_K)
        binding.synth_fill(v, wl.seed, synth.S_V)
        if wl.poison:
            used = torch.from_numpy(wl.used_slots()).to(device)
            bad = ~used[:, None, :, None].expand(shp_kv)
            k.view(torch.int16)[bad] = synth.BF16_NAN
            v.view(torch.int16)[bad] = synth.BF16_NAN
    else:
        raise ValueError(values)
    n = B * Qmax * Hq * D
    out_full = torch.full((n + 2 * GUARD,), CANARY, dtype=torch.int16, device=device)
    out = out_full[GUARD:GUARD + n].view(torch.bfloat16).view(shp_q)
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)  # noqa: E731
    return dict(q=q, k_pages=k, v_pages=v, page_table=i32(wl.page_table), ctx_lens=i32(wl.ctx_lens),
                q_lens=i32(wl.q_lens), out=out, out_full=out_full)


def run(wl: synth.Workload, t: Dict[str, object], num_workers: int = 0, workspace=None, events=None,
        variant: int = 0):
    from . import binding
    return binding.decode_attn(t["q"], t["k_pages"], t["v_pages"], t["page_table"], t["ctx_lens"],
                               t["q_lens"], t["out"], wl.scale, workspace=workspace,
                               max_ctx_len=max(1, wl.max_ctx_len), num_workers=num_workers,
                               events=events, variant=variant)


def out_as_f64(t: Dict[str, object]) -> np.ndarray:
    """``out`` widened to float64 (bf16 bit patterns -> float)."""
    raw = t["out"].view(__import__("torch").int16).cpu().numpy().view(np.uint16)
    return synth.bf16_bits_to_f32(raw).astype(np.float64)
