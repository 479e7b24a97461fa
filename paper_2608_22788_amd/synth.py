"""Seeded synthetic workloads for paged decode / verify attention.

This module is the single source of inputs for both sides of every parity
check: it draws context lengths, draft-block lengths, page tables and the
bf16 values of q, K and V.  It holds none of the attention arithmetic.

The paper runs its rollouts on real prompt sets and model weights (Sec. 4.1
and App. A.1) that are not available here; these synthetic inputs stand in
for them with the batch sizes, head shapes, context-length distributions and
draft depths of the five workloads listed in ``CONFIGS``.

Randomness
----------
Every random number is a counter-based draw from SplitMix64 (Steele, Lea and
Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014), used
in its published form: the n-th output (n = 0, 1, ...) for a 64-bit state
``key`` is ``mix64(key + (n + 1) * 0x9E3779B97F4A7C15 mod 2^64)`` with
``mix64`` the variant-13 finaliser.  A draw is therefore addressed by
``(seed, stream, index)`` and any subset can be regenerated on its own, which
is what lets a test rebuild only the pages of a few sampled sequences of a
multi-gigabyte pool.  The library's device fill and its host sweep generator
implement the same definitions independently; tests check that they agree.

* ``key(seed, stream) = mix64((seed << 8) + stream)``.
* uniform integer in ``[lo, hi]``: ``lo + ((z >> 32) * (hi - lo + 1)) >> 32``.
* unit uniforms: ``u1 = ((z >> 32) + 1) / 2^32`` in (0, 1],
  ``u2 = (z & 0xffffffff) / 2^32`` in [0, 1).
* standard normal (Box-Muller, cosine branch), in float64:
  ``sqrt(-2 ln u1) * cos(u2 * 6.283185307179586)``.
* bf16 value: the float64 normal rounded to float32 (round to nearest even),
  then float32 rounded to bf16 (round to nearest even).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess
from typing import Dict, Optional, Sequence

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1
PAGE_SIZE = 16

# stream identifiers (one independent SplitMix64 stream per purpose)
S_LEN_A = 1      # first length component (uniform part / prompt)
S_LEN_B = 2      # second length component (lognormal or Pareto response)
S_PERM = 3       # page permutation keys
S_Q = 4          # query values
S_K = 5          # key-page values
S_V = 6          # value-page values

BF16_NAN = 0x7FC0

_U64 = np.uint64


def _mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> _U64(30))) * _U64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> _U64(27))) * _U64(0x94D049BB133111EB)
    return z ^ (z >> _U64(31))


def mix64_int(z: int) -> int:
    """Scalar ``mix64`` on Python integers (used for keys and tests)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def stream_key(seed: int, stream: int) -> int:
    return mix64_int(((seed & ((1 << 56) - 1)) << 8) + stream)


def draws(seed: int, stream: int, index) -> np.ndarray:
    """SplitMix64 outputs number ``index`` (array) of stream ``(seed, stream)``."""
    idx = np.asarray(index, dtype=np.uint64)
    with np.errstate(over="ignore"):
        x = _U64(stream_key(seed, stream)) + (idx + _U64(1)) * _U64(GAMMA)
        return _mix64(x)


def uniform_int(z: np.ndarray, lo: int, hi: int) -> np.ndarray:
    n = _U64(hi - lo + 1)
    with np.errstate(over="ignore"):
        return (lo + (((z >> _U64(32)) * n) >> _U64(32)).astype(np.int64)).astype(np.int64)


def unit_uniforms(z: np.ndarray):
    hi = (z >> _U64(32)).astype(np.float64)
    lo = (z & _U64(0xFFFFFFFF)).astype(np.float64)
    return (hi + 1.0) * 2.0 ** -32, lo * 2.0 ** -32


def normal_f64(z: np.ndarray) -> np.ndarray:
    u1, u2 = unit_uniforms(z)
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(u2 * 6.283185307179586)


def f32_to_bf16_bits(f: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern, round to nearest even (NaN kept quiet)."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = (u + _U64(0x7FFF) + ((u >> _U64(16)) & _U64(1))) >> _U64(16)
    out = r.astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(seed: int, stream: int, index) -> np.ndarray:
    """bf16 bit patterns of N(0,1) draws number ``index`` of a stream."""
    x = normal_f64(draws(seed, stream, index))
    return f32_to_bf16_bits(x.astype(np.float32))


def normal_bf16_range_numpy(seed: int, stream: int, start: int, count: int,
                            chunk: int = 1 << 22) -> np.ndarray:
    out = np.empty(count, dtype=np.uint16)
    for s in range(0, count, chunk):
        n = min(chunk, count - s)
        out[s:s + n] = normal_bf16(seed, stream, np.arange(start + s, start + s + n, dtype=np.uint64))
    return out


_HOST_SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "synth_host.c")
_HOST_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtssynth.so")
_host = None


def build_host(out: str = _HOST_LIB) -> str:
    """Compile the OpenMP C version of the value generator (gcc)."""
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
                    "-shared", _HOST_SRC, "-o", out + ".tmp", "-lm"], check=True)
    os.replace(out + ".tmp", out)
    return out


def _host_lib():
    global _host
    if _host is None and os.path.exists(_HOST_LIB):
        lib = ctypes.CDLL(_HOST_LIB)
        lib.ts_synth_normal_bf16_host.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                                  ctypes.c_int64, ctypes.c_void_p]
        lib.ts_synth_normal_bf16_host.restype = None
        _host = lib
    return _host


def normal_bf16_range(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """bf16 bits of draws [start, start + count) of a stream (C if built)."""
    lib = _host_lib()
    if lib is None:
        return normal_bf16_range_numpy(seed, stream, start, count)
    out = np.empty(count, dtype=np.uint16)
    if count:
        lib.ts_synth_normal_bf16_host(seed, stream, start, count, out.ctypes.data)
    return out


# ---------------------------------------------------------------------------
# context-length distributions
# ---------------------------------------------------------------------------

def lengths_uniform(seed: int, B: int, lo: int, hi: int) -> np.ndarray:
    return uniform_int(draws(seed, S_LEN_A, np.arange(B)), lo, hi)


def lengths_bulk(seed: int, B: int) -> np.ndarray:
    """Prompt U{256..1024} plus response min(rint(2048 exp(0.8 Z)), 16384).

    The response cap equals the paper's maximum response length (App. A.1,
    shared rollout sampling table); the lognormal body (median 2048,
    sigma 0.8) is a synthetic stand-in for the real response-length traces.
    """
    prompt = uniform_int(draws(seed, S_LEN_A, np.arange(B)), 256, 1024)
    z = normal_f64(draws(seed, S_LEN_B, np.arange(B)))
    resp = np.minimum(np.rint(2048.0 * np.exp(0.8 * z)), 16384.0).astype(np.int64)
    return prompt + resp


def lengths_sweep(seed: int, B: int) -> np.ndarray:
    """512 + min(floor(1024 u^(-1/1.5)), 65536): a Pareto(x_min=1024, alpha=1.5)
    response by inverse transform, u in (0, 1]."""
    u1, _ = unit_uniforms(draws(seed, S_LEN_B, np.arange(B)))
    resp = np.minimum(np.floor(1024.0 * np.power(u1, -1.0 / 1.5)), 65536.0).astype(np.int64)
    return 512 + resp


# ---------------------------------------------------------------------------
# workload configurations
# ---------------------------------------------------------------------------

CONFIGS: Dict[str, dict] = {
    # tiny decode: correctness only
    "tiny": dict(B=4, Hq=8, Hkv=2, D=64, q_len=1, lengths=("uniform", 16, 256),
                 scale=1.0 / math.sqrt(64.0)),
    # bulk pool: high concurrency, one query token per sequence
    "bulk": dict(B=256, Hq=32, Hkv=8, D=128, q_len=1, lengths=("bulk",),
                 scale=1.0 / math.sqrt(128.0)),
    # tail pool, multi-token-prediction verify: 1 + 3 drafts
    "mtp": dict(B=8, Hq=32, Hkv=8, D=128, q_len=4, lengths=("uniform", 16384, 65536),
                scale=1.0 / math.sqrt(128.0)),
    # tail pool, block-draft verify: 1 + 15 drafts
    "dflash": dict(B=4, Hq=32, Hkv=8, D=128, q_len=16, lengths=("uniform", 32768, 98304),
                   scale=1.0 / math.sqrt(128.0)),
}

SWEEP_BATCHES = (1, 2, 4, 8, 16, 32, 64, 128, 256, 512)


def sweep_q_len(B: int) -> int:
    return 4 if B <= 8 else 1


def sweep_config(B: int) -> dict:
    return dict(B=B, Hq=32, Hkv=8, D=128, q_len=sweep_q_len(B), lengths=("sweep",),
                scale=1.0 / math.sqrt(128.0))


def draw_lengths(cfg: dict, seed: int) -> np.ndarray:
    kind = cfg["lengths"][0]
    B = cfg["B"]
    if kind == "uniform":
        return lengths_uniform(seed, B, cfg["lengths"][1], cfg["lengths"][2])
    if kind == "bulk":
        return lengths_bulk(seed, B)
    if kind == "sweep":
        return lengths_sweep(seed, B)
    raise ValueError(kind)


def permutation(seed: int, n: int) -> np.ndarray:
    """Uniform random permutation of [0, n): stable argsort of SplitMix64 keys."""
    keys = draws(seed, S_PERM, np.arange(n, dtype=np.uint64))
    return np.argsort(keys, kind="stable").astype(np.int64)


@dataclasses.dataclass
class Workload:
    """Host description of one paged-attention call.

    Layouts (all C-contiguous):
      q, out       [B, Qmax, Hq, D]           bf16
      k/v pages    [num_pages, Hkv, P, D]     bf16
      page_table   [B, max_pages_per_seq]     int32
      ctx_lens, q_lens [B]                    int32
    ``ctx_lens[b]`` counts the draft tokens, whose keys and values are already
    in the pages; row i of sequence b sits at absolute position L - Q + i.
    Values are addressed by *physical* page id ``value_page[p]`` so that a
    compacted sub-workload regenerates exactly the values of its parent.
    """
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    P: int
    Qmax: int
    scale: float
    seed: int
    ctx_lens: np.ndarray
    q_lens: np.ndarray
    page_table: np.ndarray
    num_pages: int
    value_page: np.ndarray      # [num_pages] page id used to address values
    q_seq: np.ndarray           # [B] sequence index used to address q values
    q_batch: int                # batch size of the parent q tensor
    poison: bool = False
    spare_pages: int = 0

    @property
    def page_elems(self) -> int:
        return self.Hkv * self.P * self.D

    @property
    def max_pages(self) -> int:
        return self.page_table.shape[1]

    @property
    def max_ctx_len(self) -> int:
        return int(self.ctx_lens.max()) if self.B else 0

    def kv_bytes(self) -> int:
        """Algorithmic K+V bytes of one call: every context token's key and
        value rows of every KV head, read once."""
        return int(self.ctx_lens.astype(np.int64).sum()) * self.Hkv * self.D * 2 * 2

    def algorithmic_bytes(self) -> int:
        qtok = int(self.q_lens.astype(np.int64).sum())
        pages = int(((self.ctx_lens.astype(np.int64) + self.P - 1) // self.P).sum())
        return self.kv_bytes() + qtok * self.Hq * self.D * 2 * 2 + pages * 4 + self.B * 8

    def flops(self) -> int:
        L = self.ctx_lens.astype(np.int64)
        Q = self.q_lens.astype(np.int64)
        vis = (Q * (L - Q) + Q * (Q + 1) // 2).sum()
        return int(4 * self.D * self.Hq * vis)

    # --- values ------------------------------------------------------------
    def q_values(self) -> np.ndarray:
        per_seq = self.Qmax * self.Hq * self.D
        out = np.empty((self.B, per_seq), dtype=np.uint16)
        for i, s in enumerate(self.q_seq):
            out[i] = normal_bf16_range(self.seed, S_Q, int(s) * per_seq, per_seq)
        return out.reshape(self.B, self.Qmax, self.Hq, self.D)

    def _pool(self, stream: int) -> np.ndarray:
        pe = self.page_elems
        out = np.empty((self.num_pages, pe), dtype=np.uint16)
        vp = self.value_page
        # contiguous runs of value-page ids are generated in one call
        p = 0
        while p < self.num_pages:
            r = p
            while r + 1 < self.num_pages and vp[r + 1] == vp[r] + 1:
                r += 1
            n = r - p + 1
            out[p:r + 1] = normal_bf16_range(self.seed, stream, int(vp[p]) * pe, n * pe).reshape(n, pe)
            p = r + 1
        out = out.reshape(self.num_pages, self.Hkv, self.P, self.D)
        if self.poison:
            self._apply_poison(out)
        return out

    def k_pages(self) -> np.ndarray:
        return self._pool(S_K)

    def v_pages(self) -> np.ndarray:
        return self._pool(S_V)

    def used_slots(self) -> np.ndarray:
        """Boolean [num_pages, P]: slot holds a context token of some sequence."""
        used = np.zeros((self.num_pages, self.P), dtype=bool)
        for b in range(self.B):
            L = int(self.ctx_lens[b])
            n = (L + self.P - 1) // self.P
            for j in range(n):
                p = int(self.page_table[b, j])
                used[p, :min(self.P, L - j * self.P)] = True
        return used

    def _apply_poison(self, pool: np.ndarray) -> None:
        used = self.used_slots()
        pool[~used[:, None, :, None].repeat(self.Hkv, 1).repeat(self.D, 3)] = BF16_NAN

    def subset(self, seqs: Sequence[int]) -> "Workload":
        """Sub-workload of the given sequences, pages compacted, values kept."""
        seqs = [int(s) for s in seqs]
        lens = self.ctx_lens[seqs]
        npg = (lens.astype(np.int64) + self.P - 1) // self.P
        maxp = max(1, int(npg.max()))
        pt = np.zeros((len(seqs), maxp), dtype=np.int32)
        vpage = []
        for i, b in enumerate(seqs):
            for j in range(int(npg[i])):
                pt[i, j] = len(vpage)
                vpage.append(int(self.value_page[int(self.page_table[b, j])]))
        return Workload(self.name + "[sub]", len(seqs), self.Hq, self.Hkv, self.D, self.P,
                        self.Qmax, self.scale, self.seed, lens.astype(np.int32).copy(),
                        self.q_lens[seqs].astype(np.int32).copy(), pt, len(vpage),
                        np.asarray(vpage, dtype=np.int64), self.q_seq[seqs].copy(),
                        self.q_batch, False, 0)


def make_workload(name: str, seed: int = 0, cfg: Optional[dict] = None,
                  ctx_lens: Optional[Sequence[int]] = None,
                  q_lens: Optional[Sequence[int]] = None,
                  Qmax: Optional[int] = None, poison: bool = False,
                  spare_pages: int = 0, max_pages: Optional[int] = None) -> Workload:
    """Build a workload from a named config (or ``cfg``), optionally with
    explicit lengths.  Physical pages are a uniform random permutation."""
    if cfg is None:
        cfg = CONFIGS[name] if name in CONFIGS else sweep_config(int(name.split("_b")[-1]))
    B = cfg["B"] if ctx_lens is None else len(ctx_lens)
    L = draw_lengths(cfg, seed) if ctx_lens is None else np.asarray(ctx_lens, dtype=np.int64)
    if q_lens is None:
        Q = np.full(B, cfg["q_len"], dtype=np.int64)
    else:
        Q = np.asarray(q_lens, dtype=np.int64)
    if Qmax is None:
        Qmax = int(max(1, Q.max() if B else 1))
    P = PAGE_SIZE
    npg = (L + P - 1) // P
    total = int(npg.sum())
    maxp = int(max(1, npg.max() if B else 1)) if max_pages is None else max_pages
    perm = permutation(seed, total)
    pt = np.zeros((B, maxp), dtype=np.int32)
    off = 0
    for b in range(B):
        n = int(npg[b])
        pt[b, :n] = perm[off:off + n]
        off += n
    num_pages = total + spare_pages
    if spare_pages:
        # unreferenced table entries point at the first spare page
        for b in range(B):
            pt[b, int(npg[b]):] = total
    return Workload(name, B, cfg["Hq"], cfg["Hkv"], cfg["D"], P, Qmax, float(cfg["scale"]),
                    seed, L.astype(np.int32), Q.astype(np.int32), pt, num_pages,
                    np.arange(num_pages, dtype=np.int64), np.arange(B, dtype=np.int64), B,
                    poison, spare_pages)
