"""Float64 CPU oracle for paged decode / speculative-verify attention.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product library
never does.  ``ts_oracle.c`` holds the arithmetic (plain C loops in double,
written from the textbook definition of scaled-dot-product attention with a
causal draft block; see its header); this module compiles it with gcc and
calls it through ctypes.  It imports nothing from the product package.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ts_oracle.c")
LIB = os.path.join(HERE, "libts_oracle.so")

CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared"]


def build(src: str = SRC, out: str = LIB) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    cmd = ["gcc", *CFLAGS, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_p = ctypes.c_void_p
_i = ctypes.c_int


class Oracle:
    def __init__(self, path: str = LIB):
        self.path = path
        self.lib = ctypes.CDLL(path)
        common = [_i] * 7 + [_p] * 6 + [ctypes.c_double]
        self.lib.ts_oracle_paged_attention.argtypes = common + [_p, _i]
        self.lib.ts_oracle_paged_attention.restype = None
        self.lib.ts_oracle_partial_attention.argtypes = common + [_i, _i, _p, _p, _i]
        self.lib.ts_oracle_partial_attention.restype = None
        self.lib.ts_oracle_row_weights.argtypes = common + [_i, _i, _i, _p]
        self.lib.ts_oracle_row_weights.restype = None
        self.lib.ts_oracle_lse_merge.argtypes = [_i, ctypes.c_int64, _i, _p, _p, _p]
        self.lib.ts_oracle_lse_merge.restype = None

    @staticmethod
    def _prep(q, k_pages, v_pages, page_table, ctx_lens, q_lens):
        q = np.ascontiguousarray(q, dtype=np.uint16)
        kp = np.ascontiguousarray(k_pages, dtype=np.uint16)
        vp = np.ascontiguousarray(v_pages, dtype=np.uint16)
        pt = np.ascontiguousarray(page_table, dtype=np.int32)
        cl = np.ascontiguousarray(ctx_lens, dtype=np.int32)
        ql = np.ascontiguousarray(q_lens, dtype=np.int32)
        B, Qmax, Hq, D = q.shape
        NP, Hkv, P, D2 = kp.shape
        assert D2 == D and vp.shape == kp.shape and pt.shape[0] == B
        assert cl.shape == (B,) and ql.shape == (B,) and Hq % Hkv == 0
        assert (ql <= cl).all() and (ql <= Qmax).all() and (ql >= 0).all()
        assert (((cl.astype(np.int64) + P - 1) // P) <= pt.shape[1]).all()
        dims = (B, Hq, Hkv, D, P, Qmax, pt.shape[1])
        arrs = (q, kp, vp, pt, cl, ql)
        return dims, arrs

    @staticmethod
    def _ptrs(arrs):
        return [a.ctypes.data_as(_p) for a in arrs]

    def attention(self, q, k_pages, v_pages, page_table, ctx_lens, q_lens, scale: float,
                  nthreads: int = 0) -> np.ndarray:
        """Full attention; rows i >= q_lens[b] come back as NaN."""
        dims, arrs = self._prep(q, k_pages, v_pages, page_table, ctx_lens, q_lens)
        out = np.full(arrs[0].shape, np.nan, dtype=np.float64)
        self.lib.ts_oracle_paged_attention(*dims, *self._ptrs(arrs), float(scale),
                                           out.ctypes.data_as(_p), int(nthreads))
        return out

    def partial(self, q, k_pages, v_pages, page_table, ctx_lens, q_lens, scale: float,
                t_begin: int, t_end: int, nthreads: int = 0):
        """Normalised output and natural-log LSE over keys [t_begin, t_end)."""
        dims, arrs = self._prep(q, k_pages, v_pages, page_table, ctx_lens, q_lens)
        out = np.full(arrs[0].shape, np.nan, dtype=np.float64)
        lse = np.full(arrs[0].shape[:3], np.nan, dtype=np.float64)
        self.lib.ts_oracle_partial_attention(*dims, *self._ptrs(arrs), float(scale), int(t_begin),
                                             int(t_end), out.ctypes.data_as(_p),
                                             lse.ctypes.data_as(_p), int(nthreads))
        return out, lse

    def row_weights(self, q, k_pages, v_pages, page_table, ctx_lens, q_lens, scale: float,
                    b: int, i: int, h: int) -> np.ndarray:
        dims, arrs = self._prep(q, k_pages, v_pages, page_table, ctx_lens, q_lens)
        w = np.zeros(int(arrs[4][b]), dtype=np.float64)
        self.lib.ts_oracle_row_weights(*dims, *self._ptrs(arrs), float(scale), int(b), int(i),
                                       int(h), w.ctypes.data_as(_p))
        return w

    def lse_merge(self, o_parts: np.ndarray, lse_parts: np.ndarray) -> np.ndarray:
        """o_parts [S, R, D], lse_parts [S, R] -> merged [R, D]."""
        o = np.ascontiguousarray(o_parts, dtype=np.float64)
        l = np.ascontiguousarray(lse_parts, dtype=np.float64)
        S, R, D = o.shape
        out = np.zeros((R, D), dtype=np.float64)
        self.lib.ts_oracle_lse_merge(S, R, D, o.ctypes.data_as(_p), l.ctypes.data_as(_p),
                                     out.ctypes.data_as(_p))
        return out


_default: Optional[Oracle] = None


def load(path: Optional[str] = None) -> Oracle:
    """The oracle compiled from ``ts_oracle.c`` (built on first use)."""
    global _default
    if path is not None:
        return Oracle(path)
    if _default is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _default = Oracle(LIB)
    return _default
