"""Thin ctypes binding of libtsattn (include/ts_attn.h).

Argument marshalling only: every step of the attention runs in the HIP
kernels of libtsattn.so.  PyTorch supplies device memory (``data_ptr()``)
and the stream (``torch.cuda.current_stream().cuda_stream``); nothing here
computes on tensors.  If the library is missing the import of this module
fails loudly; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtsattn.so")

# TS_ATTN_ABI_VERSION of the header these structures mirror: a library built
# from another version may lay its structures out differently, so loading
# one is refused.
ABI_VERSION = 4

TS_OK = 0
STATUS = {0: "TS_OK", -1: "TS_ERR_NULL", -2: "TS_ERR_SHAPE", -3: "TS_ERR_WORKSPACE",
          -4: "TS_ERR_UNSUPPORTED", -5: "TS_ERR_HIP", -6: "TS_ERR_ARG"}


class AttnShape(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_q_len", ctypes.c_int32),
                ("max_pages_per_seq", ctypes.c_int32), ("max_ctx_len", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("num_workers", ctypes.c_int32),
                ("variant", ctypes.c_int32)]


VARIANT_AUTO, VARIANT_WAVE, VARIANT_TEAM, VARIANT_VALU = 0, 1, 2, 3
COMBINE_MERGE_KERNEL, COMBINE_LAST_ARRIVER, COMBINE_IN_LAUNCH = 0, 1, 2


class AttnPlan(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int32), ("num_workers", ctypes.c_int32), ("combine", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("threads", ctypes.c_int32), ("merge_blocks", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64)]


class SweepConfig(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("num_batches", ctypes.c_int32),
                ("batches", ctypes.c_int32 * 32), ("verify_max_batch", ctypes.c_int32),
                ("verify_q_len", ctypes.c_int32), ("num_seeds", ctypes.c_int32),
                ("warmup", ctypes.c_int32), ("iters", ctypes.c_int32),
                ("min_rotation_bytes", ctypes.c_int64), ("verify_tokens_per_step", ctypes.c_double)]


class SweepPoint(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("q_len", ctypes.c_int32), ("seed", ctypes.c_int32),
                ("num_pools", ctypes.c_int32), ("sum_ctx", ctypes.c_int64),
                ("kv_bytes", ctypes.c_int64), ("t_median_us", ctypes.c_double),
                ("t_p10_us", ctypes.c_double), ("t_p90_us", ctypes.c_double),
                ("kv_gbps", ctypes.c_double), ("hbm_frac", ctypes.c_double),
                ("tokens_per_s", ctypes.c_double), ("tau_us", ctypes.c_double),
                ("gather_median_us", ctypes.c_double)]


EXPORTS = ["ts_decode_attn_workspace_size", "ts_decode_attn", "ts_decode_attn_events", "ts_decode_attn_noalloc",
           "ts_decode_attn_plan",
           "ts_concurrency_sweep", "ts_synth_fill_bf16", "ts_synth_sweep_lengths",
           "ts_synth_page_table", "ts_copy_bytes", "ts_stream_read", "ts_page_gather_read", "ts_event_create", "ts_event_destroy",
           "ts_event_record", "ts_event_elapsed_ms", "ts_status_string", "ts_last_error",
           "ts_version", "ts_tau_table", "ts_replica_time", "ts_request_shares", "ts_step_makespan",
           "ts_kv_append", "ts_spec_accept_workspace_size", "ts_spec_accept"]


def _load() -> ctypes.CDLL:
    # torch ships its own HIP runtime (libamdhip64.so.7).  Importing it first
    # makes the dynamic loader bind libtsattn to that same runtime by soname;
    # loading libtsattn first would map a second HIP runtime from /opt/rocm
    # into the process, and that instance sees no device once torch's is up.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; "
                          f"g.build()'` (needs hipcc)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64, U32, SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                 ctypes.c_uint32, ctypes.c_size_t)
    pshape = ctypes.POINTER(AttnShape)
    lib.ts_decode_attn_workspace_size.argtypes = [pshape]
    lib.ts_decode_attn_workspace_size.restype = SZ
    attn_args = [pshape, P, P, P, P, P, P, P, ctypes.c_float, P, SZ, P]
    lib.ts_decode_attn.argtypes = attn_args
    lib.ts_decode_attn.restype = ctypes.c_int
    lib.ts_decode_attn_events.argtypes = attn_args + [P, P]
    lib.ts_decode_attn_events.restype = ctypes.c_int
    lib.ts_concurrency_sweep.argtypes = [ctypes.POINTER(SweepConfig), ctypes.POINTER(SweepPoint),
                                         I32, ctypes.POINTER(I32)]
    lib.ts_concurrency_sweep.restype = ctypes.c_int
    lib.ts_synth_fill_bf16.argtypes = [P, I64, U64, U32, I64, P]
    lib.ts_synth_fill_bf16.restype = ctypes.c_int
    lib.ts_synth_sweep_lengths.argtypes = [I32, U64, P]
    lib.ts_synth_sweep_lengths.restype = ctypes.c_int
    lib.ts_synth_page_table.argtypes = [I32, P, I32, I32, U64, P]
    lib.ts_synth_page_table.restype = ctypes.c_int
    lib.ts_copy_bytes.argtypes = [P, P, SZ, P]
    lib.ts_copy_bytes.restype = ctypes.c_int
    lib.ts_stream_read.argtypes = [P, SZ, P, SZ, P]
    lib.ts_stream_read.restype = ctypes.c_int
    lib.ts_page_gather_read.argtypes = [pshape, P, P, P, P, P, P, SZ, P, P, P]
    lib.ts_page_gather_read.restype = ctypes.c_int
    lib.ts_event_create.argtypes = [ctypes.POINTER(P)]
    lib.ts_event_create.restype = ctypes.c_int
    lib.ts_event_destroy.argtypes = [P]
    lib.ts_event_destroy.restype = ctypes.c_int
    lib.ts_event_record.argtypes = [P, P]
    lib.ts_event_record.restype = ctypes.c_int
    lib.ts_event_elapsed_ms.argtypes = [P, P, ctypes.POINTER(ctypes.c_float)]
    lib.ts_event_elapsed_ms.restype = ctypes.c_int
    lib.ts_tau_table.argtypes = [P, P, I32, I32, P]
    lib.ts_tau_table.restype = ctypes.c_int
    lib.ts_replica_time.argtypes = [P, I32, P, I32, ctypes.POINTER(ctypes.c_double)]
    lib.ts_replica_time.restype = ctypes.c_int
    lib.ts_request_shares.argtypes = [P, I32, P, I32, P]
    lib.ts_request_shares.restype = ctypes.c_int
    lib.ts_step_makespan.argtypes = [P, I32, P, P, I32, I32, P, ctypes.POINTER(ctypes.c_double)]
    lib.ts_step_makespan.restype = ctypes.c_int
    lib.ts_decode_attn_noalloc.argtypes = [pshape, P, P, P, P, P, P, P, ctypes.c_float, P]
    lib.ts_decode_attn_noalloc.restype = ctypes.c_int
    lib.ts_decode_attn_plan.argtypes = [pshape, ctypes.POINTER(AttnPlan)]
    lib.ts_decode_attn_plan.restype = ctypes.c_int
    lib.ts_kv_append.argtypes = [pshape, P, P, P, P, P, P, P, P]
    lib.ts_kv_append.restype = ctypes.c_int
    lib.ts_spec_accept_workspace_size.argtypes = [I32, I32]
    lib.ts_spec_accept_workspace_size.restype = SZ
    lib.ts_spec_accept.argtypes = [I32, I32, I32, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.ts_spec_accept.restype = ctypes.c_int
    lib.ts_status_string.argtypes = [ctypes.c_int]
    lib.ts_status_string.restype = ctypes.c_char_p
    lib.ts_last_error.argtypes = []
    lib.ts_last_error.restype = ctypes.c_char_p
    lib.ts_version.argtypes = []
    lib.ts_version.restype = ctypes.c_int
    if lib.ts_version() != ABI_VERSION:
        raise ImportError(f"{LIB_PATH} has ABI version {lib.ts_version()}, this binding expects "
                          f"{ABI_VERSION}; rebuild the library")
    return lib


lib = _load()


class TsError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib.ts_last_error().decode()
        super().__init__(f"{where}: {STATUS.get(status, status)}: {msg}")


def check(status: int, where: str) -> None:
    if status != TS_OK:
        raise TsError(status, where)


def make_shape(num_seqs, num_q_heads, num_kv_heads, head_dim, max_q_len, max_pages_per_seq,
               max_ctx_len, num_pages, num_workers=0, page_size=16, variant=0) -> AttnShape:
    return AttnShape(num_seqs, num_q_heads, num_kv_heads, head_dim, page_size, max_q_len,
                     max_pages_per_seq, max_ctx_len, num_pages, num_workers, variant)


def workspace_size(shape: AttnShape) -> int:
    n = lib.ts_decode_attn_workspace_size(ctypes.byref(shape))
    if n == 0:
        raise TsError(-2, "ts_decode_attn_workspace_size")
    return int(n)


def decode_attn_plan(shape: AttnShape) -> dict:
    """What ts_decode_attn launches for `shape` on the current device
    (kernel, workers, how splits are combined, launch sizes)."""
    plan = AttnPlan()
    check(lib.ts_decode_attn_plan(ctypes.byref(shape), ctypes.byref(plan)), "ts_decode_attn_plan")
    return {f: getattr(plan, f) for f, _ in AttnPlan._fields_}


def _stream_ptr(stream) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def shape_of(q, k_pages, page_table, max_ctx_len=None, num_workers=0, variant=0) -> AttnShape:
    B, Qmax, Hq, D = q.shape
    NP, Hkv, P, D2 = k_pages.shape
    assert D == D2, "q and k_pages head_dim differ"
    maxp = page_table.shape[1]
    return make_shape(B, Hq, Hkv, D, Qmax, maxp, maxp * P if max_ctx_len is None else int(max_ctx_len),
                      NP, num_workers, P, variant)


def _check_tensors(q, k_pages, v_pages, page_table, ctx_lens, q_lens, out):
    import torch
    for name, t, dt in (("q", q, torch.bfloat16), ("k_pages", k_pages, torch.bfloat16),
                        ("v_pages", v_pages, torch.bfloat16), ("out", out, torch.bfloat16),
                        ("page_table", page_table, torch.int32), ("ctx_lens", ctx_lens, torch.int32),
                        ("q_lens", q_lens, torch.int32)):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {dt} CUDA tensor")
    if out.shape != q.shape or v_pages.shape != k_pages.shape:
        raise ValueError("out must match q and v_pages must match k_pages")


def new_workspace(nbytes: int, device="cuda"):
    """A zero-filled workspace of nbytes (the library requires zeros before
    the first use and leaves its split counters zero after every call)."""
    import torch
    return torch.zeros(nbytes, dtype=torch.uint8, device=device)


def decode_attn(q, k_pages, v_pages, page_table, ctx_lens, q_lens, out, scale: float,
                workspace=None, max_ctx_len: Optional[int] = None, num_workers: int = 0,
                stream=None, events=None, variant: int = 0):
    """ts_decode_attn on torch tensors; returns the workspace tensor used.

    ``events`` = (begin, end) handles from ``Event`` to time the main kernel.
    """
    import torch
    _check_tensors(q, k_pages, v_pages, page_table, ctx_lens, q_lens, out)
    shape = shape_of(q, k_pages, page_table, max_ctx_len, num_workers, variant)
    need = workspace_size(shape)
    if workspace is None:
        workspace = new_workspace(need, q.device)
    elif workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace has {workspace.numel() * workspace.element_size()} bytes, "
                         f"this call needs {need}")
    args = (ctypes.byref(shape), q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
            page_table.data_ptr(), ctx_lens.data_ptr(), q_lens.data_ptr(), out.data_ptr(),
            ctypes.c_float(scale), workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream_ptr(stream))
    if events is None:
        check(lib.ts_decode_attn(*args), "ts_decode_attn")
    else:
        check(lib.ts_decode_attn_events(*args, events[0].h, events[1].h), "ts_decode_attn_events")
    return workspace


def decode_attn_noalloc(q, k_pages, v_pages, page_table, ctx_lens, q_lens, out, scale: float,
                        max_ctx_len: Optional[int] = None, num_workers: int = 0, stream=None,
                        variant: int = 0) -> None:
    """ts_decode_attn_noalloc on torch tensors (no workspace: the library's
    static device scratch)."""
    _check_tensors(q, k_pages, v_pages, page_table, ctx_lens, q_lens, out)
    shape = shape_of(q, k_pages, page_table, max_ctx_len, num_workers, variant)
    check(lib.ts_decode_attn_noalloc(ctypes.byref(shape), q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
                                     page_table.data_ptr(), ctx_lens.data_ptr(), q_lens.data_ptr(),
                                     out.data_ptr(), ctypes.c_float(scale), _stream_ptr(stream)),
          "ts_decode_attn_noalloc")


def synth_fill(t, seed: int, stream_id: int, index_offset: int = 0, stream=None) -> None:
    """Fill a contiguous bf16 CUDA tensor with the seeded N(0,1) values."""
    import torch
    if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
        raise ValueError("synth_fill needs a contiguous bf16 CUDA tensor")
    check(lib.ts_synth_fill_bf16(t.data_ptr(), t.numel(), seed, stream_id, index_offset,
                                 _stream_ptr(stream)), "ts_synth_fill_bf16")


def sweep_lengths(batch: int, seed: int) -> np.ndarray:
    out = np.zeros(batch, dtype=np.int32)
    check(lib.ts_synth_sweep_lengths(batch, seed, out.ctypes.data), "ts_synth_sweep_lengths")
    return out


def page_table(ctx_lens: Sequence[int], max_pages_per_seq: int, seed: int) -> np.ndarray:
    lens = np.ascontiguousarray(ctx_lens, dtype=np.int32)
    out = np.zeros((len(lens), max_pages_per_seq), dtype=np.int32)
    check(lib.ts_synth_page_table(len(lens), lens.ctypes.data, 16, max_pages_per_seq, seed,
                                  out.ctypes.data), "ts_synth_page_table")
    return out


def copy_bytes(dst, src, stream=None) -> None:
    n = src.numel() * src.element_size()
    check(lib.ts_copy_bytes(dst.data_ptr(), src.data_ptr(), n, _stream_ptr(stream)), "ts_copy_bytes")


def stream_read(src, sink, stream=None) -> None:
    """Read every byte of `src` once (HBM read-ceiling probe); `sink` >= 2 MiB."""
    n = src.numel() * src.element_size()
    check(lib.ts_stream_read(src.data_ptr(), n, sink.data_ptr(), sink.numel() * sink.element_size(),
                             _stream_ptr(stream)), "ts_stream_read")


def page_gather_read(k_pages, v_pages, page_table, ctx_lens, q_lens, sink, max_ctx_len=None,
                     num_workers=0, stream=None, events=None) -> None:
    """Stream the K/V pages an attention call over the same arguments reads,
    computing nothing (the paged-access bandwidth ceiling).  `sink` is a
    uint32/int32 CUDA tensor of at least workers x 64 words (1,024 workers by
    default); ``events`` = (begin, end) handles from ``Event`` time the kernel."""
    import torch
    for name, t, dt in (("k_pages", k_pages, torch.bfloat16), ("v_pages", v_pages, torch.bfloat16),
                        ("page_table", page_table, torch.int32), ("ctx_lens", ctx_lens, torch.int32),
                        ("q_lens", q_lens, torch.int32)):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {dt} CUDA tensor")
    if v_pages.shape != k_pages.shape:
        raise ValueError("v_pages must match k_pages")
    NP, Hkv, P, D = k_pages.shape
    maxp = page_table.shape[1]
    shape = make_shape(ctx_lens.numel(), Hkv, Hkv, D, 1, maxp, maxp * P if max_ctx_len is None else int(max_ctx_len),
                       NP, num_workers, P)
    ev = (None, None) if events is None else (events[0].h, events[1].h)
    check(lib.ts_page_gather_read(ctypes.byref(shape), k_pages.data_ptr(), v_pages.data_ptr(),
                                  page_table.data_ptr(), ctx_lens.data_ptr(), q_lens.data_ptr(),
                                  sink.data_ptr(), sink.numel() * sink.element_size(), _stream_ptr(stream),
                                  ev[0], ev[1]), "ts_page_gather_read")


class Event:
    """A HIP event owned by the library (recorded on a caller's stream)."""

    def __init__(self):
        h = ctypes.c_void_p()
        check(lib.ts_event_create(ctypes.byref(h)), "ts_event_create")
        self.h = h.value

    def record(self, stream=None):
        check(lib.ts_event_record(self.h, _stream_ptr(stream)), "ts_event_record")

    def elapsed_ms(self, end: "Event") -> float:
        ms = ctypes.c_float()
        check(lib.ts_event_elapsed_ms(self.h, end.h, ctypes.byref(ms)), "ts_event_elapsed_ms")
        return float(ms.value)

    def __del__(self):
        try:
            if self.h:
                lib.ts_event_destroy(self.h)
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass


def concurrency_sweep(batches: Sequence[int] = (1, 2, 4, 8, 16, 32, 64, 128, 256, 512),
                      seeds: int = 5, warmup: int = 5, iters: int = 50,
                      num_q_heads: int = 32, num_kv_heads: int = 8, head_dim: int = 128,
                      verify_max_batch: int = 8, verify_q_len: int = 4,
                      min_rotation_bytes: int = 1 << 30, verify_tokens_per_step: float = 1.0) -> List[dict]:
    cfg = SweepConfig()
    cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim = num_q_heads, num_kv_heads, head_dim
    cfg.num_batches = len(batches)
    for i, b in enumerate(batches):
        cfg.batches[i] = b
    cfg.verify_max_batch, cfg.verify_q_len = verify_max_batch, verify_q_len
    cfg.num_seeds, cfg.warmup, cfg.iters = seeds, warmup, iters
    cfg.min_rotation_bytes = min_rotation_bytes
    cfg.verify_tokens_per_step = verify_tokens_per_step
    cap = len(batches) * seeds
    pts = (SweepPoint * cap)()
    n = ctypes.c_int32()
    check(lib.ts_concurrency_sweep(ctypes.byref(cfg), pts, cap, ctypes.byref(n)), "ts_concurrency_sweep")
    return [{f: getattr(pts[i], f) for f, _ in SweepPoint._fields_} for i in range(n.value)]


# ---- replica completion-time model (host only) ------------------------------

def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int64)


def tau_table(batch: Sequence[int], tau: Sequence[float], bmax: int) -> np.ndarray:
    """Dense tau(b), b = 1..bmax, from measured (batch, tau) points."""
    b = np.ascontiguousarray(batch, dtype=np.int32)
    t = _f64(tau)
    if b.shape != t.shape:
        raise ValueError("batch and tau differ in length")
    out = np.empty(bmax, dtype=np.float64)
    check(lib.ts_tau_table(b.ctypes.data, t.ctypes.data, len(b), bmax, out.ctypes.data), "ts_tau_table")
    return out


def replica_time(tau: Sequence[float], lengths: Sequence[int]) -> float:
    t, L = _f64(tau), _i64(lengths)
    T = ctypes.c_double()
    check(lib.ts_replica_time(t.ctypes.data, len(t), L.ctypes.data, len(L), ctypes.byref(T)),
          "ts_replica_time")
    return T.value


def request_shares(tau: Sequence[float], lengths: Sequence[int]) -> np.ndarray:
    t, L = _f64(tau), _i64(lengths)
    out = np.empty(len(L), dtype=np.float64)
    check(lib.ts_request_shares(t.ctypes.data, len(t), L.ctypes.data, len(L), out.ctypes.data),
          "ts_request_shares")
    return out


def step_makespan(tau: Sequence[float], lengths: Sequence[int], replica: Sequence[int], n_replicas: int):
    """(completion time per replica, step makespan)."""
    t, L = _f64(tau), _i64(lengths)
    r = np.ascontiguousarray(replica, dtype=np.int32)
    if len(r) != len(L):
        raise ValueError("lengths and replica differ in length")
    times = np.empty(max(n_replicas, 0), dtype=np.float64)
    T = ctypes.c_double()
    check(lib.ts_step_makespan(t.ctypes.data, len(t), L.ctypes.data, r.ctypes.data, len(L), n_replicas,
                               times.ctypes.data, ctypes.byref(T)), "ts_step_makespan")
    return times, T.value


# ---- steps around the verify attention ----------------------------------------

def kv_append(k_new, v_new, k_pages, v_pages, page_table, ctx_lens, q_lens, stream=None) -> None:
    """ts_kv_append on torch tensors (k_new, v_new: bf16 [B][Qmax][Hkv][D])."""
    B, Qmax, Hkv, D = k_new.shape
    NP = k_pages.shape[0]
    shape = make_shape(B, Hkv, Hkv, D, Qmax, page_table.shape[1], page_table.shape[1] * 16, NP)
    for t in (k_new, v_new, k_pages, v_pages, page_table, ctx_lens, q_lens):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("kv_append needs contiguous CUDA tensors")
    check(lib.ts_kv_append(ctypes.byref(shape), k_new.data_ptr(), v_new.data_ptr(), k_pages.data_ptr(),
                           v_pages.data_ptr(), page_table.data_ptr(), ctx_lens.data_ptr(), q_lens.data_ptr(),
                           _stream_ptr(stream)), "ts_kv_append")


def spec_accept(p_target, q_draft, draft_tokens, num_draft, u_accept, u_sample, num_accepted, next_token,
                workspace=None, stream=None):
    """ts_spec_accept on torch tensors; returns the workspace used."""
    import torch
    B, G1, V = p_target.shape
    G = G1 - 1
    need = int(lib.ts_spec_accept_workspace_size(B, V))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=p_target.device)
    ptr = lambda t: t.data_ptr() if t is not None else None  # noqa: E731
    check(lib.ts_spec_accept(B, V, G, p_target.data_ptr(), ptr(q_draft), ptr(draft_tokens),
                             num_draft.data_ptr(), ptr(u_accept), u_sample.data_ptr(), num_accepted.data_ptr(),
                             next_token.data_ptr(), workspace.data_ptr(),
                             workspace.numel() * workspace.element_size(), _stream_ptr(stream)),
          "ts_spec_accept")
    return workspace
