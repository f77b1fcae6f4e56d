"""Thin ctypes binding of libdash (include/dash.h), same names as the C ABI.

Argument marshalling only: shapes, raw device pointers and the current HIP
stream are taken from torch tensors and passed through; every step of the
computation runs in the library's HIP kernels.  If libdash.so is missing this
module raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdash.so")

DASH_SCHED_ATOMIC, DASH_SCHED_NAIVE, DASH_SCHED_DESCENDING = 0, 1, 2
DASH_SCHED_SHIFT, DASH_SCHED_SYMSHIFT, DASH_SCHED_AUTO, DASH_SCHED_PARTIALS, DASH_SCHED_SPLIT = 3, 4, 5, 6, 7
SCHEDULES = {"atomic": 0, "naive": 1, "descending": 2, "shift": 3, "symshift": 4, "auto": 5, "partials": 6,
             "split": 7}
DASH_OK, DASH_ERR_INVALID_ARG, DASH_ERR_UNSUPPORTED = 0, -1, -2
DASH_ERR_HIP, DASH_ERR_TIMEOUT, DASH_ERR_NO_DEVICE = -3, -4, -5
DASH_FLAG_POISON_COUNTERS = 1
DASH_TICKETS_AUTO, DASH_TICKETS_HEAD_MAJOR, DASH_TICKETS_CHAIN_MAJOR = 0, 1, 2
DASH_PLACEMENT_AUTO, DASH_PLACEMENT_GLOBAL, DASH_PLACEMENT_XCD = 0, 1, 2

# every symbol include/dash.h declares
EXPORTS = ("dash_attn_fwd", "dash_attn_fwd_ex", "dash_attn_bwd", "dash_bwd_workspace_size",
           "dash_attn_bwd_ex", "dash_attn_bwd_noalloc", "dash_bwd_check", "dash_resolve_schedule", "dash_schedule_table",
           "dash_bwd_placement", "dash_mfma_peak", "dash_last_error", "dash_release_workspace",
           "dash_auto_schedule", "dash_model_makespan")


class DashError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libdash error {code}: {msg}")
        self.code = code


class dash_bwd_options_t(ctypes.Structure):
    _fields_ = [("spin_limit", ctypes.c_int), ("flags", ctypes.c_int),
                ("witness", ctypes.c_void_p), ("partials", ctypes.c_void_p),
                ("dq_accum", ctypes.c_void_p), ("event_main_begin", ctypes.c_void_p),
                ("event_main_end", ctypes.c_void_p), ("max_workgroups", ctypes.c_int),
                ("ticket_order", ctypes.c_int), ("placement", ctypes.c_int),
                ("wait_stats", ctypes.c_void_p)]


_lib = None


def load():
    """Load libdash.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise DashError(DASH_ERR_NO_DEVICE, f"{LIB_PATH} is not built (run __graft_entry__.build())")
        lib = ctypes.CDLL(LIB_PATH)
        vp, ci, cf, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        ip = ctypes.POINTER(ctypes.c_int)
        lib.dash_attn_fwd.argtypes = [vp] * 5 + [ci] * 5
        lib.dash_attn_fwd_ex.argtypes = [vp] * 5 + [ci] * 5 + [cf, vp]
        lib.dash_attn_bwd.argtypes = [vp] * 9 + [ci] * 6
        lib.dash_attn_bwd_ex.argtypes = ([vp] * 9 + [ci] * 6 + [cf, vp, sz,
                                         ctypes.POINTER(dash_bwd_options_t), vp])
        lib.dash_attn_bwd_noalloc.argtypes = [vp] * 9 + [ci] * 6 + [cf, vp, vp]
        lib.dash_bwd_workspace_size.argtypes = [ci] * 5
        lib.dash_bwd_workspace_size.restype = sz
        lib.dash_bwd_check.argtypes = [vp, vp]
        lib.dash_resolve_schedule.argtypes = [ci] * 3
        lib.dash_schedule_table.argtypes = [ci] * 6 + [ip] * 5
        lib.dash_bwd_placement.argtypes = [ci] * 6
        lib.dash_mfma_peak.argtypes = [ci, ctypes.POINTER(ctypes.c_double)]
        dp = ctypes.POINTER(ctypes.c_double)
        lib.dash_auto_schedule.argtypes = [ci] * 6 + [ip, dp]
        lib.dash_model_makespan.argtypes = [ci] * 9 + [ctypes.c_double, ctypes.c_double, dp]
        lib.dash_last_error.restype = ctypes.c_char_p
        lib.dash_release_workspace.restype = None
        for f in ("dash_attn_fwd", "dash_attn_fwd_ex", "dash_attn_bwd", "dash_attn_bwd_ex", "dash_attn_bwd_noalloc",
                  "dash_bwd_check", "dash_resolve_schedule", "dash_schedule_table", "dash_bwd_placement",
                  "dash_mfma_peak", "dash_auto_schedule", "dash_model_makespan"):
            getattr(lib, f).restype = ci
        _lib = lib
    return _lib


def _check(rc: int):
    if rc != DASH_OK:
        raise DashError(rc, load().dash_last_error().decode())
    return rc


def _sched(s) -> int:
    return SCHEDULES[s] if isinstance(s, str) else int(s)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return ctypes.c_void_p(stream if isinstance(stream, int) else stream.cuda_stream)


def _shape(q):
    if q.dim() != 4:
        raise DashError(DASH_ERR_INVALID_ARG, "tensors must be [B, H, N, d]")
    return tuple(int(x) for x in q.shape)


def _require(ts, dtype_name):
    import torch
    dt = {"bf16": torch.bfloat16, "f32": torch.float32}[dtype_name]
    for t in ts:
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise DashError(DASH_ERR_INVALID_ARG, f"expected contiguous {dtype_name} device tensors")


def dash_last_error() -> str:
    return load().dash_last_error().decode()


def dash_release_workspace():
    load().dash_release_workspace()


def dash_resolve_schedule(schedule, d: int, causal: bool) -> int:
    return load().dash_resolve_schedule(_sched(schedule), d, int(causal))


def dash_auto_schedule(B: int, H: int, N: int, d: int, causal: bool, workers: int = 0):
    """(schedule, predicted ms) that DASH_SCHED_AUTO runs for this shape."""
    s, ms = ctypes.c_int(), ctypes.c_double()
    _check(load().dash_auto_schedule(B, H, N, d, int(causal), workers, ctypes.byref(s), ctypes.byref(ms)))
    return s.value, ms.value


def dash_model_makespan(schedule, B: int, H: int, N: int, d: int, causal: bool, workers: int, c: float, r: float,
                        ticket_order: int = DASH_TICKETS_AUTO, max_heads: int = 0) -> float:
    """Makespan of the DAG model with block-step costs c (compute) and r (reduction)."""
    m = ctypes.c_double()
    _check(load().dash_model_makespan(_sched(schedule), B, H, N, d, int(causal), workers, ticket_order,
                                      max_heads, c, r, ctypes.byref(m)))
    return m.value


def dash_bwd_workspace_size(B: int, H: int, N: int, d: int, schedule="shift") -> int:
    return int(load().dash_bwd_workspace_size(B, H, N, d, _sched(schedule)))


def dash_attn_fwd(q, k, v, o, lse, causal: bool, scale=None, stream=None):
    """O and L of attention into o (bf16) and lse (fp32) on the current stream."""
    B, H, N, d = _shape(q)
    _require((q, k, v, o), "bf16")
    _require((lse,), "f32")
    s = 0.0 if scale is None else float(scale)  # 0: the library's default 1/sqrt(d)
    _check(load().dash_attn_fwd_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, N, d,
                                   int(causal), s, _stream(stream)))


def dash_attn_bwd(q, k, v, o, dO, lse, dq, dk, dv, causal: bool, schedule, scale=None,
                  workspace=None, options: dash_bwd_options_t | None = None, stream=None):
    """Backward into dq, dk, dv.  With ``workspace`` (a device uint8 tensor of at
    least dash_bwd_workspace_size bytes) the call is asynchronous on the
    current stream; without it the library's own workspace is used and the
    call synchronizes and reports wait timeouts."""
    B, H, N, d = _shape(q)
    _require((q, k, v, o, dO, dq, dk, dv), "bf16")
    _require((lse,), "f32")
    lib = load()
    if workspace is None and options is None and scale is None:
        _check(lib.dash_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dO), _ptr(lse),
                                 _ptr(dq), _ptr(dk), _ptr(dv), B, H, N, d, int(causal),
                                 _sched(schedule)))
        return
    if workspace is None:
        raise DashError(DASH_ERR_INVALID_ARG, "scale/options need an explicit workspace")
    s = 0.0 if scale is None else float(scale)  # 0: the library's default 1/sqrt(d)
    opt = ctypes.byref(options) if options is not None else None
    _check(lib.dash_attn_bwd_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dO), _ptr(lse),
                                _ptr(dq), _ptr(dk), _ptr(dv), B, H, N, d, int(causal),
                                _sched(schedule), s, _ptr(workspace), workspace.numel(), opt,
                                _stream(stream)))


def dash_attn_bwd_noalloc(q, k, v, o, dO, lse, dq, dk, dv, causal: bool, schedule, scale=None, status=None,
                          stream=None):
    """Backward into dq, dk, dv on the library's fixed per-device scratch: no
    allocation, asynchronous on the current stream.  ``status``: optional
    device int32 tensor (one element) that receives 0, or 1 after a wait
    timeout, once the stream has run the call."""
    B, H, N, d = _shape(q)
    _require((q, k, v, o, dO, dq, dk, dv), "bf16")
    _require((lse,), "f32")
    if status is not None and (not status.is_cuda or status.dtype.itemsize != 4):
        raise DashError(DASH_ERR_INVALID_ARG, "status must be a device int32 tensor")
    s = 0.0 if scale is None else float(scale)
    _check(load().dash_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dO), _ptr(lse),
                                        _ptr(dq), _ptr(dk), _ptr(dv), B, H, N, d, int(causal),
                                        _sched(schedule), s, _ptr(status), _stream(stream)))


def dash_bwd_check(workspace, stream=None) -> int:
    """Synchronize and return the status of the last backward on ``workspace``
    (DASH_OK or DASH_ERR_TIMEOUT) without raising."""
    return load().dash_bwd_check(_ptr(workspace), _stream(stream))


def dash_bwd_placement(B: int, H: int, N: int, d: int, causal: bool, schedule="auto") -> int:
    """The placement AUTO picks on the current device (DASH_PLACEMENT_GLOBAL / _XCD)."""
    rc = load().dash_bwd_placement(B, H, N, d, int(causal), _sched(schedule))
    if rc < 0:
        _check(rc)
    return rc


def dash_mfma_peak(iters: int = 0) -> float:
    """Measured bf16 dense MFMA throughput of the current device in TFLOP/s."""
    out = ctypes.c_double(0.0)
    _check(load().dash_mfma_peak(int(iters), ctypes.byref(out)))
    return out.value


def dash_schedule_table(schedule, N: int, d: int, causal: bool, placement=DASH_PLACEMENT_GLOBAL, heads: int = 1) -> dict:
    """The schedule the kernels follow for one head of a call of ``heads`` (= B*H)
    heads under ``placement`` (host computation)."""
    lib = load()
    geo = (ctypes.c_int * 6)()
    _check(lib.dash_schedule_table(_sched(schedule), heads, N, d, int(causal), placement, geo, None, None, None, None))
    t_r, t_c, br, chains, bc, grp = list(geo)
    cap = t_r + 1
    chain_len = np.zeros(chains, np.int32)
    task_kv = np.full(chains * cap, -1, np.int32)
    task_q = np.full(chains * cap, -1, np.int32)
    rank = np.zeros(t_r * t_c, np.int32)
    p = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
    _check(lib.dash_schedule_table(_sched(schedule), heads, N, d, int(causal), placement, geo, p(chain_len), p(task_kv),
                                   p(task_q), p(rank)))
    return dict(t_r=t_r, t_c=t_c, br=br, chains=chains, bc=bc, group=grp, chain_len=chain_len,
                task_kv=task_kv.reshape(chains, cap), task_q=task_q.reshape(chains, cap),
                rank=rank.reshape(t_r, t_c))


# ----------------------------------------------------------------- helpers
def new_workspace(B, H, N, d, schedule="shift"):
    import torch
    n = dash_bwd_workspace_size(B, H, N, d, schedule)
    return torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")


def attn_fwd(q, k, v, causal: bool, scale=None):
    import torch
    B, H, N, d = _shape(q)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    dash_attn_fwd(q, k, v, o, lse, causal, scale)
    return o, lse


def attn_bwd(q, k, v, o, dO, lse, causal: bool, schedule="auto", scale=None, workspace=None,
             options=None):
    import torch
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    dash_attn_bwd(q, k, v, o, dO, lse, dq, dk, dv, causal, schedule, scale, workspace, options)
    return dq, dk, dv
