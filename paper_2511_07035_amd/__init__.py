"""MI355X GoCkpt hot path -- thin Python binding of ``include/gockpt.h``.

Every function here marshals arguments into the HIP library
``libgockpt.so`` and raises :class:`GockptError` on a negative status; all
arithmetic runs in the library (HIP kernels on the device, the C++ replay on
the host).  PyTorch is used only to allocate device memory, pinned host
memory and streams (see :class:`Session`).  If the library is missing the
import of a function fails loudly -- there is no fallback.

Build it with ``python -m paper_2511_07035_amd.build``.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgockpt.so")
BENCH_LIB_PATH = os.path.join(_HERE, "libgockpt_bench.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "gockpt.h")

GOCKPT_OK = 0
GOCKPT_EAGAIN = 1
GOCKPT_EINVAL = -1
GOCKPT_ESTATE = -2
GOCKPT_EBUSY = -3
GOCKPT_ENOMEM = -4
GOCKPT_EHIP = -5
GOCKPT_EFAILED = -6
GOCKPT_MAX_K = 256
GOCKPT_ALIGN_ELEMS = 8

_NAMES = {0: "OK", 1: "EAGAIN", -1: "EINVAL", -2: "ESTATE", -3: "EBUSY", -4: "ENOMEM", -5: "EHIP",
          -6: "EFAILED"}


class GockptError(RuntimeError):
    def __init__(self, code: int, func: str, msg: str):
        self.code = code
        super().__init__(f"{func} -> {_NAMES.get(code, code)}: {msg}")


class _Strict(ctypes.Structure):
    """A ctypes struct that refuses attributes it does not declare, so a
    misspelt field fails loudly instead of being ignored."""

    def __setattr__(self, name, value):
        if not name.startswith("_") and name not in {f[0] for f in type(self)._fields_}:
            raise AttributeError(f"{type(self).__name__} has no field {name!r}")
        super().__setattr__(name, value)


class gockpt_config(_Strict):
    _fields_ = [
        ("n", ctypes.c_int64),
        ("master", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p), ("exp_avg_sq", ctypes.c_void_p),
        ("weight_bf16", ctypes.c_void_p), ("grad16", ctypes.c_void_p),
        ("beta1", ctypes.c_double), ("beta2", ctypes.c_double), ("eps", ctypes.c_double),
        ("weight_decay", ctypes.c_double),
        ("check_overflow", ctypes.c_int32), ("dynamic_scale", ctypes.c_int32),
        ("init_scale", ctypes.c_float), ("growth_factor", ctypes.c_float),
        ("backoff_factor", ctypes.c_float), ("min_scale", ctypes.c_float),
        ("growth_interval", ctypes.c_int64), ("init_step", ctypes.c_int64), ("init_tracker", ctypes.c_int64),
        ("ring", ctypes.c_void_p), ("ring_bytes", ctypes.c_size_t), ("copy_bytes", ctypes.c_size_t),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
        ("compute_stream", ctypes.c_void_p), ("copy_stream", ctypes.c_void_p),
        ("timing", ctypes.c_int32), ("copy_threads", ctypes.c_int32),
        ("host_staging", ctypes.c_void_p), ("host_staging_bytes", ctypes.c_size_t),
        ("grad_dtype", ctypes.c_int32), ("grad_norm_off", ctypes.c_int32),
        ("found_inf", ctypes.c_void_p),
    ]


GOCKPT_GRAD_BF16, GOCKPT_GRAD_FP16 = 0, 1


class gockpt_window_opts(_Strict):
    _fields_ = [("replay_every", ctypes.c_int32), ("replay_threads", ctypes.c_int32),
                ("wait_policy", ctypes.c_int32), ("ring_off", ctypes.c_int32),
                ("late_plan", ctypes.c_int32), ("no_timing", ctypes.c_int32), ("defer_copies", ctypes.c_int32),
                ("reserved_", ctypes.c_int32 * 1)]


GOCKPT_WAIT_LAZY, GOCKPT_WAIT_GRADS, GOCKPT_WAIT_ALL = 0, 1, 2
GOCKPT_RING_QUERY, GOCKPT_RING_HOST_WAIT, GOCKPT_RING_DEVICE_WAIT = 0, 1, 2


class gockpt_step_record(ctypes.Structure):
    _fields_ = [
        ("t", ctypes.c_int64), ("tracker", ctypes.c_int64),
        ("scale_used", ctypes.c_float), ("scale_next", ctypes.c_float), ("lr", ctypes.c_float),
        ("skip", ctypes.c_int32), ("nonfinite", ctypes.c_int32), ("window_step", ctypes.c_int32),
        ("gnorm2", ctypes.c_double),
        ("step_size", ctypes.c_float), ("sqrt_bc2", ctypes.c_float), ("decay", ctypes.c_float),
        ("inv_scale", ctypes.c_float),
    ]


class gockpt_window_stats(ctypes.Structure):
    _fields_ = [
        ("K", ctypes.c_int32), ("steps_done", ctypes.c_int32), ("skipped", ctypes.c_int32),
        ("n_gates", ctypes.c_int32),
        ("bytes_ring", ctypes.c_uint64), ("bytes_spilled", ctypes.c_uint64), ("bytes_d2h", ctypes.c_uint64),
        ("n_copies", ctypes.c_uint64),
        ("copy_ms", ctypes.c_double), ("prepass_ms", ctypes.c_double), ("update_ms", ctypes.c_double),
        ("wait_ms", ctypes.c_double),
        ("bytes_host_copied", ctypes.c_uint64),
        ("host_copy_ms", ctypes.c_double),
        ("replay_ms", ctypes.c_double),
    ]


class gockpt_ckpt_meta(ctypes.Structure):
    _fields_ = [
        ("t", ctypes.c_int64), ("tracker", ctypes.c_int64), ("scale", ctypes.c_float),
        ("K", ctypes.c_int32), ("skipped", ctypes.c_int32), ("reserved_", ctypes.c_int32),
        ("restore_ms", ctypes.c_double), ("element_updates", ctypes.c_int64),
    ]


class gockpt_arena_layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in ("records", "master", "exp_avg", "exp_avg_sq", "grads", "total")]


class gockpt_plan_params(_Strict):
    _fields_ = [("n", ctypes.c_int64), ("tensor_ends", ctypes.c_void_p), ("n_tensors", ctypes.c_int32),
                ("wait_policy", ctypes.c_int32), ("align", ctypes.c_int64),
                ("t_fwd_ms", ctypes.c_double), ("t_bwd_ms", ctypes.c_double), ("t_upd_ms", ctypes.c_double),
                ("pack_gbs", ctypes.c_double), ("link_gbs", ctypes.c_double),
                ("ring_bytes", ctypes.c_uint64), ("copy_bytes", ctypes.c_uint64),
                ("state_bytes", ctypes.c_double), ("grad_bytes", ctypes.c_double),
                ("max_K", ctypes.c_int32), ("ring_plan", ctypes.c_int32),
                ("staging_bytes", ctypes.c_uint64), ("host_gbs", ctypes.c_double)]


class gockpt_plan_result(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("reserved_", ctypes.c_int32), ("stall_ms", ctypes.c_double),
                ("latency_ms", ctypes.c_double), ("d2h_bytes", ctypes.c_double), ("spilled_bytes", ctypes.c_double)]


class gockpt_ckpt_info(_Strict):
    _fields_ = [("n", ctypes.c_int64), ("t", ctypes.c_int64), ("tracker", ctypes.c_int64), ("scale", ctypes.c_float),
                ("K", ctypes.c_int32), ("skipped", ctypes.c_int32), ("has_user", ctypes.c_int32),
                ("beta1", ctypes.c_double), ("beta2", ctypes.c_double), ("eps", ctypes.c_double),
                ("weight_decay", ctypes.c_double), ("piece_bytes", ctypes.c_uint64), ("data_bytes", ctypes.c_uint64)]


class gockpt_io_stats(ctypes.Structure):
    _fields_ = [("bytes", ctypes.c_double), ("ms", ctypes.c_double), ("pieces", ctypes.c_int64)]


assert ctypes.sizeof(gockpt_step_record) == 64

RECORD_DTYPE = np.dtype([
    ("t", "<i8"), ("tracker", "<i8"), ("scale_used", "<f4"), ("scale_next", "<f4"), ("lr", "<f4"),
    ("skip", "<i4"), ("nonfinite", "<i4"), ("window_step", "<i4"), ("gnorm2", "<f8"),
    ("step_size", "<f4"), ("sqrt_bc2", "<f4"), ("decay", "<f4"), ("inv_scale", "<f4")])
assert RECORD_DTYPE.itemsize == 64

_P = ctypes.c_void_p
_CTX = ctypes.c_void_p
_lib = None


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2511_07035_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.gockpt_workspace_bytes.argtypes = [ctypes.c_int64]
        L.gockpt_workspace_bytes.restype = ctypes.c_size_t
        L.gockpt_arena_layout_for.argtypes = [ctypes.c_int, _P, ctypes.c_int64,
                                              ctypes.POINTER(gockpt_arena_layout), _P]
        L.gockpt_plan_bounds.argtypes = [ctypes.c_int, ctypes.c_int64, _P, ctypes.c_int, ctypes.c_int64, _P]
        L.gockpt_create.argtypes = [ctypes.POINTER(gockpt_config), ctypes.POINTER(_CTX)]
        L.gockpt_create_noalloc.argtypes = [ctypes.POINTER(gockpt_config), ctypes.POINTER(_CTX)]
        L.gockpt_destroy.argtypes = [_CTX]
        L.gockpt_last_error.argtypes = [_CTX]
        L.gockpt_last_error.restype = ctypes.c_char_p
        L.gockpt_begin_window.argtypes = [_CTX, ctypes.c_int, _P, _P, ctypes.c_size_t]
        L.gockpt_begin_window_ex.argtypes = [_CTX, ctypes.c_int, _P, _P, ctypes.c_size_t,
                                             ctypes.POINTER(gockpt_window_opts)]
        L.gockpt_arena_layout_ex.argtypes = [ctypes.c_int, _P, ctypes.c_int64, ctypes.c_int,
                                             ctypes.POINTER(gockpt_arena_layout), _P]
        L.gockpt_backward_begin.argtypes = [_CTX, _P]
        L.gockpt_step.argtypes = [_CTX, ctypes.c_float]
        L.gockpt_drain.argtypes = [_CTX, ctypes.c_int, ctypes.POINTER(gockpt_window_stats)]
        L.gockpt_restore.argtypes = [_CTX, _P, _P, _P, _P, ctypes.POINTER(gockpt_ckpt_meta), ctypes.c_int]
        L.gockpt_restore_async.argtypes = [_CTX, _P, _P, _P, _P, ctypes.c_int]
        L.gockpt_scan_grads.argtypes = [_CTX, ctypes.c_int64, ctypes.c_int64, _P]
        L.gockpt_restore_wait.argtypes = [_CTX, ctypes.POINTER(gockpt_ckpt_meta)]
        L.gockpt_abort_window.argtypes = [_CTX]
        L.gockpt_get_scaler.argtypes = [_CTX, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_float),
                                        ctypes.POINTER(ctypes.c_int64)]
        L.gockpt_window_records.argtypes = [_CTX, _P, ctypes.c_int]
        L.gockpt_replay_arena.argtypes = [ctypes.c_int, _P, ctypes.c_int64, _P, ctypes.c_size_t,
                                          ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                          ctypes.c_int, _P, _P, _P, _P, ctypes.POINTER(gockpt_ckpt_meta),
                                          ctypes.c_int]
        L.gockpt_window_step_times.argtypes = [_CTX, _P, ctypes.c_int]
        L.gockpt_host_alloc.argtypes = [ctypes.c_size_t, ctypes.POINTER(_P)]
        L.gockpt_host_free.argtypes = [_P]
        L.gockpt_simulate_window.argtypes = [ctypes.POINTER(gockpt_plan_params), ctypes.c_int, _P,
                                             ctypes.POINTER(gockpt_plan_result), _P]
        L.gockpt_plan_window.argtypes = [ctypes.POINTER(gockpt_plan_params), _P, ctypes.POINTER(gockpt_plan_result)]
        L.gockpt_write_checkpoint.argtypes = [ctypes.c_char_p, _P, _P, _P, ctypes.POINTER(gockpt_ckpt_info),
                                              ctypes.c_char_p, ctypes.c_int, ctypes.POINTER(gockpt_io_stats)]
        L.gockpt_read_checkpoint_info.argtypes = [ctypes.c_char_p, ctypes.POINTER(gockpt_ckpt_info)]
        L.gockpt_read_checkpoint.argtypes = [ctypes.c_char_p, ctypes.c_int64, _P, _P, _P,
                                             ctypes.POINTER(gockpt_ckpt_info), ctypes.c_int,
                                             ctypes.POINTER(gockpt_io_stats)]
        L.gockpt_read_checkpoint_user.argtypes = [ctypes.c_char_p, _P, ctypes.c_size_t,
                                                  ctypes.POINTER(ctypes.c_size_t)]
        L.gockpt_find_latest_checkpoint.argtypes = [ctypes.c_char_p, _P, ctypes.c_size_t]
        L.gockpt_persist.argtypes = [_CTX, ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int, ctypes.c_int]
        L.gockpt_persist_wait.argtypes = [_CTX, ctypes.POINTER(gockpt_io_stats)]
        L.gockpt_load.argtypes = [_CTX, ctypes.c_char_p, _P, ctypes.c_size_t, ctypes.c_int,
                                  ctypes.POINTER(gockpt_ckpt_info)]
        for name in ("gockpt_begin_window_ex", "gockpt_arena_layout_ex", "gockpt_window_step_times",
                     "gockpt_host_alloc", "gockpt_host_free", "gockpt_plan_bounds", "gockpt_arena_layout_for",
                     "gockpt_create", "gockpt_destroy",
                     "gockpt_begin_window", "gockpt_backward_begin", "gockpt_step", "gockpt_drain",
                     "gockpt_restore", "gockpt_restore_async", "gockpt_restore_wait", "gockpt_abort_window",
                     "gockpt_scan_grads", "gockpt_get_scaler", "gockpt_window_records",
                     "gockpt_replay_arena", "gockpt_simulate_window", "gockpt_plan_window",
                     "gockpt_write_checkpoint", "gockpt_read_checkpoint_info", "gockpt_read_checkpoint",
                     "gockpt_read_checkpoint_user", "gockpt_find_latest_checkpoint", "gockpt_persist",
                     "gockpt_persist_wait", "gockpt_load"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int, func: str, ctx=None) -> int:
    if rc < 0:
        msg = lib().gockpt_last_error(ctx)
        raise GockptError(rc, func, msg.decode() if msg else "")
    return rc


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int64)


# ---- host-only planning ----------------------------------------------------

def gockpt_workspace_bytes(n: int) -> int:
    return int(lib().gockpt_workspace_bytes(int(n)))


def gockpt_arena_layout_for(K: int, bounds, n: int):
    """Returns (layout, grad_offsets[K])."""
    b = _i64(bounds)
    lay = gockpt_arena_layout()
    goff = np.zeros(max(int(K), 1), dtype=np.uint64)
    _check(lib().gockpt_arena_layout_for(int(K), b.ctypes.data, int(n), ctypes.byref(lay), goff.ctypes.data),
           "gockpt_arena_layout_for")
    return lay, goff[:K]


def gockpt_arena_layout_ex(K: int, bounds, n: int, replay_every: int = 0):
    """Returns (layout, grad_offsets[K]) for a window with in-window replay."""
    b = _i64(bounds)
    lay = gockpt_arena_layout()
    goff = np.zeros(max(int(K), 1), dtype=np.uint64)
    _check(lib().gockpt_arena_layout_ex(int(K), b.ctypes.data, int(n), int(replay_every), ctypes.byref(lay),
                                        goff.ctypes.data), "gockpt_arena_layout_ex")
    return lay, goff[:K]


def gockpt_plan_bounds(K: int, n: int, tensor_ends=None, align: int = 256) -> np.ndarray:
    out = np.zeros(int(K) + 1, dtype=np.int64)
    if tensor_ends is None:
        rc = lib().gockpt_plan_bounds(int(K), int(n), None, 0, int(align), out.ctypes.data)
    else:
        te = _i64(tensor_ends)
        rc = lib().gockpt_plan_bounds(int(K), int(n), te.ctypes.data, int(te.size), int(align), out.ctypes.data)
    _check(rc, "gockpt_plan_bounds")
    return out


def _plan_params(n, t_fwd_ms, t_bwd_ms, t_upd_ms, link_gbs, *, tensor_ends=None, wait_policy=0, align=256,
                 pack_gbs=0.0, ring_bytes=0, copy_bytes=0, state_bytes=0.0, grad_bytes=0.0, max_K=0,
                 ring_plan=GOCKPT_RING_QUERY, staging_bytes=0, host_gbs=0.0):
    te = None if tensor_ends is None else _i64(tensor_ends)
    p = gockpt_plan_params(int(n), te.ctypes.data if te is not None else None, int(te.size) if te is not None else 0,
                           int(wait_policy), int(align), float(t_fwd_ms), float(t_bwd_ms), float(t_upd_ms),
                           float(pack_gbs), float(link_gbs), int(ring_bytes), int(copy_bytes), float(state_bytes),
                           float(grad_bytes), int(max_K), int(ring_plan), int(staging_bytes), float(host_gbs))
    return p, te


def gockpt_simulate_window(bounds, n, t_fwd_ms, t_bwd_ms, t_upd_ms, link_gbs, **kw):
    """Predicted stall of a window: (gockpt_plan_result, per-step delays [K+1])."""
    p, te = _plan_params(n, t_fwd_ms, t_bwd_ms, t_upd_ms, link_gbs, **kw)
    b = _i64(bounds)
    K = b.size - 1
    out = gockpt_plan_result()
    per = np.zeros(K + 1, dtype=np.float64)
    _check(lib().gockpt_simulate_window(ctypes.byref(p), K, b.ctypes.data, ctypes.byref(out), per.ctypes.data),
           "gockpt_simulate_window")
    del te
    return out, per


def gockpt_plan_window(n, t_fwd_ms, t_bwd_ms, t_upd_ms, link_gbs, **kw):
    """K and bounds with the least predicted stall: (bounds, gockpt_plan_result)."""
    p, te = _plan_params(n, t_fwd_ms, t_bwd_ms, t_upd_ms, link_gbs, **kw)
    cap = p.max_K if p.max_K > 0 else 7
    b = np.zeros(cap + 1, dtype=np.int64)
    out = gockpt_plan_result()
    _check(lib().gockpt_plan_window(ctypes.byref(p), b.ctypes.data, ctypes.byref(out)), "gockpt_plan_window")
    del te
    return b[:out.K + 1].copy(), out


# ---- pinned host memory ------------------------------------------------------

def gockpt_host_alloc(nbytes: int) -> int:
    out = _P()
    _check(lib().gockpt_host_alloc(int(nbytes), ctypes.byref(out)), "gockpt_host_alloc", None)
    return out.value


def gockpt_host_free(ptr: int) -> None:
    _check(lib().gockpt_host_free(ptr), "gockpt_host_free", None)


def host_view(ptr: int, nbytes: int, dtype, offset: int = 0, count: int | None = None) -> np.ndarray:
    """numpy view (no copy) of host memory at ptr+offset."""
    dt = np.dtype(dtype)
    if count is None:
        count = (nbytes - offset) // dt.itemsize
    buf = (ctypes.c_uint8 * (count * dt.itemsize)).from_address(ptr + offset)
    return np.frombuffer(buf, dtype=dt, count=count)


# ---- context ------------------------------------------------------------------

def gockpt_create(cfg: gockpt_config) -> int:
    ctx = _CTX()
    _check(lib().gockpt_create(ctypes.byref(cfg), ctypes.byref(ctx)), "gockpt_create", None)
    return ctx.value


def gockpt_create_noalloc(cfg: gockpt_config) -> int:
    """gockpt_create with the library's static scratch workspace (cfg.workspace
    must be None); for callers that cannot allocate."""
    ctx = _CTX()
    _check(lib().gockpt_create_noalloc(ctypes.byref(cfg), ctypes.byref(ctx)), "gockpt_create_noalloc", None)
    return ctx.value


def gockpt_destroy(ctx) -> None:
    _check(lib().gockpt_destroy(ctx), "gockpt_destroy", None)


def gockpt_begin_window(ctx, K: int, bounds, host_arena_ptr: int, arena_bytes: int) -> None:
    b = _i64(bounds)
    _check(lib().gockpt_begin_window(ctx, int(K), b.ctypes.data, host_arena_ptr, int(arena_bytes)),
           "gockpt_begin_window", ctx)


def gockpt_begin_window_ex(ctx, K: int, bounds, host_arena_ptr: int, arena_bytes: int, replay_every: int = 0,
                           replay_threads: int = 0, wait_policy: int = GOCKPT_WAIT_LAZY,
                           ring_off: bool = False, late_plan: int = GOCKPT_RING_QUERY, timing: bool = True,
                           defer_copies: bool = False) -> None:
    """late_plan: the window's ring plan, GOCKPT_RING_* (True means HOST_WAIT);
    timing=False: no timing events in this window; defer_copies: a step's
    copies are queued at the next library call."""
    b = _i64(bounds)
    opts = gockpt_window_opts(int(replay_every), int(replay_threads), int(wait_policy), int(bool(ring_off)),
                              int(late_plan), 0 if timing else 1, int(bool(defer_copies)))
    _check(lib().gockpt_begin_window_ex(ctx, int(K), b.ctypes.data, host_arena_ptr, int(arena_bytes),
                                        ctypes.byref(opts)), "gockpt_begin_window_ex", ctx)


def gockpt_backward_begin(ctx, stream_ptr: int | None = None) -> None:
    _check(lib().gockpt_backward_begin(ctx, stream_ptr), "gockpt_backward_begin", ctx)


def gockpt_step(ctx, lr: float) -> None:
    _check(lib().gockpt_step(ctx, float(lr)), "gockpt_step", ctx)


def gockpt_drain(ctx, blocking: bool = True):
    """Returns the window stats, or None while copies are in flight."""
    st = gockpt_window_stats()
    rc = _check(lib().gockpt_drain(ctx, int(bool(blocking)), ctypes.byref(st)), "gockpt_drain", ctx)
    return None if rc == GOCKPT_EAGAIN else st


def gockpt_restore(ctx, master_out=None, exp_avg_out=None, exp_avg_sq_out=None, w_bf16_out=None,
                   nthreads: int = 0) -> gockpt_ckpt_meta:
    """Outputs are host pointers (int) or None (restore in place in the arena)."""
    meta = gockpt_ckpt_meta()
    _check(lib().gockpt_restore(ctx, master_out, exp_avg_out, exp_avg_sq_out, w_bf16_out, ctypes.byref(meta),
                                int(nthreads)), "gockpt_restore", ctx)
    return meta


def gockpt_scan_grads(ctx, begin: int, end: int, stream=None) -> None:
    """stream: a hipStream_t handle (int) or None for the compute stream."""
    _check(lib().gockpt_scan_grads(ctx, int(begin), int(end), stream), "gockpt_scan_grads", ctx)


def gockpt_restore_async(ctx, master_out=None, exp_avg_out=None, exp_avg_sq_out=None, w_bf16_out=None,
                         nthreads: int = 0) -> None:
    """Start the restore in a library thread; the outputs must stay alive
    until gockpt_restore_wait."""
    _check(lib().gockpt_restore_async(ctx, master_out, exp_avg_out, exp_avg_sq_out, w_bf16_out, int(nthreads)),
           "gockpt_restore_async", ctx)


def gockpt_restore_wait(ctx) -> gockpt_ckpt_meta:
    meta = gockpt_ckpt_meta()
    _check(lib().gockpt_restore_wait(ctx, ctypes.byref(meta)), "gockpt_restore_wait", ctx)
    return meta


def gockpt_abort_window(ctx) -> None:
    _check(lib().gockpt_abort_window(ctx), "gockpt_abort_window", ctx)


def gockpt_get_scaler(ctx):
    t = ctypes.c_int64()
    s = ctypes.c_float()
    tr = ctypes.c_int64()
    _check(lib().gockpt_get_scaler(ctx, ctypes.byref(t), ctypes.byref(s), ctypes.byref(tr)), "gockpt_get_scaler",
           ctx)
    return t.value, s.value, tr.value


def gockpt_window_records(ctx, K: int) -> np.ndarray:
    out = np.zeros(int(K), dtype=RECORD_DTYPE)
    _check(lib().gockpt_window_records(ctx, out.ctypes.data, int(K)), "gockpt_window_records", ctx)
    return out


def gockpt_window_step_times(ctx, K: int) -> np.ndarray:
    """[K, 5]: prepass+finalize ms, fused update+pack kernel ms, copy-stream ms
    of the step's copies, bytes packed into the ring by the update, ms between
    the finalize and the update kernel."""
    out = np.zeros((int(K), 5), dtype=np.float64)
    _check(lib().gockpt_window_step_times(ctx, out.ctypes.data, int(K)), "gockpt_window_step_times", ctx)
    return out


def gockpt_replay_arena(K, bounds, n, arena_ptr, arena_bytes, beta1, beta2, eps, weight_decay,
                        master_out=None, exp_avg_out=None, exp_avg_sq_out=None, w_bf16_out=None,
                        nthreads: int = 0, grad_dtype: int = GOCKPT_GRAD_BF16) -> gockpt_ckpt_meta:
    b = _i64(bounds)
    meta = gockpt_ckpt_meta()
    _check(lib().gockpt_replay_arena(int(K), b.ctypes.data, int(n), arena_ptr, int(arena_bytes), float(beta1),
                                     float(beta2), float(eps), float(weight_decay), int(grad_dtype), master_out,
                                     exp_avg_out,
                                     exp_avg_sq_out, w_bf16_out, ctypes.byref(meta), int(nthreads)),
           "gockpt_replay_arena", None)
    return meta


# ---- persistence and loading ----------------------------------------------------

def _f32(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype != np.float32 or not a.flags.c_contiguous:
        raise TypeError("expected a contiguous float32 array")
    return a


def gockpt_write_checkpoint(path: str, master, exp_avg, exp_avg_sq, *, t: int = 0, tracker: int = 0,
                            scale: float = 1.0, K: int = 0, skipped: int = 0, beta1: float = 0.9,
                            beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.01,
                            user_meta: str | None = None, nthreads: int = 0, piece_bytes: int = 0) -> gockpt_io_stats:
    p, m, v = _f32(master), _f32(exp_avg), _f32(exp_avg_sq)
    if not (p.size == m.size == v.size):
        raise ValueError("arrays differ in length")
    info = gockpt_ckpt_info(n=p.size, t=int(t), tracker=int(tracker), scale=float(scale), K=int(K),
                            skipped=int(skipped), has_user=0, beta1=float(beta1), beta2=float(beta2), eps=float(eps),
                            weight_decay=float(weight_decay), piece_bytes=int(piece_bytes), data_bytes=0)
    st = gockpt_io_stats()
    _check(lib().gockpt_write_checkpoint(os.fsencode(path), p.ctypes.data, m.ctypes.data, v.ctypes.data,
                                         ctypes.byref(info), user_meta.encode() if user_meta is not None else None,
                                         int(nthreads), ctypes.byref(st)), "gockpt_write_checkpoint", None)
    return st


def gockpt_read_checkpoint_info(path: str) -> gockpt_ckpt_info:
    info = gockpt_ckpt_info()
    _check(lib().gockpt_read_checkpoint_info(os.fsencode(path), ctypes.byref(info)), "gockpt_read_checkpoint_info",
           None)
    return info


def gockpt_read_checkpoint(path: str, n: int | None = None, nthreads: int = 0):
    """(master, exp_avg, exp_avg_sq, info, stats) of a complete checkpoint."""
    if n is None:
        n = gockpt_read_checkpoint_info(path).n
    p = np.empty(int(n), np.float32)
    m = np.empty(int(n), np.float32)
    v = np.empty(int(n), np.float32)
    info, st = gockpt_ckpt_info(), gockpt_io_stats()
    _check(lib().gockpt_read_checkpoint(os.fsencode(path), int(n), p.ctypes.data, m.ctypes.data, v.ctypes.data,
                                        ctypes.byref(info), int(nthreads), ctypes.byref(st)),
           "gockpt_read_checkpoint", None)
    return p, m, v, info, st


def gockpt_read_checkpoint_user(path: str) -> str:
    ln = ctypes.c_size_t(0)
    _check(lib().gockpt_read_checkpoint_user(os.fsencode(path), None, 0, ctypes.byref(ln)),
           "gockpt_read_checkpoint_user", None)
    buf = ctypes.create_string_buffer(ln.value + 1)
    _check(lib().gockpt_read_checkpoint_user(os.fsencode(path), ctypes.addressof(buf), ln.value + 1, None),
           "gockpt_read_checkpoint_user", None)
    return buf.value.decode()


def gockpt_find_latest_checkpoint(root: str) -> str:
    buf = ctypes.create_string_buffer(4096)
    _check(lib().gockpt_find_latest_checkpoint(os.fsencode(root), ctypes.addressof(buf), 4096),
           "gockpt_find_latest_checkpoint", None)
    return os.fsdecode(buf.value)


def gockpt_persist(ctx, path: str, user_meta: str | None = None, nthreads: int = 0, async_: bool = False) -> None:
    _check(lib().gockpt_persist(ctx, os.fsencode(path), user_meta.encode() if user_meta is not None else None,
                                int(nthreads), int(bool(async_))), "gockpt_persist", ctx)


def gockpt_persist_wait(ctx) -> gockpt_io_stats:
    st = gockpt_io_stats()
    _check(lib().gockpt_persist_wait(ctx, ctypes.byref(st)), "gockpt_persist_wait", ctx)
    return st


def gockpt_load(ctx, path: str, host_ptr: int, host_bytes: int, nthreads: int = 0) -> gockpt_ckpt_info:
    info = gockpt_ckpt_info()
    _check(lib().gockpt_load(ctx, os.fsencode(path), host_ptr, int(host_bytes), int(nthreads), ctypes.byref(info)),
           "gockpt_load", ctx)
    return info


from .session import Session, StateSlab  # noqa: E402  (torch-backed buffers around the C-ABI)

__all__ = [n for n in dir() if n.startswith(("gockpt_", "GOCKPT_"))] + ["Session", "StateSlab", "GockptError", "lib",
                                                           "RECORD_DTYPE"]
