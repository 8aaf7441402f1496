"""CPU oracle for the GoCkpt hot path (arXiv 2511.07035) -- ctypes wrapper.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library never loads it, and it shares no code with the product library.

The arithmetic lives in ``gockpt_oracle.c`` (plain C, fp32 per element, one
rounded operation per statement, ``-ffp-contract=off``).  This module only
builds that file with gcc and marshals numpy arrays into it.

Functions follow the paper:
  * ``adamw_step`` / ``sync_run``: mixed-precision AdamW with loss-scale skip
    logic (Sec. 2.2; AdamW named in Sec. 4.3.1); ``sync_run`` is the checkpoint
    a blocking snapshot after the window's last step would hold (Sec. 2.1).
  * ``window_capture``: what the multi-step window sends -- part s after step
    s, plus the gradients of parts already sent (Sec. 4.2.1).
  * ``replay_restore``: the CPU reconstruction of a consistent checkpoint
    from those pieces (Sec. 4.3.1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gockpt_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-Wall"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = ctypes.CDLL(_LIB)
        _declare(_lib)
    return _lib


class Scalars(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in
                ("b1", "b2", "omb1", "omb2", "eps", "decay", "step_size", "sqrt_bc2", "inv_scale")]


class HParams(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("check_overflow", ctypes.c_int32), ("dynamic_scale", ctypes.c_int32),
                ("growth_factor", ctypes.c_float), ("backoff_factor", ctypes.c_float),
                ("min_scale", ctypes.c_float), ("grad_fp16", ctypes.c_int32),
                ("growth_interval", ctypes.c_int64)]


class Scaler(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int64), ("scale", ctypes.c_float), ("pad_", ctypes.c_int32),
                ("tracker", ctypes.c_int64)]


class Record(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int64), ("skip", ctypes.c_int32), ("scale_used", ctypes.c_float),
                ("lr", ctypes.c_float), ("pad_", ctypes.c_int32), ("gnorm2", ctypes.c_double)]


_P = ctypes.c_void_p


def _declare(L):
    L.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
    L.oracle_bf16_to_f32.restype = ctypes.c_float
    L.oracle_fp16_to_f32.argtypes = [ctypes.c_uint16]
    L.oracle_fp16_to_f32.restype = ctypes.c_float
    L.oracle_bf16_rne.argtypes = [ctypes.c_float]
    L.oracle_bf16_rne.restype = ctypes.c_uint16
    L.oracle_bf16_rne_array.argtypes = [ctypes.c_size_t, _P, _P]
    L.oracle_bf16_rne_array.restype = None
    L.oracle_powi.argtypes = [ctypes.c_double, ctypes.c_int64]
    L.oracle_powi.restype = ctypes.c_double
    L.oracle_step_scalars.argtypes = [ctypes.c_double] * 4 + [ctypes.c_float, ctypes.c_int64,
                                                             ctypes.c_float, ctypes.POINTER(Scalars)]
    L.oracle_step_scalars.restype = None
    L.oracle_any_nonfinite.argtypes = [ctypes.c_size_t, _P, ctypes.c_int]
    L.oracle_any_nonfinite.restype = ctypes.c_int
    L.oracle_grad_norm2.argtypes = [ctypes.c_size_t, _P, ctypes.c_float, ctypes.c_int]
    L.oracle_grad_norm2.restype = ctypes.c_double
    L.oracle_adamw_step.argtypes = [ctypes.c_size_t, _P, _P, _P, _P, _P, ctypes.c_float, ctypes.c_int,
                                    ctypes.POINTER(HParams), ctypes.POINTER(Scaler), ctypes.POINTER(Record)]
    L.oracle_adamw_step.restype = None
    L.oracle_sync_run.argtypes = [ctypes.c_size_t, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P,
                                  ctypes.POINTER(HParams), ctypes.POINTER(Scaler), _P]
    L.oracle_sync_run.restype = None
    L.oracle_sent_offset.argtypes = [_P, ctypes.c_int]
    L.oracle_sent_offset.restype = ctypes.c_int64
    L.oracle_window_capture.argtypes = [ctypes.c_size_t, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P,
                                        ctypes.POINTER(HParams), ctypes.POINTER(Scaler), _P,
                                        _P, _P, _P, _P]
    L.oracle_window_capture.restype = None
    L.oracle_replay_restore.argtypes = [ctypes.c_size_t, ctypes.c_int, _P, _P, _P, _P, _P, _P,
                                        ctypes.POINTER(HParams), _P, _P, _P, _P]
    L.oracle_replay_restore.restype = None


@dataclass
class AdamWConfig:
    """Optimizer and loss-scaler settings (defaults: the 1.3B/16.7M configs)."""
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    check_overflow: bool = True
    dynamic_scale: bool = False
    init_scale: float = 1.0
    growth_factor: float = 2.0
    backoff_factor: float = 0.5
    growth_interval: int = 1000
    min_scale: float = 1.0
    grad_dtype: str = "bf16"  # or "fp16" (Sec. 2.2: FP16 or BF16 gradients)

    def hparams(self) -> HParams:
        if self.grad_dtype not in ("bf16", "fp16"):
            raise ValueError(self.grad_dtype)
        return HParams(self.beta1, self.beta2, self.eps, self.weight_decay,
                       int(self.check_overflow), int(self.dynamic_scale),
                       self.growth_factor, self.backoff_factor, self.min_scale, int(self.grad_dtype == "fp16"),
                       self.growth_interval)


RECORD_DTYPE = np.dtype([("t", "<i8"), ("skip", "<i4"), ("scale_used", "<f4"),
                         ("lr", "<f4"), ("pad_", "<i4"), ("gnorm2", "<f8")])
assert RECORD_DTYPE.itemsize == ctypes.sizeof(Record)


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def _u16(a):
    return np.ascontiguousarray(a, dtype=np.uint16)


def bf16_to_f32(b: int) -> float:
    return lib().oracle_bf16_to_f32(int(b))


def fp16_to_f32(b: int) -> float:
    return lib().oracle_fp16_to_f32(int(b))


def bf16_rne(x: float) -> int:
    return int(lib().oracle_bf16_rne(float(x)))


def bf16_rne_array(x: np.ndarray) -> np.ndarray:
    x = _f32(x)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_bf16_rne_array(x.size, _ptr(x), _ptr(out))
    return out


def powi(beta: float, t: int) -> float:
    return lib().oracle_powi(float(beta), int(t))


def step_scalars(cfg: AdamWConfig, lr: float, t: int, scale: float) -> Scalars:
    s = Scalars()
    lib().oracle_step_scalars(cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay,
                              float(lr), int(t), float(scale), ctypes.byref(s))
    return s


def any_nonfinite(g: np.ndarray, grad_dtype: str = "bf16") -> bool:
    g = _u16(g)
    return bool(lib().oracle_any_nonfinite(g.size, _ptr(g), int(grad_dtype == "fp16")))


def grad_norm2(g: np.ndarray, inv_scale: float, grad_dtype: str = "bf16") -> float:
    g = _u16(g)
    return lib().oracle_grad_norm2(g.size, _ptr(g), float(inv_scale), int(grad_dtype == "fp16"))


class State:
    """Full optimizer state of the flat parameter space, fp32 + bf16 weights,
    plus the loss-scaler state (t, scale, tracker)."""

    def __init__(self, p, m=None, v=None, w=None, t=0, scale=1.0, tracker=0):
        self.p = _f32(p).copy()
        self.m = np.zeros_like(self.p) if m is None else _f32(m).copy()
        self.v = np.zeros_like(self.p) if v is None else _f32(v).copy()
        self.w = bf16_rne_array(self.p) if w is None else _u16(w).copy()
        self.scaler = Scaler(int(t), float(scale), 0, int(tracker))

    def copy(self) -> "State":
        s = State(self.p, self.m, self.v, self.w, self.scaler.t, self.scaler.scale, self.scaler.tracker)
        return s

    @property
    def t(self):
        return self.scaler.t

    @property
    def scale(self):
        return self.scaler.scale

    @property
    def tracker(self):
        return self.scaler.tracker


def adamw_step(state: State, g: np.ndarray, cfg: AdamWConfig, lr: float | None = None,
               nonfinite: int = -1) -> np.ndarray:
    """One step in place; returns the step's record (structured array of 1)."""
    g = _u16(g)
    assert g.size == state.p.size
    rec = np.zeros(1, dtype=RECORD_DTYPE)
    hp = cfg.hparams()
    lib().oracle_adamw_step(state.p.size, _ptr(state.p), _ptr(state.m), _ptr(state.v), _ptr(state.w),
                            _ptr(g), float(cfg.lr if lr is None else lr), int(nonfinite),
                            ctypes.byref(hp), ctypes.byref(state.scaler),
                            ctypes.cast(_ptr(rec), ctypes.POINTER(Record)))
    return rec


def _lrs(cfg, K, lrs):
    if lrs is None:
        lrs = [cfg.lr] * K
    a = np.ascontiguousarray(lrs, dtype=np.float32)
    assert a.size == K
    return a


def _nf(nonfinite, K):
    if nonfinite is None:
        return None
    a = np.ascontiguousarray(nonfinite, dtype=np.int32)
    assert a.size == K
    return a


def sync_run(state: State, grads: np.ndarray, cfg: AdamWConfig, lrs=None, nonfinite=None) -> np.ndarray:
    """K synchronous steps in place (grads: [K, n] uint16).  Returns K records."""
    grads = _u16(grads)
    K, n = grads.shape
    assert n == state.p.size
    recs = np.zeros(K, dtype=RECORD_DTYPE)
    hp = cfg.hparams()
    lr_a = _lrs(cfg, K, lrs)
    nf = _nf(nonfinite, K)
    lib().oracle_sync_run(n, K, _ptr(state.p), _ptr(state.m), _ptr(state.v), _ptr(state.w),
                          _ptr(grads), _ptr(lr_a), _ptr(nf), ctypes.byref(hp),
                          ctypes.byref(state.scaler), _ptr(recs))
    return recs


def sent_offsets(bounds) -> np.ndarray:
    """Offset (elements) of step s's gradient block, s = 1..K, and the total."""
    b = np.ascontiguousarray(bounds, dtype=np.int64)
    K = b.size - 1
    return np.array([lib().oracle_sent_offset(_ptr(b), s) for s in range(1, K + 2)], dtype=np.int64)


@dataclass
class Capture:
    snap_p: np.ndarray
    snap_m: np.ndarray
    snap_v: np.ndarray
    sent: np.ndarray
    records: np.ndarray
    bounds: np.ndarray


def window_capture(state: State, grads: np.ndarray, bounds, cfg: AdamWConfig, lrs=None,
                   nonfinite=None) -> Capture:
    """Run a K-step window in place and return what it sends (Sec. 4.2.1)."""
    grads = _u16(grads)
    K, n = grads.shape
    b = np.ascontiguousarray(bounds, dtype=np.int64)
    assert b.size == K + 1 and b[0] == 0 and b[-1] == n
    offs = sent_offsets(b)
    sent = np.zeros(int(offs[-1]), dtype=np.uint16)
    snap_p = np.zeros(n, dtype=np.float32)
    snap_m = np.zeros(n, dtype=np.float32)
    snap_v = np.zeros(n, dtype=np.float32)
    recs = np.zeros(K, dtype=RECORD_DTYPE)
    hp = cfg.hparams()
    lr_a = _lrs(cfg, K, lrs)
    nf = _nf(nonfinite, K)
    lib().oracle_window_capture(n, K, _ptr(b), _ptr(state.p), _ptr(state.m), _ptr(state.v),
                                _ptr(state.w), _ptr(grads), _ptr(lr_a), _ptr(nf), ctypes.byref(hp),
                                ctypes.byref(state.scaler), _ptr(recs),
                                _ptr(snap_p), _ptr(snap_m), _ptr(snap_v), _ptr(sent))
    return Capture(snap_p, snap_m, snap_v, sent, recs, b)


def replay_restore(cap: Capture, cfg: AdamWConfig):
    """CPU reconstruction (Sec. 4.3.1).  Returns (p, m, v, w)."""
    n = cap.snap_p.size
    K = cap.bounds.size - 1
    out_p = np.empty(n, dtype=np.float32)
    out_m = np.empty(n, dtype=np.float32)
    out_v = np.empty(n, dtype=np.float32)
    out_w = np.empty(n, dtype=np.uint16)
    recs = np.ascontiguousarray(cap.records)
    hp = cfg.hparams()
    lib().oracle_replay_restore(n, K, _ptr(cap.bounds), _ptr(cap.snap_p), _ptr(cap.snap_m),
                                _ptr(cap.snap_v), _ptr(_u16(cap.sent)), _ptr(recs), ctypes.byref(hp),
                                _ptr(out_p), _ptr(out_m), _ptr(out_v), _ptr(out_w))
    return out_p, out_m, out_v, out_w
