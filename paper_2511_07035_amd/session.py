"""Torch-backed buffers around one gockpt context.

PyTorch provides device memory (state, gradients, ring, workspace) and the two
streams; the pinned host arena comes from ``gockpt_host_alloc``.  Every step
of the hot path runs in the HIP library.
"""
from __future__ import annotations

import numpy as np

import mmap

from . import (RECORD_DTYPE, gockpt_abort_window, gockpt_arena_layout_ex, gockpt_backward_begin,
               gockpt_begin_window_ex, gockpt_config, gockpt_create, gockpt_destroy, gockpt_drain,
               gockpt_get_scaler, gockpt_host_alloc, gockpt_host_free, gockpt_replay_arena,
               gockpt_restore, gockpt_step, gockpt_window_records, gockpt_window_step_times,
               gockpt_workspace_bytes, host_view)


class Session:
    """One flat parameter space on one GPU with a GoCkpt context.

    master/exp_avg/exp_avg_sq are fp32 device tensors of n elements, weight
    and grad bf16 device tensors (weight may be None).  Tensors not passed are
    allocated (master zeros, moments zeros, weight = bf16(master) is the
    caller's job).  Write gradients on ``self.compute`` (or make it wait).

    staging_bytes > 0 gives the context pinned staging slots, so windows can
    use a pageable host arena (``begin_window(..., pageable=True)``) larger
    than what the host can pin.
    """

    def __init__(self, n: int, *, master=None, exp_avg=None, exp_avg_sq=None, weight=None, grad=None,
                 with_weight: bool = True, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01,
                 check_overflow=True, dynamic_scale=False, init_scale=1.0, growth_factor=2.0,
                 backoff_factor=0.5, growth_interval=1000, min_scale=1.0, init_step=0, init_tracker=0,
                 ring_bytes: int = 256 << 20, copy_bytes: int = 64 << 20, timing: bool = False,
                 staging_bytes: int = 0, copy_threads: int = 8, device: str = "cuda:0"):
        import torch

        self.torch = torch
        self.n = int(n)
        self.device = torch.device(device)
        dev = self.device

        def need(t, dtype):
            if t is None:
                return torch.zeros(self.n, dtype=dtype, device=dev)
            assert t.dtype == dtype and t.is_contiguous() and t.numel() == self.n and t.device == dev
            return t

        self.master = need(master, torch.float32)
        self.exp_avg = need(exp_avg, torch.float32)
        self.exp_avg_sq = need(exp_avg_sq, torch.float32)
        self.grad = need(grad, torch.bfloat16)
        self.weight = need(weight, torch.bfloat16) if (with_weight or weight is not None) else None
        self.hparams = dict(beta1=beta1, beta2=beta2, eps=eps, weight_decay=weight_decay)
        self.ring = torch.empty(int(ring_bytes), dtype=torch.uint8, device=dev) if ring_bytes else None
        self.workspace = torch.zeros(gockpt_workspace_bytes(self.n), dtype=torch.uint8, device=dev)
        self.compute = torch.cuda.Stream(device=dev)
        self.copy = torch.cuda.Stream(device=dev)
        # everything allocated/initialised so far is on the current stream
        self.compute.wait_stream(torch.cuda.current_stream(dev))
        self.copy.wait_stream(torch.cuda.current_stream(dev))
        cfg = gockpt_config()
        cfg.n = self.n
        cfg.master = self.master.data_ptr()
        cfg.exp_avg = self.exp_avg.data_ptr()
        cfg.exp_avg_sq = self.exp_avg_sq.data_ptr()
        cfg.weight_bf16 = self.weight.data_ptr() if self.weight is not None else None
        cfg.grad_bf16 = self.grad.data_ptr()
        cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay = beta1, beta2, eps, weight_decay
        cfg.check_overflow = int(bool(check_overflow))
        cfg.dynamic_scale = int(bool(dynamic_scale))
        cfg.init_scale = init_scale
        cfg.growth_factor = growth_factor
        cfg.backoff_factor = backoff_factor
        cfg.min_scale = min_scale
        cfg.growth_interval = int(growth_interval)
        cfg.init_step = int(init_step)
        cfg.init_tracker = int(init_tracker)
        cfg.ring = self.ring.data_ptr() if self.ring is not None else None
        cfg.ring_bytes = int(ring_bytes) if self.ring is not None else 0
        cfg.copy_bytes = int(copy_bytes)
        cfg.workspace = self.workspace.data_ptr()
        cfg.workspace_bytes = self.workspace.numel()
        cfg.compute_stream = self.compute.cuda_stream
        cfg.copy_stream = self.copy.cuda_stream
        cfg.timing = int(bool(timing))
        self.staging_ptr = gockpt_host_alloc(int(staging_bytes)) if staging_bytes else 0
        cfg.copy_threads = int(copy_threads)
        cfg.host_staging = self.staging_ptr or None
        cfg.host_staging_bytes = int(staging_bytes) if staging_bytes else 0
        self.cfg = cfg
        self.arena_ptr = 0
        self.arena_bytes = 0
        self.arena_map = None
        self.ctx = None
        try:
            self.ctx = gockpt_create(cfg)
        except Exception:
            if self.staging_ptr:
                gockpt_host_free(self.staging_ptr)
                self.staging_ptr = 0
            raise
        self.K = 0
        self.bounds = None
        self.layout = None
        self.grad_offsets = None

    # ---- window --------------------------------------------------------------
    def _free_arena(self) -> None:
        if self.arena_map is not None:
            self.arena_view = None
            self.arena_map.close()
            self.arena_map = None
        elif self.arena_ptr:
            gockpt_host_free(self.arena_ptr)
        self.arena_ptr, self.arena_bytes = 0, 0

    def ensure_arena(self, nbytes: int, pageable: bool = False) -> None:
        if self.arena_bytes >= nbytes and (self.arena_map is not None) == pageable:
            return
        self._free_arena()
        if pageable:
            # anonymous mapping (page aligned), huge pages where the kernel allows
            m = mmap.mmap(-1, int(nbytes), flags=mmap.MAP_PRIVATE | mmap.MAP_ANONYMOUS)
            if hasattr(mmap, "MADV_HUGEPAGE"):
                try:
                    m.madvise(mmap.MADV_HUGEPAGE)
                except OSError:
                    pass
            self.arena_map = m
            self.arena_view = np.frombuffer(m, dtype=np.uint8)
            self.arena_ptr = self.arena_view.ctypes.data
        else:
            self.arena_ptr = gockpt_host_alloc(nbytes)
        self.arena_bytes = int(nbytes)

    def begin_window(self, bounds, replay_every: int = 0, pageable: bool = False, replay_threads: int = 0) -> None:
        """Open a window.  pageable: the arena lives in ordinary (pageable)
        host memory reached through the staging slots; replay_every = R:
        replay every R landed steps during the window (0: at restore)."""
        b = np.ascontiguousarray(bounds, dtype=np.int64)
        K = b.size - 1
        lay, goff = gockpt_arena_layout_ex(K, b, self.n, replay_every)
        self.ensure_arena(lay.total, pageable)
        gockpt_begin_window_ex(self.ctx, K, b, self.arena_ptr, self.arena_bytes, replay_every, replay_threads)
        self.K, self.bounds, self.layout, self.grad_offsets = K, b, lay, goff

    def backward_begin(self, stream=None) -> None:
        gockpt_backward_begin(self.ctx, stream.cuda_stream if stream is not None else None)

    def step(self, lr: float) -> None:
        gockpt_step(self.ctx, lr)

    def drain(self, blocking: bool = True):
        return gockpt_drain(self.ctx, blocking)

    def restore(self, nthreads: int = 0, out=None):
        """Replay into the arena (out=None) or into host numpy arrays
        out=(master, exp_avg, exp_avg_sq, w_or_None).  Returns the meta."""
        if out is None:
            return gockpt_restore(self.ctx, None, None, None, None, nthreads)
        p, m, v, w = out
        return gockpt_restore(self.ctx, p.ctypes.data, m.ctypes.data, v.ctypes.data,
                              w.ctypes.data if w is not None else None, nthreads)

    def abort_window(self) -> None:
        gockpt_abort_window(self.ctx)

    def records(self) -> np.ndarray:
        return gockpt_window_records(self.ctx, self.K)

    def step_times(self) -> np.ndarray:
        return gockpt_window_step_times(self.ctx, self.K)

    def scaler(self):
        return gockpt_get_scaler(self.ctx)

    # ---- arena views (no copies) ---------------------------------------------
    def arena_state(self):
        lay = self.layout
        f = lambda off: host_view(self.arena_ptr, self.arena_bytes, np.float32, int(off), self.n)
        return f(lay.master), f(lay.exp_avg), f(lay.exp_avg_sq)

    def arena_grads(self, s: int) -> np.ndarray:
        """bf16 bits of the gradient block of window step s (elements [0, bounds[s-1]))."""
        return host_view(self.arena_ptr, self.arena_bytes, np.uint16, int(self.grad_offsets[s - 1]),
                         int(self.bounds[s - 1]))

    def arena_records(self) -> np.ndarray:
        return host_view(self.arena_ptr, self.arena_bytes, RECORD_DTYPE, int(self.layout.records), self.K)

    def replay_arena(self, nthreads: int = 0, out=None):
        """Replay the drained arena with the context-free entry point."""
        hp = self.hparams
        if out is None:
            ptrs = (None, None, None, None)
        else:
            p, m, v, w = out
            ptrs = (p.ctypes.data, m.ctypes.data, v.ctypes.data, w.ctypes.data if w is not None else None)
        return gockpt_replay_arena(self.K, self.bounds, self.n, self.arena_ptr, self.arena_bytes, hp["beta1"],
                                   hp["beta2"], hp["eps"], hp["weight_decay"], *ptrs, nthreads=nthreads)

    # ---- device state to host --------------------------------------------------
    def state_to_host(self):
        """Synchronise the compute stream; copies of (master, m, v, w bits)."""
        torch = self.torch
        self.compute.synchronize()
        p = self.master.cpu().numpy()
        m = self.exp_avg.cpu().numpy()
        v = self.exp_avg_sq.cpu().numpy()
        w = self.weight.view(torch.int16).cpu().numpy().view(np.uint16) if self.weight is not None else None
        return p, m, v, w

    def close(self) -> None:
        if getattr(self, "ctx", None):
            gockpt_destroy(self.ctx)
            self.ctx = None
        if getattr(self, "arena_ptr", 0):
            self._free_arena()
        if getattr(self, "staging_ptr", 0):
            gockpt_host_free(self.staging_ptr)
            self.staging_ptr = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
