"""Torch-backed buffers around one gockpt context.

PyTorch provides device memory (state, gradients, ring, workspace) and the two
streams; the pinned host arena comes from ``gockpt_host_alloc``.  Every step
of the hot path runs in the HIP library.
"""
from __future__ import annotations

import mmap

import numpy as np

from . import (GOCKPT_GRAD_BF16, GOCKPT_GRAD_FP16, RECORD_DTYPE, GockptError, gockpt_abort_window,
               gockpt_arena_layout_ex, gockpt_backward_begin, gockpt_begin_window_ex, gockpt_config, gockpt_create, gockpt_create_noalloc, gockpt_destroy, gockpt_drain,
               gockpt_get_scaler, gockpt_host_alloc, gockpt_host_free, gockpt_load, gockpt_persist,
               gockpt_persist_wait, gockpt_replay_arena, gockpt_restore, gockpt_restore_async, gockpt_restore_wait,
               gockpt_scan_grads, gockpt_step, gockpt_window_records,
               gockpt_window_step_times, gockpt_workspace_bytes, host_view)


class StateSlab:
    """The device state of n elements laid out for MI355X HBM.

    The fused update streams five arrays at the same index at once (master,
    exp_avg, exp_avg_sq read and written; gradients read; bf16 weights
    written).  Measured on MI355X with the update's memory twin: the five
    arrays within ~20 GiB of each other run the 1:1 read/write mix at ~5.3
    TB/s, 24-40 GiB apart at ~5.8 TB/s, 48-56 GiB apart at ~6.2 TB/s.
    Separate allocations give no control over where arrays land (the caching
    allocator packs them), so this class reserves one slab over most of HBM,
    puts the five arrays `spacing` bytes apart (48 GiB by default) and hands
    out the space between them with take() -- for the staging ring and any
    other buffers -- so nothing is wasted.

    placement="packed" allocates the five arrays back to back with ordinary
    torch allocations instead (no reservation).
    """

    def __init__(self, n: int, *, placement: str = "slab", reserve_bytes: int = 16 << 30,
                 slab_bytes: int | None = None, spacing: int = 48 << 30, device: str = "cuda:0",
                 grad_dtype: str = "bf16"):
        import torch

        self.n = int(n)
        self.placement = placement
        dev = torch.device(device)
        sizes = [4 * self.n] * 3 + [2 * self.n] * 2
        dtypes = [torch.float32] * 3 + [torch.float16 if grad_dtype == "fp16" else torch.bfloat16, torch.bfloat16]
        self.gaps = []
        self.slab = None
        if placement == "packed":
            self.arrays = [torch.empty(self.n, dtype=dt, device=dev) for dt in dtypes]
            self.offsets = None
            return
        if placement != "slab":
            raise ValueError(placement)
        if slab_bytes is None:
            slab_bytes = torch.cuda.mem_get_info(dev)[0] - int(reserve_bytes)
        slab_bytes = int(slab_bytes) // (2 << 20) * (2 << 20)
        need = sum(self._round(x) for x in sizes)
        if slab_bytes < need:
            raise MemoryError(f"slab of {slab_bytes} B cannot hold the {need} B state")
        # spacing: as asked, but the five arrays must fit
        step = min(int(spacing), (slab_bytes - self._round(sizes[-1])) // 4)
        step = max(step, max(self._round(x) for x in sizes)) // 256 * 256
        self.slab = torch.empty(slab_bytes, dtype=torch.uint8, device=dev)
        self.offsets = [k * step for k in range(5)]
        self.arrays = []
        cur = 0
        for off, nb, dt in zip(self.offsets, sizes, dtypes):
            if off > cur:
                self.gaps.append([cur, off - cur])
            self.arrays.append(self.slab[off:off + nb].view(dt))
            cur = self._round(off + nb)
        if slab_bytes > cur:
            self.gaps.append([cur, slab_bytes - cur])

    @staticmethod
    def _round(x: int, a: int = 256) -> int:
        return (int(x) + a - 1) // a * a

    @property
    def master(self):
        return self.arrays[0]

    @property
    def exp_avg(self):
        return self.arrays[1]

    @property
    def exp_avg_sq(self):
        return self.arrays[2]

    @property
    def grad(self):
        return self.arrays[3]

    @property
    def weight(self):
        return self.arrays[4]

    def take(self, nbytes: int):
        """A uint8 tensor of nbytes (256-byte aligned) from the space between
        the arrays, or None when none is left (or placement is packed)."""
        nbytes = self._round(nbytes)
        for gap in self.gaps:
            if gap[1] >= nbytes:
                t = self.slab[gap[0]:gap[0] + nbytes]
                gap[0] += nbytes
                gap[1] -= nbytes
                return t
        return None


class Session:
    """One flat parameter space on one GPU with a GoCkpt context.

    master/exp_avg/exp_avg_sq are fp32 device tensors of n elements, weight
    and grad bf16 device tensors (weight may be None).  Tensors not passed are
    allocated (master zeros, moments zeros, weight = bf16(master) is the
    caller's job).  Write gradients on ``self.compute`` (or make it wait).

    staging_bytes > 0 gives the context pinned staging slots, so windows can
    use a pageable host arena (``begin_window(..., pageable=True)``) larger
    than what the host can pin.

    grad_norm=False stops the per-step gradient norm; found_inf (a
    one-element float32 device tensor the caller's own overflow test writes
    before each step, as a gradient scaler's found-inf flag) takes the skip
    decisions.  With both, or with check_overflow=False and grad_norm=False,
    no prepass reads the gradients.  scan_grads() moves the library's own
    test into the backward, bucket by bucket.
    """

    def __init__(self, n: int, *, master=None, exp_avg=None, exp_avg_sq=None, weight=None, grad=None,
                 with_weight: bool = True, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01,
                 check_overflow=True, dynamic_scale=False, init_scale=1.0, growth_factor=2.0,
                 backoff_factor=0.5, growth_interval=1000, min_scale=1.0, init_step=0, init_tracker=0,
                 ring_bytes: int = 256 << 20, copy_bytes: int = 64 << 20, timing: bool = False,
                 staging_bytes: int = 0, copy_threads: int = 8, ring=None, device: str = "cuda:0",
                 grad_dtype: str = "bf16", grad_norm: bool = True, found_inf=None, noalloc: bool = False):
        import torch

        self.torch = torch
        self.n = int(n)
        self.device = torch.device(device)
        dev = self.device

        def need(t, dtype):
            if t is None:
                return torch.zeros(self.n, dtype=dtype, device=dev)
            if not (t.dtype == dtype and t.is_contiguous() and t.numel() == self.n and t.device == dev):
                raise ValueError(f"expected a contiguous {dtype} tensor of {self.n} elements on {dev}, got "
                                 f"{t.dtype} {tuple(t.shape)} on {t.device}")
            return t

        self.master = need(master, torch.float32)
        self.exp_avg = need(exp_avg, torch.float32)
        self.exp_avg_sq = need(exp_avg_sq, torch.float32)
        if grad_dtype not in ("bf16", "fp16"):
            raise ValueError(f"grad_dtype {grad_dtype!r}: bf16 or fp16")
        self.grad_dtype = grad_dtype
        self.grad = need(grad, torch.float16 if grad_dtype == "fp16" else torch.bfloat16)
        self.weight = need(weight, torch.bfloat16) if (with_weight or weight is not None) else None
        self.hparams = dict(beta1=beta1, beta2=beta2, eps=eps, weight_decay=weight_decay)
        if ring is not None:  # caller-provided device bytes (e.g. StateSlab.take)
            if not (ring.dtype == torch.uint8 and ring.is_contiguous() and ring.device == dev):
                raise ValueError("ring must be a contiguous uint8 tensor on the session's device")
            ring_bytes = ring.numel() // 256 * 256
            self.ring = ring[:ring_bytes]
        else:
            self.ring = torch.empty(int(ring_bytes), dtype=torch.uint8, device=dev) if ring_bytes else None
        # noalloc: the context uses the library's static scratch workspace
        # (gockpt_create_noalloc) instead of one allocated here
        self.noalloc = bool(noalloc)
        self.workspace = None if self.noalloc else torch.zeros(gockpt_workspace_bytes(self.n), dtype=torch.uint8,
                                                               device=dev)
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
        cfg.grad16 = self.grad.data_ptr()
        cfg.grad_dtype = GOCKPT_GRAD_FP16 if grad_dtype == "fp16" else GOCKPT_GRAD_BF16
        cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay = beta1, beta2, eps, weight_decay
        cfg.check_overflow = int(bool(check_overflow))
        cfg.grad_norm_off = 0 if grad_norm else 1
        if found_inf is not None:  # a one-element float32 device tensor the caller's overflow test writes
            if not (found_inf.dtype == torch.float32 and found_inf.numel() == 1 and found_inf.device == dev):
                raise ValueError("found_inf must be a one-element float32 tensor on the session's device")
            cfg.found_inf = found_inf.data_ptr()
        self.found_inf = found_inf
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
        cfg.workspace = self.workspace.data_ptr() if self.workspace is not None else None
        cfg.workspace_bytes = self.workspace.numel() if self.workspace is not None else 0
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
            self.ctx = gockpt_create_noalloc(cfg) if self.noalloc else gockpt_create(cfg)
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

    def begin_window(self, bounds, replay_every: int = 0, pageable: bool = False, replay_threads: int = 0,
                     wait_policy: int = 0, ring_off: bool = False, late_plan: int = 0, timing: bool = True,
                     defer_copies: bool = False) -> None:
        """Open a window.  pageable: the arena lives in ordinary (pageable)
        host memory reached through the staging slots; replay_every = R:
        replay every R landed steps during the window (0: at restore);
        wait_policy: GOCKPT_WAIT_LAZY / _GRADS / _ALL; ring_off: copy
        everything straight from the live buffers; late_plan: the ring plan,
        GOCKPT_RING_QUERY (0), _HOST_WAIT (1 or True: step() blocks until the
        device reaches the update) or _DEVICE_WAIT (2: the whole ring, the
        device waits for the copies of the ranges reused); timing=False:
        no timing events in this window (a context made with timing=True
        otherwise records them around every window step); defer_copies: a
        step's copies are queued at the next library call (backward_begin,
        step or drain) rather than by step() itself."""
        b = np.ascontiguousarray(bounds, dtype=np.int64)
        K = b.size - 1
        lay, goff = gockpt_arena_layout_ex(K, b, self.n, replay_every)
        self._join_restore()  # a background restore or persist may still read the arena
        self._join_persist()
        self.ensure_arena(lay.total, pageable)
        gockpt_begin_window_ex(self.ctx, K, b, self.arena_ptr, self.arena_bytes, replay_every, replay_threads,
                               wait_policy, ring_off, late_plan, timing, defer_copies)
        self.K, self.bounds, self.layout, self.grad_offsets = K, b, lay, goff

    def backward_begin(self, stream=None) -> None:
        gockpt_backward_begin(self.ctx, stream.cuda_stream if stream is not None else None)

    def scan_grads(self, begin: int, end: int, stream=None) -> None:
        """Overflow test and norm of gradient elements [begin, end) for the
        coming step, on `stream` (a torch stream; None: the compute stream)."""
        gockpt_scan_grads(self.ctx, begin, end, stream.cuda_stream if stream is not None else None)

    def step(self, lr: float) -> None:
        gockpt_step(self.ctx, lr)

    def drain(self, blocking: bool = True):
        return gockpt_drain(self.ctx, blocking)

    def _out_ptrs(self, out):
        """Host pointers of out = (master, exp_avg, exp_avg_sq, w_or_None):
        float32, float32, float32 and uint16 numpy arrays of n elements, C-
        contiguous and writeable (the replay writes n elements through each
        pointer); None for all four restores in place in the arena."""
        if out is None:
            return (None, None, None, None)
        if len(out) != 4:
            raise ValueError("out must be (master, exp_avg, exp_avg_sq, w_or_None)")
        ptrs = []
        for a, dt, name in zip(out, (np.float32, np.float32, np.float32, np.uint16),
                               ("master", "exp_avg", "exp_avg_sq", "w")):
            if a is None and name == "w":
                ptrs.append(None)
                continue
            if not (isinstance(a, np.ndarray) and a.dtype == dt and a.size == self.n and a.flags.c_contiguous
                    and a.flags.writeable):
                raise ValueError(f"out {name}: expected a writeable C-contiguous {np.dtype(dt).name} array of "
                                 f"{self.n} elements, got {type(a).__name__} "
                                 f"{getattr(a, 'dtype', None)} {getattr(a, 'shape', None)}")
            ptrs.append(a.ctypes.data)
        return tuple(ptrs)

    def restore(self, nthreads: int = 0, out=None, async_: bool = False):
        """Replay into the arena (out=None) or into host numpy arrays
        out=(master, exp_avg, exp_avg_sq, w_or_None).  Returns the meta, or
        with async_=True starts the replay in a library thread and returns
        None (plain steps may run meanwhile; restore_wait() gives the meta)."""
        ptrs = self._out_ptrs(out)
        if async_:
            gockpt_restore_async(self.ctx, *ptrs, nthreads=nthreads)
            self._restore_out = out  # the arrays stay alive until the wait
            self._restoring = True
            return None
        return gockpt_restore(self.ctx, *ptrs, nthreads)

    def restore_wait(self):
        try:
            return gockpt_restore_wait(self.ctx)
        finally:
            self._restore_out = None
            self._restoring = False

    def _join_restore(self) -> None:
        """A background restore reads the arena: wait for it before the arena
        is reallocated or reused (its failure surfaces at the next call)."""
        if getattr(self, "_restoring", False):
            try:
                self.restore_wait()
            except GockptError as e:
                self.restore_error = e

    def persist(self, path: str, user_meta: str | None = None, nthreads: int = 0, async_: bool = False) -> None:
        """Write the checkpoint the last in-place restore left in the arena."""
        gockpt_persist(self.ctx, path, user_meta, nthreads, async_)

    def persist_wait(self):
        return gockpt_persist_wait(self.ctx)

    def _join_persist(self) -> None:
        """Wait for a background persist; its failure is kept in
        persist_error (gockpt_persist_wait reports it as well)."""
        try:
            gockpt_persist_wait(self.ctx)
        except GockptError as e:
            self.persist_error = e

    def load(self, path: str, nthreads: int = 0):
        """Load a checkpoint into the device state (through the arena when it
        is large enough, else a temporary host buffer)."""
        need = 12 * self.n
        self._join_restore()
        if self.arena_ptr and self.arena_bytes >= need:
            return gockpt_load(self.ctx, path, self.arena_ptr, self.arena_bytes, nthreads)
        buf = np.empty(max(need, 4), dtype=np.uint8)
        return gockpt_load(self.ctx, path, buf.ctypes.data, buf.nbytes, nthreads)

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
        ptrs = self._out_ptrs(out)
        return gockpt_replay_arena(self.K, self.bounds, self.n, self.arena_ptr, self.arena_bytes, hp["beta1"],
                                   hp["beta2"], hp["eps"], hp["weight_decay"], *ptrs, nthreads=nthreads,
                                   grad_dtype=GOCKPT_GRAD_FP16 if self.grad_dtype == "fp16" else GOCKPT_GRAD_BF16)

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
