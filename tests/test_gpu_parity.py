"""Parity of the HIP path (through the C-ABI) with the CPU oracle, bit for bit.

Every case drives a Session (libgockpt.so) and the oracle on the same seeded
inputs and compares, after every window step, the device state (master,
exp_avg, exp_avg_sq, bf16 weights) with the oracle's synchronous state; after
the drain, the host arena (the part sent at each step and the gradient blocks)
with the oracle's window capture; after the restore, the replayed checkpoint
with the oracle's synchronous state after the last step (Sec. 4.3.1).
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bits_equal, assert_bits_equal_nan, load_state, to_device_grad16

pytestmark = pytest.mark.gpu


def _run_window(n, K, bounds, *, seed, ring_bytes, copy_bytes=64 << 20, dynamic=False, inf_steps=(),
                law="normal", lrs=None, with_weight=True, p0=None, m0=None, v0=None, grads=None,
                init_scale=None, per_step=True, nthreads=8, pageable=False, staging_slots=0, replay_every=0,
                timing=False, wait_policy=0, ring_off=False, late_plan=False, grad_dtype="bf16", hp=None,
                check_overflow=True, grad_norm=True, nan_equiv=False, found_inf=None, scan_buckets=None,
                defer_copies=False):
    import torch
    from paper_2511_07035_amd import Session

    print(f"[case] n={n} K={K} seed={seed} ring={ring_bytes} dynamic={dynamic} inf={inf_steps} "
          f"pageable={pageable} slots={staging_slots} replay_every={replay_every} wait={wait_policy} "
          f"ring_off={ring_off} late_plan={late_plan} grads={grad_dtype} defer={defer_copies}", flush=True)
    eq = assert_bits_equal_nan if nan_equiv else assert_bits_equal
    scale0 = init_scale if init_scale is not None else (65536.0 if dynamic else 1.0)
    cfg = oracle.AdamWConfig(dynamic_scale=dynamic, init_scale=scale0, grad_dtype=grad_dtype,
                             check_overflow=check_overflow, **(hp or {}))
    if lrs is None:
        lrs = np.full(K, cfg.lr, dtype=np.float32)
    if p0 is None:
        p0 = synth.master_cpu(n, seed)
    if grads is None:
        sched = synth.DYNSCALE_SCHEDULE if dynamic else {}
        grads = np.stack([synth.grads_cpu(n, seed, s, law=law, scale=sched.get(s, scale0),
                                          plant_inf=s in inf_steps, dtype=grad_dtype) for s in range(1, K + 1)])
    sync = oracle.State(p0, m0, v0, scale=scale0)
    win = oracle.State(p0, m0, v0, scale=scale0)
    # a caller-side overflow flag decides the skips (the oracle takes the same decisions)
    nf = None if found_inf is None else [int(f != 0) for f in found_inf]
    cap = oracle.window_capture(win, grads, bounds, cfg, lrs=lrs, nonfinite=nf)
    fi = None if found_inf is None else torch.zeros(1, dtype=torch.float32, device="cuda")

    sess = Session(n, with_weight=with_weight, dynamic_scale=dynamic, init_scale=scale0,
                   ring_bytes=ring_bytes, copy_bytes=copy_bytes, staging_bytes=staging_slots * copy_bytes,
                   copy_threads=3, timing=timing, grad_dtype=grad_dtype, check_overflow=check_overflow,
                   grad_norm=grad_norm, found_inf=fi,
                   **{k: v for k, v in (hp or {}).items() if k != "lr"})
    try:
        load_state(sess, p0, m0, v0, w=sync.w)
        sess.begin_window(bounds, replay_every=replay_every, pageable=pageable, wait_policy=wait_policy,
                          ring_off=ring_off, late_plan=late_plan, defer_copies=defer_copies)
        for s in range(1, K + 1):
            sess.backward_begin()
            to_device_grad16(sess, grads[s - 1])
            if fi is not None:
                with torch.cuda.stream(sess.compute):
                    fi.fill_(float(found_inf[s - 1]))
            if scan_buckets is not None:
                # the buckets as a backward would finish them: last first, on
                # a side stream ordered after the gradient writes
                side = torch.cuda.Stream()
                side.wait_stream(sess.compute)
                for a, b in reversed(list(zip(scan_buckets[:-1], scan_buckets[1:]))):
                    sess.scan_grads(a, b, stream=side)
            sess.step(float(lrs[s - 1]))
            rec = oracle.adamw_step(sync, grads[s - 1], cfg, lr=float(lrs[s - 1]),
                                    nonfinite=-1 if nf is None else nf[s - 1])
            if per_step or s == K:
                p, m, v, w = sess.state_to_host()
                eq(p, sync.p, f"master after step {s}")
                eq(m, sync.m, f"exp_avg after step {s}")
                eq(v, sync.v, f"exp_avg_sq after step {s}")
                if with_weight:
                    eq(w, sync.w, f"bf16 weights after step {s}")
        stats = sess.drain(blocking=True)
        assert stats.steps_done == K
        if timing:
            times = sess.step_times()
            assert times.shape == (K, 5) and np.all(times[:, :2] > 0) and np.all(times[:, 4] >= 0)
            assert int(times[:, 3].sum()) == stats.bytes_ring  # per-step ring bytes add up
        recs = sess.records()
        assert list(recs["t"]) == list(cap.records["t"])
        assert list(recs["skip"]) == list(cap.records["skip"])
        assert list(recs["scale_used"]) == list(cap.records["scale_used"])
        assert list(recs["window_step"]) == list(range(1, K + 1))
        # the device squares in fp32: a gradient above sqrt(FLT_MAX) makes the
        # telemetry norm inf there, while the oracle sums in fp64
        dev_n, ora_n = recs["gnorm2"], cap.records["gnorm2"]
        if not grad_norm:
            assert np.all(dev_n == -1.0)
        else:
            fin = np.isfinite(dev_n)
            assert np.all(ora_n[~fin] >= 3.4e38) or np.all(~np.isfinite(ora_n[~fin]))
            np.testing.assert_allclose(dev_n[fin], ora_n[fin], rtol=1e-5)
        ap, am, av = sess.arena_state()
        if 0 < replay_every < K:
            # the window already replayed every step: the arena holds the checkpoint
            eq(ap, sync.p, "arena master after the in-window replay")
            eq(am, sync.m, "arena exp_avg after the in-window replay")
            eq(av, sync.v, "arena exp_avg_sq after the in-window replay")
        else:
            # what reached the host: part j as it stood after step j ...
            eq(ap, cap.snap_p, "arena master")
            eq(am, cap.snap_m, "arena exp_avg")
            eq(av, cap.snap_v, "arena exp_avg_sq")
            # ... and, for every applied step, the gradients of the parts sent before it
            offs = oracle.sent_offsets(bounds)
            for s in range(2, K + 1):
                if cap.records["skip"][s - 1]:
                    continue
                got = sess.arena_grads(s)
                assert np.array_equal(got, cap.sent[offs[s - 1]:offs[s]]), f"gradient block of step {s}"
        # reconstruction: the synchronous checkpoint after step K
        outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
        meta = sess.restore(nthreads=nthreads, out=outs)
        eq(outs[0], sync.p, "restored master")
        eq(outs[1], sync.m, "restored exp_avg")
        eq(outs[2], sync.v, "restored exp_avg_sq")
        assert np.array_equal(outs[3], sync.w), "restored bf16 weights"
        assert meta.t == sync.t and meta.scale == sync.scale and meta.tracker == sync.tracker
        assert meta.K == K
        return sess, stats, meta
    finally:
        sess.close()


def test_flat16m_k4_window_bitwise():
    """The 16.7M flat workload: 4 equal parts, 256 MiB ring, restore target =
    state after step 4."""
    n = 16_777_216
    K = 4
    bounds = [0, n // 4, n // 2, 3 * n // 4, n]
    _, stats, _ = _run_window(n, K, bounds, seed=0, ring_bytes=256 << 20)
    assert stats.bytes_spilled == 0  # the ring holds the whole 240 MiB window
    assert stats.bytes_ring == 12 * n + 2 * (n // 4) * (0 + 1 + 2 + 3)


@pytest.mark.parametrize("late_plan", [0, 1, 2])
def test_ragged_with_small_ring_wraps_and_spills(late_plan):
    """n not a multiple of 8, unequal parts, a 192 KiB ring: the pack list
    wraps around the ring and the rest is copied straight from the live
    buffers; the result must not change, whether the ring use is decided when
    the host calls the step (QUERY), when the device reaches the update
    (HOST_WAIT), or as if the ring were drained with the device waiting for
    the copies of the reused ranges (DEVICE_WAIT)."""
    n = 100_003
    bounds = [0, 8, 20_008, 20_016, 61_440, 99_992, n]
    _, stats, _ = _run_window(n, len(bounds) - 1, bounds, seed=3, ring_bytes=192 << 10, copy_bytes=16 << 10,
                              timing=True, late_plan=late_plan)
    assert stats.bytes_spilled > 0 and stats.bytes_ring > 0


@pytest.mark.parametrize("replay_every", [0, 1, 2, 3])
@pytest.mark.parametrize("pageable", [False, True])
def test_staging_and_in_window_replay(pageable, replay_every):
    """Pageable arena through 3 pinned staging slots of 16 KiB, and in-window
    replay every R steps (R = 0: at restore), on top of ring wrap and direct
    spill (a 96 KiB ring), under the three ring plans."""
    n = 60_011
    bounds = [0, 8, 12_000, 24_000, 30_000, 41_000, n]
    _, stats, meta = _run_window(n, 6, bounds, seed=20 + replay_every, ring_bytes=96 << 10, copy_bytes=16 << 10,
                                 pageable=pageable, staging_slots=3, replay_every=replay_every,
                                 late_plan=(2, 1, 2, 0)[replay_every])
    assert stats.bytes_spilled > 0 and stats.bytes_ring > 0
    assert meta.t == 6


@pytest.mark.parametrize("wait_policy,ring_off", [(1, True), (1, False), (2, True), (0, True)])
def test_wait_policies_same_checkpoint(wait_policy, ring_off):
    """GoCkpt's explicit gradient wait (GRADS), a blocking copy of every step
    (ALL) and the lazy waits, with and without the ring: only the moment the
    compute stream may go on changes, never a bit of what reaches the host."""
    n = 50_017
    bounds = [0, 16, 12_504, 25_000, n]
    _, stats, _ = _run_window(n, 4, bounds, seed=40 + wait_policy, ring_bytes=64 << 10, copy_bytes=8 << 10,
                              wait_policy=wait_policy, ring_off=ring_off, timing=True)
    if ring_off:
        assert stats.bytes_ring == 0 and stats.bytes_spilled == stats.bytes_d2h
    else:
        assert stats.bytes_ring > 0


@pytest.mark.parametrize("wait_policy", [0, 2])
def test_single_step_snapshot_schemes(wait_policy):
    """K = 1 with the ring off: the Async-O (lazy) and Async (blocking)
    snapshots of the whole state.  Two plain steps follow at once; the arena
    must still hold the state after the window step (the next update waits for
    the copies of the live state), and the restore returns it unchanged."""
    import torch
    from paper_2511_07035_amd import Session

    n = 70_001
    seed = 50 + wait_policy
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, seed)
    sync = oracle.State(p0)
    sess = Session(n, ring_bytes=1 << 20, copy_bytes=16 << 10)
    try:
        load_state(sess, p0, w=sync.w)
        sess.begin_window([0, n], wait_policy=wait_policy, ring_off=True)
        for step in range(1, 4):
            g = synth.grads_cpu(n, seed, step)
            sess.backward_begin()
            to_device_grad16(sess, g)
            sess.step(cfg.lr)
            oracle.adamw_step(sync, g, cfg)
            if step == 1:
                want = (sync.p.copy(), sync.m.copy(), sync.v.copy(), sync.w.copy())
        stats = sess.drain(blocking=True)
        assert stats.bytes_ring == 0 and stats.bytes_d2h == 12 * n
        ap, am, av = sess.arena_state()
        assert_bits_equal(ap, want[0], "arena master")
        assert_bits_equal(am, want[1], "arena exp_avg")
        assert_bits_equal(av, want[2], "arena exp_avg_sq")
        outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
        meta = sess.restore(out=outs)
        for got, ref, what in zip(outs[:3], want[:3], ("master", "exp_avg", "exp_avg_sq")):
            assert_bits_equal(got, ref, "restored " + what)
        assert np.array_equal(outs[3], want[3])
        assert meta.t == 1 and meta.K == 1
        p, m, v, w = sess.state_to_host()
        assert_bits_equal(p, sync.p, "device master after the plain steps")
        torch.cuda.synchronize()
    finally:
        sess.close()


def test_staged_replay_with_skips():
    """Dynamic scaling, infs at steps 3 and 7, in-window replay every 3 steps
    through staging into a pageable arena."""
    n = (1 << 18) + 24
    bounds = list(np.linspace(0, n, 9).astype(np.int64) // 8 * 8)
    bounds[-1] = n
    _, stats, meta = _run_window(n, 8, bounds, seed=25, ring_bytes=1 << 20, copy_bytes=64 << 10, dynamic=True,
                                 inf_steps=(3, 7), pageable=True, staging_slots=4, replay_every=3)
    assert stats.skipped == 2 and meta.t == 6 and meta.scale == 16384.0


def test_no_ring_everything_spills():
    n = 50_000
    bounds = [0, 10_000, 25_000, 40_000, n]
    _, stats, _ = _run_window(n, 4, bounds, seed=4, ring_bytes=0)
    assert stats.bytes_ring == 0 and stats.bytes_spilled == stats.bytes_d2h - 0


@pytest.mark.parametrize("knobs", [dict(GOCKPT_QUADS="2"), dict(GOCKPT_QUADS="4", GOCKPT_FUSED_NT="0"),
                                   dict(GOCKPT_FUSED_BLOCK="1024"), dict(GOCKPT_FUSED_BLOCK="1024", GOCKPT_FUSED_NT="0"),
                                   dict(GOCKPT_RING_NT="0", GOCKPT_PREPASS_NT="0")])
def test_kernel_variants_same_bits(knobs, monkeypatch):
    """The tuning variants a context can be created with (quads per lane,
    1024-thread blocks, nontemporal state, ring and prepass accesses) change
    only the memory access pattern: ragged parts, a wrapping and spilling ring and skipped
    steps give the oracle's bits under each."""
    for k, v in knobs.items():
        monkeypatch.setenv(k, v)
    n = 100_003
    bounds = [0, 8, 20_008, 20_016, 61_440, 99_992, n]
    _, stats, _ = _run_window(n, len(bounds) - 1, bounds, seed=47, ring_bytes=192 << 10, copy_bytes=16 << 10,
                              dynamic=True, inf_steps=(3,))
    assert stats.bytes_spilled > 0 and stats.bytes_ring > 0 and stats.skipped == 1


@pytest.mark.parametrize("grad_norm", [True, False])
def test_overflow_check_off(grad_norm):
    """check_overflow = 0: no step is skipped, so an inf gradient reaches the
    update and turns its element's master weight into NaN on both sides; every
    other element keeps the oracle's bits.  With the norm off as well, the
    step runs no prepass (the records say nonfinite 0, gnorm2 -1)."""
    n = 50_003
    bounds = [0, 12_000, 30_000, n]
    sess, stats, meta = _run_window(n, 3, bounds, seed=48, ring_bytes=128 << 10, copy_bytes=16 << 10,
                                    inf_steps=(2,), check_overflow=False, grad_norm=grad_norm, nan_equiv=True)
    assert stats.skipped == 0 and meta.t == 3


def test_caller_found_inf_flag():
    """A caller-side overflow test (a gradient scaler's found-inf flag) takes
    the skip decisions.  With the norm off no prepass runs, and a planted inf
    is still skipped because the flag says so; with the norm on, a flag set
    on finite gradients skips those steps too: the flag governs."""
    n = (1 << 18) + 40
    bounds = [0, 65_536, 131_072, 196_608, n]
    _, stats, meta = _run_window(n, 4, bounds, seed=49, ring_bytes=1 << 20, dynamic=True, inf_steps=(3,),
                                 grad_norm=False, found_inf=[0.0, 0.0, 1.0, 0.0])
    assert stats.skipped == 1 and meta.t == 3 and meta.scale == 32768.0
    _, stats, meta = _run_window(n, 4, bounds, seed=50, ring_bytes=1 << 20, found_inf=[0.0, 1.0, 0.0, float("nan")])
    assert stats.skipped == 2 and meta.t == 2


@pytest.mark.parametrize("grad_dtype", ["bf16", "fp16"])
def test_bucket_scans_replace_the_prepass(grad_dtype):
    """The overflow test and norm done bucket by bucket on a side stream
    (gockpt_scan_grads), as buckets of a backward complete: the same skips,
    the same bits, and the norm within the telemetry tolerance."""
    n = 200_003
    bounds = [0, 40_000, 90_000, 150_000, n]
    buckets = [0, 8, 65_536, 100_000, 180_000, n]  # a tiny bucket and a ragged last one
    _, stats, meta = _run_window(n, 4, bounds, seed=53, ring_bytes=512 << 10, copy_bytes=64 << 10, dynamic=True,
                                 inf_steps=(3,), grad_dtype=grad_dtype, scan_buckets=buckets)
    assert stats.skipped == 1 and meta.t == 3


def test_bucket_scan_rules():
    """Scans must tile [0, n): an overlap is refused at once, a step with
    partial coverage is refused (and may be retried once the rest is
    scanned), misaligned ranges are refused."""
    from paper_2511_07035_amd import GOCKPT_EINVAL, GOCKPT_ESTATE, GockptError, Session

    n = 10_007
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, 54)
    ref = oracle.State(p0)
    sess = Session(n, ring_bytes=0)
    try:
        load_state(sess, p0, w=ref.w)
        g = synth.grads_cpu(n, 54, 1)
        to_device_grad16(sess, g)
        sess.scan_grads(0, 4096)
        with pytest.raises(GockptError) as e:
            sess.scan_grads(4088, 8000)
        assert e.value.code == GOCKPT_ESTATE
        with pytest.raises(GockptError) as e:
            sess.scan_grads(4100, 8000)
        assert e.value.code == GOCKPT_EINVAL
        with pytest.raises(GockptError) as e:
            sess.step(cfg.lr)  # [4096, n) not scanned
        assert e.value.code == GOCKPT_ESTATE
        sess.scan_grads(8000, n)
        with pytest.raises(GockptError) as e:
            sess.scan_grads(4096, 8008)  # runs into [8000, n)
        assert e.value.code == GOCKPT_ESTATE
        sess.scan_grads(4096, 8000)
        sess.step(cfg.lr)
        oracle.adamw_step(ref, g, cfg)
        # the next step without scans runs the prepass again
        g = synth.grads_cpu(n, 54, 2)
        to_device_grad16(sess, g)
        sess.step(cfg.lr)
        oracle.adamw_step(ref, g, cfg)
        p, m, v, w = sess.state_to_host()
        assert_bits_equal(p, ref.p, "master")
        assert_bits_equal(v, ref.v, "exp_avg_sq")
    finally:
        sess.close()


def test_dynamic_scale_skips_replayed_exactly():
    """Dynamic loss scaling with +inf planted at steps 3 and 7 of an 8-step
    window (the 1.3B dynamic-scaling workload's recipe at a reduced size)."""
    n = (1 << 20) + 40
    bounds = list(np.linspace(0, n, 9).astype(np.int64) // 8 * 8)
    bounds[-1] = n
    _, stats, meta = _run_window(n, 8, bounds, seed=5, ring_bytes=64 << 20, dynamic=True, inf_steps=(3, 7))
    assert stats.skipped == 2
    assert meta.t == 6 and meta.scale == 16384.0 and meta.tracker == 1


def test_laplace_gradients_tensor_bounds_lr_schedule():
    """Laplace(0, 5e-4) gradients (the 13B workload's law), parts cut at
    tensor boundaries of a small Llama-shaped layout, a changing lr."""
    lay = synth.layout_llama(layers=2, hidden=64, ffn=176, vocab=320)
    n = synth.numel(lay)
    from paper_2511_07035_amd import gockpt_plan_bounds
    K = 6
    bounds = gockpt_plan_bounds(K, n, synth.tensor_ends(lay))
    lrs = np.array([1e-4, 2e-4, 3e-4, 2.5e-4, 1e-4, 5e-5], dtype=np.float32)
    _run_window(n, K, bounds, seed=6, ring_bytes=1 << 20, law="laplace", lrs=lrs)


def test_without_bf16_weights():
    n = 4096 + 24
    _run_window(n, 2, [0, 2048, n], seed=7, ring_bytes=1 << 20, with_weight=False)


def test_tiny_spaces():
    for n, bounds in [(1, [0, 1]), (7, [0, 7]), (8, [0, 8]), (9, [0, 8, 9]), (16, [0, 8, 16]),
                      (23, [0, 8, 16, 23])]:
        _run_window(n, len(bounds) - 1, bounds, seed=8 + n, ring_bytes=4096)


def test_longest_window():
    """K = GOCKPT_MAX_K: 256 parts of 64 elements and a ragged last one,
    through a 64 KiB ring that wraps many times; one more part is refused."""
    from paper_2511_07035_amd import GOCKPT_MAX_K, GockptError, Session

    K = GOCKPT_MAX_K
    n = 64 * K + 40
    bounds = list(range(0, 64 * K, 64)) + [n]
    _run_window(n, K, bounds, seed=46, ring_bytes=64 << 10, copy_bytes=16 << 10, per_step=False)
    n2 = n + 64  # the same layout with one part more: valid bounds, K = 257
    sess = Session(n2, ring_bytes=0)
    try:
        with pytest.raises(GockptError):
            sess.begin_window(list(range(0, 64 * (K + 1), 64)) + [n2])
    finally:
        sess.close()


def test_empty_space():
    """n = 0: plain steps still decide the skip and count the step; a window
    has no part to send and is refused."""
    from paper_2511_07035_amd import GockptError, Session

    sess = Session(0, ring_bytes=0)
    try:
        sess.step(1e-3)
        sess.step(1e-3)
        assert sess.scaler()[0] == 2
        p, m, v, w = sess.state_to_host()
        assert p.size == m.size == v.size == w.size == 0
        with pytest.raises(GockptError):
            sess.begin_window([0, 0])
    finally:
        sess.close()


def test_edge_values_bitwise():
    """Crafted values: zero and subnormal moments, subnormal and huge
    gradients, signed zeros, values at bf16 rounding ties, the largest finite
    bf16 gradient.  Exercises correctly rounded division and square root and
    subnormal handling of the device against the oracle."""
    rng = np.random.default_rng(9)
    n = 4096
    tiny = np.float32(1e-39)  # subnormal
    p0 = rng.normal(0, 1, n).astype(np.float32)
    p0[:64] = np.array([0.0, -0.0, tiny, -tiny, 1e-38, 3.0e38, -3.0e38, 1.0] * 8, dtype=np.float32)
    # values whose bf16 rounding is a tie after a tiny update
    p0[64:128] = (np.uint32(0x3F800000) + (np.arange(64, dtype=np.uint32) << 16) + np.uint32(0x8000)) \
        .view(np.float32)
    m0 = rng.normal(0, 1e-4, n).astype(np.float32)
    v0 = np.abs(rng.normal(0, 1e-8, n)).astype(np.float32)
    m0[:32] = tiny
    v0[:32] = np.float32(1e-45)  # smallest subnormal
    v0[32:64] = 0.0
    g = rng.normal(0, 1e-3, n).astype(np.float32)
    g[:16] = np.float32(1e-39)
    g[16:32] = np.float32(-0.0)
    g[32:48] = np.float32(3.0e38)
    g[48:64] = np.float32(1e-20)
    gbits = synth._bf16_bits_cpu(g)
    gbits[100] = 0x7F7F  # largest finite bf16
    gbits[101] = 0x0001  # smallest subnormal bf16
    grads = np.stack([gbits, np.roll(gbits, 7)])
    _run_window(n, 2, [0, 2048, n], seed=10, ring_bytes=1 << 20, p0=p0, m0=m0, v0=v0, grads=grads)


@pytest.mark.parametrize("hp", [dict(lr=3e-3, beta1=0.95, beta2=0.98, eps=1e-6, weight_decay=0.0),
                                dict(lr=0.1, beta1=0.8, beta2=0.99, eps=1e-3, weight_decay=0.5)])
def test_other_hyperparameters(hp):
    """The optimizer constants enter the contract through the per-step
    scalars: other betas, eps, weight decay and a large learning rate give the
    oracle's bits too."""
    n = 70_001
    bounds = [0, 16_000, 40_000, n]
    lrs = np.full(3, hp["lr"], dtype=np.float32)
    _run_window(n, 3, bounds, seed=44, ring_bytes=512 << 10, lrs=lrs, hp=hp)


def test_fp16_gradients_window_with_skips():
    """fp16 gradients (Sec. 2.2) under dynamic scaling with planted fp16
    infinities, ragged parts, ring wrap and spill."""
    n = 150_001
    bounds = [0, 8, 30_000, 60_000, 90_000, 120_000, 149_992, 150_000, n]
    _, stats, meta = _run_window(n, 8, bounds, seed=33, ring_bytes=256 << 10, copy_bytes=32 << 10, dynamic=True,
                                 inf_steps=(3, 7), grad_dtype="fp16")
    assert stats.skipped == 2 and meta.t == 6 and stats.bytes_spilled > 0


def test_fp16_edge_values_bitwise():
    """fp16 gradient patterns at the format's edges: every subnormal
    exponent position, the largest finite value (65504), signed zeros, the
    smallest normal; with subnormal and zero moments."""
    rng = np.random.default_rng(19)
    n = 4096
    g = rng.normal(0, 1e-3, n).astype(np.float16).view(np.uint16)
    sub = np.array([1 << k for k in range(10)] + [0x03FF, 0x0155], np.uint16)
    g[:12] = sub
    g[12:24] = sub | 0x8000
    g[24:28] = [0x7BFF, 0xFBFF, 0x0400, 0x8400]
    g[28:30] = [0x0000, 0x8000]
    p0 = rng.normal(0, 1, n).astype(np.float32)
    m0 = rng.normal(0, 1e-4, n).astype(np.float32)
    v0 = np.abs(rng.normal(0, 1e-8, n)).astype(np.float32)
    v0[:16] = np.float32(1e-45)
    v0[16:32] = 0.0
    grads = np.stack([g, np.roll(g, 5), np.roll(g, 11)])
    _run_window(n, 3, [0, 1024, 2048, n], seed=12, ring_bytes=1 << 20, p0=p0, m0=m0, v0=v0, grads=grads,
                grad_dtype="fp16")


def test_plain_steps_outside_window_and_state_machine():
    import torch
    from paper_2511_07035_amd import GOCKPT_EBUSY, GOCKPT_ESTATE, GockptError, Session

    n = 10_000
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, 12)
    ref = oracle.State(p0)
    sess = Session(n, ring_bytes=1 << 20)
    try:
        load_state(sess, p0, w=ref.w)
        # plain steps (no window) are the fused update alone
        for s in range(1, 4):
            g = synth.grads_cpu(n, 12, s)
            to_device_grad16(sess, g)
            sess.step(cfg.lr)
            oracle.adamw_step(ref, g, cfg)
        p, m, v, w = sess.state_to_host()
        assert_bits_equal(p, ref.p, "plain master")
        assert_bits_equal(v, ref.v, "plain exp_avg_sq")
        assert sess.scaler()[0] == 3
        with pytest.raises(GockptError) as e:
            sess.drain()
        assert e.value.code == GOCKPT_ESTATE
        with pytest.raises(GockptError) as e:
            sess.restore()
        assert e.value.code == GOCKPT_ESTATE
        sess.begin_window([0, 5000, n])
        with pytest.raises(GockptError) as e:
            sess.begin_window([0, 5000, n])
        assert e.value.code == GOCKPT_EBUSY
        with pytest.raises(GockptError) as e:
            sess.drain()  # window not complete
        assert e.value.code == GOCKPT_ESTATE
        sess.step(cfg.lr)
        sess.abort_window()  # discard the half-done window
        sess.begin_window([0, 5000, n])
        sess.step(cfg.lr)
        sess.step(cfg.lr)
        while sess.drain(blocking=False) is None:
            pass
        sess.restore(nthreads=2)  # in place in the arena
        torch.cuda.synchronize()
    finally:
        sess.close()


def test_plain_step_graph_replay():
    """A plain step (outside a window) is three kernels on the compute stream
    and no host work, so it can be captured in a HIP graph and replayed; the
    step count and the loss scale live on the device and advance with every
    replay.  Each replay, with new gradients written eagerly before it and a
    skipped step among them, must give the oracle's bits."""
    import torch
    from paper_2511_07035_amd import Session

    n = 100_003
    cfg = oracle.AdamWConfig(dynamic_scale=True, init_scale=1024.0, growth_interval=2)
    p0 = synth.master_cpu(n, 51)
    ref = oracle.State(p0, scale=1024.0)
    sess = Session(n, ring_bytes=0, dynamic_scale=True, init_scale=1024.0, growth_interval=2)
    try:
        load_state(sess, p0, w=ref.w)
        # a window without a ring first: its last step copies state and
        # gradients straight from the live buffers, and after the drain no
        # later step may still wait for those copies (a capture could not)
        sess.begin_window([0, 50_000, n])
        for k in (1, 2):
            grads = synth.grads_cpu(n, 51, k, scale=ref.scale)
            sess.backward_begin()
            to_device_grad16(sess, grads)
            sess.step(cfg.lr)
            oracle.adamw_step(ref, grads, cfg)
        sess.drain(blocking=True)
        sess.restore()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=sess.compute):  # records the launches, runs nothing
            sess.step(cfg.lr)
        for k in range(3, 9):
            scale = ref.scale
            grads = synth.grads_cpu(n, 51, k, scale=scale, plant_inf=k == 5)
            to_device_grad16(sess, grads)
            with torch.cuda.stream(sess.compute):
                g.replay()
            oracle.adamw_step(ref, grads, cfg)
            p, m, v, w = sess.state_to_host()
            assert_bits_equal(p, ref.p, f"master after replay {k}")
            assert_bits_equal(m, ref.m, f"exp_avg after replay {k}")
            assert_bits_equal(v, ref.v, f"exp_avg_sq after replay {k}")
            assert np.array_equal(w, ref.w), f"bf16 weights after replay {k}"
            assert sess.scaler() == (ref.t, ref.scale, ref.tracker)
        assert ref.t == 7
    finally:
        sess.close()


def test_restore_in_background():
    """gockpt_restore_async: the host replay runs in a library thread while
    plain steps go on; the wait gives the checkpoint of the window's last
    step, bitwise.  A window begun while an in-place restore still runs
    waits for it, and restores exactly in turn."""
    from paper_2511_07035_amd import Session

    n, K, seed = 300_007, 4, 52
    bounds = [0, 60_000, 150_000, 220_000, n]
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, seed)
    sync = oracle.State(p0)
    sess = Session(n, ring_bytes=1 << 20, copy_bytes=64 << 10)
    gstep = 0

    def step(window: bool):
        nonlocal gstep
        gstep += 1
        g = synth.grads_cpu(n, seed, gstep)
        if window:
            sess.backward_begin()
        to_device_grad16(sess, g)
        sess.step(cfg.lr)
        oracle.adamw_step(sync, g, cfg)

    try:
        load_state(sess, p0, w=sync.w)
        sess.begin_window(bounds)
        for _ in range(K):
            step(True)
        sess.drain(blocking=True)
        want = sync.copy()
        out = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
        sess.restore(nthreads=2, out=out, async_=True)
        for _ in range(3):  # training goes on during the replay
            step(False)
        meta = sess.restore_wait()
        assert_bits_equal(out[0], want.p, "restored master")
        assert_bits_equal(out[1], want.m, "restored exp_avg")
        assert_bits_equal(out[2], want.v, "restored exp_avg_sq")
        assert np.array_equal(out[3], want.w) and meta.t == want.t == K
        p, _, v, _ = sess.state_to_host()
        assert_bits_equal(p, sync.p, "device master after the steps beside the replay")
        # an in-place restore still running when the next window begins
        sess.begin_window([0, 100_000, n])
        for _ in range(2):
            step(True)
        sess.drain(blocking=True)
        sess.restore(async_=True)
        sess.begin_window(bounds)  # waits for the replay first
        for _ in range(K):
            step(True)
        sess.drain(blocking=True)
        meta = sess.restore(out=out)
        assert_bits_equal(out[0], sync.p, "restored master after the next window")
        assert_bits_equal(out[2], sync.v, "restored exp_avg_sq after the next window")
        assert meta.t == sync.t
    finally:
        sess.close()


def test_state_slab_layout_and_window():
    """StateSlab: the five arrays sit `spacing` apart inside one reservation,
    take() carves disjoint buffers from the space between them, and a window
    over slab-carved state (ring carved too) is bit-exact."""
    import torch
    from paper_2511_07035_amd import Session, StateSlab

    n = 60_011
    st = StateSlab(n, slab_bytes=64 << 20, spacing=8 << 20)
    base = st.slab.data_ptr()
    offs = [a.data_ptr() - base for a in st.arrays]
    assert offs == [0, 8 << 20, 16 << 20, 24 << 20, 32 << 20]
    ring = st.take(1 << 20)
    other = st.take(3 << 20)
    spans = [(o, o + a.numel() * a.element_size()) for o, a in zip(offs, st.arrays)]
    spans += [(t.data_ptr() - base, t.data_ptr() - base + t.numel()) for t in (ring, other)]
    spans.sort()
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:])), spans
    assert st.take(1 << 30) is None
    cfg = oracle.AdamWConfig()
    bounds = [0, 8, 12_000, 24_000, 41_000, n]
    p0 = synth.master_cpu(n, 30)
    grads = np.stack([synth.grads_cpu(n, 30, s) for s in range(1, 6)])
    ref = oracle.State(p0)
    oracle.sync_run(ref, grads, cfg)
    sess = Session(n, master=st.master, exp_avg=st.exp_avg, exp_avg_sq=st.exp_avg_sq, grad=st.grad,
                   weight=st.weight, ring=ring, copy_bytes=64 << 10)
    try:
        load_state(sess, p0, w=oracle.State(p0).w)
        sess.begin_window(bounds)
        for s in range(1, 6):
            sess.backward_begin()
            to_device_grad16(sess, grads[s - 1])
            sess.step(cfg.lr)
        sess.drain()
        out = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
        sess.restore(out=out)
        assert_bits_equal(out[0], ref.p, "restored master (slab layout)")
        assert_bits_equal(out[2], ref.v, "restored exp_avg_sq (slab layout)")
        torch.cuda.synchronize()
    finally:
        sess.close()


def test_grad_spill_requires_backward_begin():
    """While gradients are being copied straight from the gradient buffer, a
    step that comes without gockpt_backward_begin is refused; once the window
    is drained every copy has finished and plain steps need no such call."""
    from paper_2511_07035_amd import GOCKPT_ESTATE, GockptError, Session

    n = 4096
    sess = Session(n, ring_bytes=0)
    try:
        load_state(sess, synth.master_cpu(n, 13))
        to_device_grad16(sess, synth.grads_cpu(n, 13, 1))
        sess.begin_window([0, 1024, 2048, n])
        sess.step(1e-4)  # step 1 sends no gradients
        sess.step(1e-4)  # step 2 copies gradients straight from the buffer
        with pytest.raises(GockptError) as e:
            sess.step(1e-4)
        assert e.value.code == GOCKPT_ESTATE
        sess.backward_begin()
        sess.step(1e-4)
        sess.drain()
        sess.restore()
        sess.step(1e-4)  # plain, after the drain
        sess.step(1e-4)
        assert sess.scaler()[0] == 5
    finally:
        sess.close()


def _run_ahead_window(n, K, bounds, *, seed, ring_bytes, copy_bytes, late_plan, pageable=False, staging_slots=0,
                      dynamic=False, inf_steps=(), replay_every=0, defer_copies=False):
    """A window whose K steps are queued without any host synchronisation in
    between: every step's gradients are uploaded to the device first, and a
    step copies them into the gradient buffer on the compute stream, so the
    host runs ahead of the device and the ring (and the staging slots) are
    reused while earlier copies may still be in flight.  The device-side
    waits alone must keep every byte in order."""
    import torch
    from paper_2511_07035_amd import Session

    print(f"[case] run-ahead n={n} K={K} ring={ring_bytes} copy={copy_bytes} plan={late_plan} "
          f"pageable={pageable} slots={staging_slots} R={replay_every} defer={defer_copies}", flush=True)
    scale0 = 65536.0 if dynamic else 1.0
    cfg = oracle.AdamWConfig(dynamic_scale=dynamic, init_scale=scale0)
    sched = synth.DYNSCALE_SCHEDULE if dynamic else {}
    p0 = synth.master_cpu(n, seed)
    grads = np.stack([synth.grads_cpu(n, seed, s, scale=sched.get(s, scale0), plant_inf=s in inf_steps)
                      for s in range(1, K + 1)])
    sync = oracle.State(p0, scale=scale0)
    win = oracle.State(p0, scale=scale0)
    cap = oracle.window_capture(win, grads, bounds, cfg)
    for s in range(K):
        oracle.adamw_step(sync, grads[s], cfg)
    sess = Session(n, dynamic_scale=dynamic, init_scale=scale0, ring_bytes=ring_bytes, copy_bytes=copy_bytes,
                   staging_bytes=staging_slots * copy_bytes, copy_threads=3, timing=True)
    try:
        load_state(sess, p0)
        dev_grads = torch.from_numpy(grads.view(np.int16)).to("cuda")
        torch.cuda.synchronize()
        sess.begin_window(bounds, late_plan=late_plan, pageable=pageable, replay_every=replay_every,
                          defer_copies=defer_copies)
        # hold the compute stream for a while, so that everything below is
        # queued before the device runs any of it
        import ctypes
        from paper_2511_07035_amd import BENCH_LIB_PATH
        bl = ctypes.CDLL(BENCH_LIB_PATH)
        bl.gockpt_bench_spin.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_int]
        assert bl.gockpt_bench_spin(sess.compute.cuda_stream, 200.0, 1) == 0
        for s in range(K):
            sess.backward_begin()
            with torch.cuda.stream(sess.compute):
                sess.grad.view(torch.int16).copy_(dev_grads[s])
            sess.step(cfg.lr)
        stats = sess.drain(blocking=True)
        recs = sess.records()
        assert list(recs["skip"]) == list(cap.records["skip"])
        ap, am, av = sess.arena_state()
        if not (0 < replay_every < K):
            assert_bits_equal(ap, cap.snap_p, "arena master")
            assert_bits_equal(am, cap.snap_m, "arena exp_avg")
            assert_bits_equal(av, cap.snap_v, "arena exp_avg_sq")
            offs = oracle.sent_offsets(bounds)
            for s in range(2, K + 1):
                if not cap.records["skip"][s - 1]:
                    assert np.array_equal(sess.arena_grads(s), cap.sent[offs[s - 1]:offs[s]]), f"gradients of step {s}"
        outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
        meta = sess.restore(nthreads=4, out=outs)
        assert_bits_equal(outs[0], sync.p, "restored master")
        assert_bits_equal(outs[1], sync.m, "restored exp_avg")
        assert_bits_equal(outs[2], sync.v, "restored exp_avg_sq")
        assert np.array_equal(outs[3], sync.w), "restored bf16 weights"
        assert meta.t == sync.t
        p, m, v, w = sess.state_to_host()
        assert_bits_equal(p, sync.p, "device master after the window")
        return stats
    finally:
        sess.close()


@pytest.mark.parametrize("late_plan", [0, 2])
def test_run_ahead_ring_reuse(late_plan):
    """The host queues all 8 steps before the device runs them; a 128 KiB
    ring smaller than one step's pack list is reused every step.  With
    DEVICE_WAIT the plan takes the whole ring at every step, and only the
    compute stream's waits on the earlier ring copies stop an update from
    overwriting bytes not yet on the host."""
    n = 200_003
    bounds = [0, 8, 30_000, 60_000, 90_000, 120_000, 150_000, 180_000, n]
    stats = _run_ahead_window(n, 8, bounds, seed=61, ring_bytes=128 << 10, copy_bytes=8 << 10,
                              late_plan=late_plan)
    assert stats.bytes_ring > 0 and stats.bytes_spilled > 0


@pytest.mark.parametrize("replay_every", [0, 2])
def test_run_ahead_staged_gates(replay_every):
    """A pageable arena through 4 staging slots of 8 KiB while the host runs
    ahead: hundreds of copies are queued at once, and before each copy that
    reuses a slot the copy stream runs a gate kernel that waits until a
    library thread has moved the slot's previous copy into the arena."""
    n = 150_011
    bounds = [0, 16, 40_000, 80_000, 110_000, n]
    stats = _run_ahead_window(n, 5, bounds, seed=62, ring_bytes=256 << 10, copy_bytes=8 << 10, late_plan=2,
                              pageable=True, staging_slots=4, replay_every=replay_every)
    assert stats.n_gates > 0


@pytest.mark.parametrize("late_plan", [1, 2])
def test_skipped_steps_send_no_gradients(late_plan):
    """Dynamic scaling with infs at steps 3 and 7.  The update packs no
    gradients on a skipped step; with HOST_WAIT the host also knows the skip
    before it plans, so the window copies 12 n + 2 * (sum of bounds[s-1] over
    the applied steps) bytes plus the records -- nothing for the skipped
    steps.  The checkpoint is the same either way."""
    n = (1 << 17) + 40
    bounds = list(np.linspace(0, n, 9).astype(np.int64) // 8 * 8)
    bounds[-1] = n
    _, stats, meta = _run_window(n, 8, bounds, seed=63, ring_bytes=4 << 20, copy_bytes=64 << 10, dynamic=True,
                                 inf_steps=(3, 7), timing=True, late_plan=late_plan)
    assert stats.skipped == 2 and meta.t == 6
    applied = [s for s in range(1, 9) if s not in (3, 7)]
    grads_applied = sum(2 * int(bounds[s - 1]) for s in applied)
    grads_all = sum(2 * int(bounds[s - 1]) for s in range(1, 9))
    base = 12 * n  # the step records are not counted in bytes_d2h
    if late_plan == 1:
        assert stats.bytes_d2h == base + grads_applied, (stats.bytes_d2h, base + grads_applied)
    else:
        # the host does not know the skips when it plans: every gradient
        # block is sent, and the replay never reads those of skipped steps
        assert stats.bytes_d2h == base + grads_all, (stats.bytes_d2h, base + grads_all)
    # what the kernel packed: a skipped step only its part's state
    assert stats.bytes_ring == 12 * n + grads_applied


@pytest.mark.parametrize("ring_kib", [0, 512])
def test_planner_chosen_window(ring_kib):
    """A window whose K and bounds come from gockpt_plan_window (Sec. 4.2.3's
    stall model, capped at 7 steps) over a reduced model-shaped layout: a
    tiny Llama-style stack whose tensor ends restrict the bounds, a slow
    link, with and without a ring.  The chosen window must run and restore
    bitwise like any other."""
    from paper_2511_07035_amd import gockpt_plan_window

    layout = synth.layout_llama(layers=3, hidden=64, ffn=176, vocab=320)
    n = synth.numel(layout)
    ends = synth.tensor_ends(layout)
    bounds, plan = gockpt_plan_window(n, 1.0, 2.0, 0.05, 0.05, tensor_ends=ends, ring_bytes=ring_kib << 10,
                                      copy_bytes=16 << 10, max_K=7)
    K = plan.K
    assert 1 <= K <= 7 and bounds[0] == 0 and bounds[-1] == n and len(bounds) == K + 1
    assert set(int(x) for x in bounds[1:-1]) <= set(int(x) for x in ends)
    print(f"[case] planner window n={n} K={K} bounds={list(bounds)} predicted {plan.stall_ms:.3f} ms", flush=True)
    _run_window(n, K, [int(x) for x in bounds], seed=70 + ring_kib, ring_bytes=ring_kib << 10,
                copy_bytes=16 << 10, late_plan=2)


@pytest.mark.parametrize("late_plan", [0, 1, 2])
def test_debug_poison_and_order_checks(late_plan, monkeypatch):
    """The debug switches: every ring range and staging slot is filled with
    0xFF bytes (a NaN pattern) as soon as its copy has taken it, and the ring
    and staging order invariants are checked on the host at every window
    step.  A copy that read a range before the pack wrote it, or a pack that
    overwrote one before its copy, would now carry NaNs into the arena; the
    windows -- a wrapping, spilling ring, and a run-ahead staged window --
    must still be bitwise and no check may fire.  roctx ranges are on too
    (no profiler attached: they cost nothing and change nothing)."""
    for k in ("GOCKPT_DEBUG_POISON", "GOCKPT_DEBUG_CHECKS", "GOCKPT_ROCTX"):
        monkeypatch.setenv(k, "1")
    n = 100_003
    bounds = [0, 8, 20_008, 20_016, 61_440, 99_992, n]
    _run_window(n, len(bounds) - 1, bounds, seed=80 + late_plan, ring_bytes=192 << 10, copy_bytes=16 << 10,
                late_plan=late_plan)
    _run_ahead_window(150_011, 5, [0, 16, 40_000, 80_000, 110_000, 150_011], seed=83 + late_plan,
                      ring_bytes=256 << 10, copy_bytes=8 << 10, late_plan=late_plan, pageable=True,
                      staging_slots=4, replay_every=2 if late_plan == 2 else 0)


def test_window_without_timing_events():
    """A context with timing on can run a window without its timing events
    (gockpt_window_opts.no_timing): the window is the same bits, and its step
    times are not available; the next timed window has them again."""
    from paper_2511_07035_amd import GockptError, Session

    n = 30_011
    bounds = [0, 8_000, 16_000, n]
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, 90)
    sync = oracle.State(p0)
    sess = Session(n, ring_bytes=1 << 20, copy_bytes=16 << 10, timing=True)
    try:
        load_state(sess, p0)
        for timing in (False, True):
            sess.begin_window(bounds, late_plan=2, timing=timing)
            for s in range(1, 4):
                g = synth.grads_cpu(n, 90, s + (0 if timing else 10))
                sess.backward_begin()
                to_device_grad16(sess, g)
                sess.step(cfg.lr)
                oracle.adamw_step(sync, g, cfg)
            sess.drain(blocking=True)
            if timing:
                assert sess.step_times().shape == (3, 5)
            else:
                with pytest.raises(GockptError, match="ESTATE"):
                    sess.step_times()
            outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), None)
            sess.restore(out=outs)
            assert_bits_equal(outs[0], sync.p, f"restored master (timing={timing})")
            assert_bits_equal(outs[2], sync.v, f"restored exp_avg_sq (timing={timing})")
    finally:
        sess.close()


@pytest.mark.parametrize("case", ["wrap_query", "wrap_device", "staged_replay", "run_ahead_ring", "run_ahead_staged",
                                  "single_step"])
def test_deferred_copies_same_checkpoint(case):
    """defer_copies: each window step's copies are queued at the next call
    into the library (backward_begin, the next step or the drain) instead of
    by the step itself.  Only when the copies start changes: the ring waits,
    spills, staging gates and in-window replays must give the same bits,
    including with the host far ahead of the device and for a one-step
    window whose copies are queued by the drain."""
    if case == "wrap_query" or case == "wrap_device":
        n = 100_003
        bounds = [0, 8, 20_008, 20_016, 61_440, 99_992, n]
        _, stats, _ = _run_window(n, len(bounds) - 1, bounds, seed=101, ring_bytes=192 << 10, copy_bytes=16 << 10,
                                  timing=True, late_plan=0 if case == "wrap_query" else 2, defer_copies=True)
        assert stats.bytes_spilled > 0 and stats.bytes_ring > 0
    elif case == "staged_replay":
        n = 60_011
        bounds = [0, 8, 12_000, 24_000, 30_000, 41_000, n]
        _, stats, _ = _run_window(n, 6, bounds, seed=102, ring_bytes=96 << 10, copy_bytes=16 << 10, pageable=True,
                                  staging_slots=3, replay_every=2, late_plan=2, defer_copies=True)
        assert stats.bytes_spilled > 0
    elif case == "run_ahead_ring":
        n = 200_003
        bounds = [0, 8, 30_000, 60_000, 90_000, 120_000, 150_000, 180_000, n]
        stats = _run_ahead_window(n, 8, bounds, seed=103, ring_bytes=128 << 10, copy_bytes=8 << 10, late_plan=2,
                                  defer_copies=True)
        assert stats.bytes_ring > 0 and stats.bytes_spilled > 0
    elif case == "run_ahead_staged":
        n = 150_011
        bounds = [0, 16, 40_000, 80_000, 110_000, n]
        stats = _run_ahead_window(n, 5, bounds, seed=104, ring_bytes=256 << 10, copy_bytes=8 << 10, late_plan=2,
                                  pageable=True, staging_slots=4, replay_every=2, defer_copies=True)
        assert stats.n_gates > 0
    else:
        n = 40_009
        _, stats, _ = _run_window(n, 1, [0, n], seed=105, ring_bytes=1 << 20, copy_bytes=16 << 10, late_plan=2,
                                  defer_copies=True)
        assert stats.bytes_d2h == 12 * n


def test_deferred_copies_rules():
    """defer_copies needs the lazy policy; a step whose deferred copies take
    gradients straight from the gradient buffer still needs
    gockpt_backward_begin before the next step; and an abort drops the
    deferred copies, after which a new window restores bitwise."""
    from paper_2511_07035_amd import GOCKPT_EINVAL, GOCKPT_ESTATE, GockptError, Session

    n = 4096
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, 106)
    sync = oracle.State(p0)
    sess = Session(n, ring_bytes=0, copy_bytes=4096)
    try:
        load_state(sess, p0, w=sync.w)
        with pytest.raises(GockptError) as e:
            sess.begin_window([0, 1024, 2048, n], wait_policy=1, defer_copies=True)
        assert e.value.code == GOCKPT_EINVAL
        g = synth.grads_cpu(n, 106, 1)
        to_device_grad16(sess, g)
        sess.begin_window([0, 1024, 2048, n], defer_copies=True)
        sess.step(cfg.lr)  # step 1 sends no gradients
        oracle.adamw_step(sync, g, cfg)
        sess.step(cfg.lr)  # step 2 copies gradients straight from the buffer (queued at the next call)
        oracle.adamw_step(sync, g, cfg)
        with pytest.raises(GockptError) as e:
            sess.step(cfg.lr)
        assert e.value.code == GOCKPT_ESTATE
        sess.abort_window()
        # a new window from the state after the two updates
        sess.begin_window([0, 2048, n], defer_copies=True)
        for s in range(1, 3):
            g = synth.grads_cpu(n, 106, 10 + s)
            sess.backward_begin()
            to_device_grad16(sess, g)
            sess.step(cfg.lr)
            oracle.adamw_step(sync, g, cfg)
        sess.drain(blocking=True)
        outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), None)
        meta = sess.restore(out=outs)
        assert_bits_equal(outs[0], sync.p, "restored master")
        assert_bits_equal(outs[1], sync.m, "restored exp_avg")
        assert_bits_equal(outs[2], sync.v, "restored exp_avg_sq")
        assert meta.t == 4
    finally:
        sess.close()
