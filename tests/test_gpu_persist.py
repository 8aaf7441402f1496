"""Crash and resume through the C-ABI (Sec. 4.4.3 persistence, Sec. 4.3.2
loading): a window is restored and persisted, the process's context goes
away, a fresh context loads the checkpoint and trains on; every state after
that must equal, bit for bit, the oracle's uninterrupted run."""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bits_equal, load_state, to_device_grad16

pytestmark = pytest.mark.gpu


def _grads(n, seed, steps, scales, inf_steps):
    return [synth.grads_cpu(n, seed, s, scale=scales[s], plant_inf=s in inf_steps) for s in steps]


@pytest.mark.parametrize("async_persist", [False, True])
def test_crash_and_resume_bitwise(tmp_path, async_persist):
    from paper_2511_07035_amd import GockptError, Session, gockpt_find_latest_checkpoint

    n, K, J, seed = 200_003, 4, 3, 70 + int(async_persist)
    bounds = [0, 50_000, 100_000, 150_000, n]
    # dynamic scaling with a skip inside the window and growth after it, so
    # the step count, scale and tracker of the checkpoint all matter
    cfg = oracle.AdamWConfig(dynamic_scale=True, init_scale=1024.0, growth_interval=3)
    scales = {1: 1024.0, 2: 1024.0, 3: 512.0, 4: 512.0, 5: 512.0, 6: 1024.0, 7: 1024.0}
    grads = _grads(n, seed, range(1, K + J + 1), scales, inf_steps=(2,))
    p0 = synth.master_cpu(n, seed)
    sync = oracle.State(p0, scale=1024.0)
    kw = dict(dynamic_scale=True, init_scale=1024.0, growth_interval=3, ring_bytes=1 << 20, copy_bytes=64 << 10)
    print(f"[case] crash/resume n={n} K={K} J={J} async={async_persist}", flush=True)

    a = Session(n, **kw)
    root = tmp_path / "ckpts"
    root.mkdir()
    try:
        load_state(a, p0, w=sync.w)
        a.begin_window(bounds)
        for s in range(1, K + 1):
            a.backward_begin()
            to_device_grad16(a, grads[s - 1])
            a.step(cfg.lr)
            oracle.adamw_step(sync, grads[s - 1], cfg, lr=cfg.lr)
        a.drain(blocking=True)
        meta = a.restore()  # in place: the arena holds the checkpoint
        assert (meta.t, meta.scale, meta.tracker) == (sync.t, sync.scale, sync.tracker)
        a.persist(str(root / f"step{meta.t}"), user_meta=f"window {K}\n", nthreads=4, async_=async_persist)
        st = a.persist_wait()
        assert st.bytes == 12 * n
        # a second, interrupted persist: its metadata never lands
        a.persist(str(root / "step999"), nthreads=2)
        os.unlink(root / "step999" / "meta")
    finally:
        a.close()  # the "crash": the training process's context is gone

    want = sync.copy()
    path = gockpt_find_latest_checkpoint(str(root))
    assert path.endswith(f"step{want.t}")
    b = Session(n, **kw)
    try:
        with pytest.raises(GockptError, match="meta missing"):
            b.load(str(root / "step999"))
        info = b.load(path, nthreads=4)
        assert (info.t, info.scale, info.tracker, info.K, info.skipped) == (want.t, want.scale, want.tracker, K, 1)
        assert b.scaler() == (want.t, want.scale, want.tracker)
        p, m, v, w = b.state_to_host()
        assert_bits_equal(p, want.p, "loaded master")
        assert_bits_equal(m, want.m, "loaded exp_avg")
        assert_bits_equal(v, want.v, "loaded exp_avg_sq")
        assert np.array_equal(w, want.w), "loaded bf16 weights (re-derived on the device)"
        # training resumes at the step after the checkpoint
        for s in range(K + 1, K + J + 1):
            b.backward_begin()
            to_device_grad16(b, grads[s - 1])
            b.step(cfg.lr)
            oracle.adamw_step(sync, grads[s - 1], cfg, lr=cfg.lr)
            p, m, v, w = b.state_to_host()
            assert_bits_equal(p, sync.p, f"master at step {s} after the resume")
            assert_bits_equal(m, sync.m, f"exp_avg at step {s} after the resume")
            assert_bits_equal(v, sync.v, f"exp_avg_sq at step {s} after the resume")
            assert np.array_equal(w, sync.w), f"bf16 weights at step {s}"
        assert b.scaler() == (sync.t, sync.scale, sync.tracker)
    finally:
        b.close()


def test_load_rejects_other_hyperparameters(tmp_path):
    from paper_2511_07035_amd import GockptError, Session, gockpt_write_checkpoint

    n = 4096
    p = synth.master_cpu(n, 1)
    z = np.zeros(n, np.float32)
    d = str(tmp_path / "ck")
    gockpt_write_checkpoint(d, p, z, z, t=3, weight_decay=0.05)
    s = Session(n, weight_decay=0.01, ring_bytes=0)
    try:
        with pytest.raises(GockptError, match="hyperparameters"):
            s.load(d)
    finally:
        s.close()
    s = Session(n, weight_decay=0.05, ring_bytes=0)
    try:
        info = s.load(d)
        assert info.t == 3 and s.scaler()[0] == 3
        got, _, _, w = s.state_to_host()
        assert_bits_equal(got, p, "loaded master")
        assert np.array_equal(w, oracle.bf16_rne_array(p))
    finally:
        s.close()


def test_background_persist_survives_the_next_window(tmp_path):
    """A background persist reads the arena; the next window waits for it
    (Sec. 4.4.3's wait-for-previous rule) even when it needs a larger arena,
    so the checkpoint on disk is the one restored."""
    from paper_2511_07035_amd import Session, gockpt_read_checkpoint

    n, seed = 300_007, 90
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, seed)
    sync = oracle.State(p0)
    grads = [synth.grads_cpu(n, seed, s) for s in range(1, 7)]
    s = Session(n, ring_bytes=1 << 20, copy_bytes=64 << 10)
    print(f"[case] background persist then a larger window n={n}", flush=True)
    try:
        load_state(s, p0, w=sync.w)
        s.begin_window([0, 100_000, n])
        for k in range(2):
            s.backward_begin()
            to_device_grad16(s, grads[k])
            s.step(cfg.lr)
            oracle.adamw_step(sync, grads[k], cfg)
        s.drain(blocking=True)
        s.restore()
        want = sync.copy()
        d = str(tmp_path / "ck")
        s.persist(d, nthreads=2, async_=True)
        # a 4-part window needs more arena than the 2-part one: reallocated
        s.begin_window([0, 80_000, 160_000, 240_000, n])
        for k in range(2, 6):
            s.backward_begin()
            to_device_grad16(s, grads[k])
            s.step(cfg.lr)
            oracle.adamw_step(sync, grads[k], cfg)
        s.drain(blocking=True)
        s.restore()
        assert getattr(s, "persist_error", None) is None
    finally:
        s.close()
    p, m, v, info, _ = gockpt_read_checkpoint(d, n)
    assert info.t == 2
    assert_bits_equal(p, want.p, "persisted master")
    assert_bits_equal(m, want.m, "persisted exp_avg")
    assert_bits_equal(v, want.v, "persisted exp_avg_sq")
