"""Error paths, forced from the host: a device-to-host copy that reports an
error (GOCKPT_TEST_FAIL_COPY makes the N-th window copy of a context fail
without reaching the device -- no kernel faults).  The window must turn
FAILED, drain and restore must refuse it, abort must recover, the device
state must be the oracle's after the updates that ran, and the next window
must work and restore bit for bit."""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bits_equal, load_state, to_device_grad16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("defer", [False, True])
@pytest.mark.parametrize("pageable", [False, True])
def test_failed_copy_poisons_the_window_and_abort_recovers(pageable, defer):
    """defer: the window queues each step's copies at the next library call,
    so the failing copy is queued (and its error reported) by the next
    step's gockpt_backward_begin, or by the drain."""
    from paper_2511_07035_amd import GOCKPT_EFAILED, GockptError, Session

    n, seed = 50_003, 5 + int(pageable)
    cfg = oracle.AdamWConfig()
    p0 = synth.master_cpu(n, seed)
    grads = [synth.grads_cpu(n, seed, s) for s in range(1, 12)]
    print(f"[case] failed copy pageable={pageable} defer={defer}", flush=True)
    os.environ["GOCKPT_TEST_FAIL_COPY"] = "4"
    try:
        sess = Session(n, ring_bytes=64 << 10, copy_bytes=16 << 10, staging_bytes=4 * (16 << 10), copy_threads=2)
    finally:
        del os.environ["GOCKPT_TEST_FAIL_COPY"]
    try:
        load_state(sess, p0)
        sess.begin_window([0, 8, 20_000, 40_000, n], pageable=pageable, defer_copies=defer)
        used = 0
        failed = None
        for s in range(4):
            try:
                sess.backward_begin()
                to_device_grad16(sess, grads[used])
                sess.step(cfg.lr)
            except GockptError as e:
                failed = e
                break
            finally:
                used += 1
        if failed is None:  # the error surfaced only at the drain (deferred or staged copies)
            with pytest.raises(GockptError) as ei:
                sess.drain(blocking=True)
            failed = ei.value
        assert failed is not None
        with pytest.raises(GockptError) as ei:
            sess.restore()
        assert ei.value.code in (GOCKPT_EFAILED, -2)
        sess.abort_window()
        # the device state is the oracle's after the updates that ran
        t, _, _ = sess.scaler()
        sync = oracle.State(p0)
        for k in range(t):
            oracle.adamw_step(sync, grads[k], cfg)
        p, m, v, w = sess.state_to_host()
        assert_bits_equal(p, sync.p, "master after the failed window")
        assert_bits_equal(v, sync.v, "exp_avg_sq after the failed window")
        # abort waited for every copy, so a plain step may overwrite the
        # gradients at once (no gockpt_backward_begin needed)
        to_device_grad16(sess, grads[t])
        sess.step(cfg.lr)
        oracle.adamw_step(sync, grads[t], cfg)
        # the next window, shorter than the failed one, works and restores
        # exactly
        sess.begin_window([0, 24_000, n], pageable=pageable, defer_copies=defer)
        for k in range(t + 1, t + 3):
            sess.backward_begin()
            to_device_grad16(sess, grads[k])
            sess.step(cfg.lr)
            oracle.adamw_step(sync, grads[k], cfg)
        sess.drain(blocking=True)
        outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
        meta = sess.restore(out=outs)
        assert_bits_equal(outs[0], sync.p, "restored master after recovery")
        assert_bits_equal(outs[2], sync.v, "restored exp_avg_sq after recovery")
        assert meta.t == sync.t
    finally:
        sess.close()
