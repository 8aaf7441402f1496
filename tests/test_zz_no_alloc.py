"""gockpt_create_noalloc against gockpt_create, through the C ABI: the
context whose device workspace is the library's static scratch array must
compute the same bits as the one with a caller-allocated workspace -- the
device state after every step, the records, what reaches the host and the
restored checkpoint -- on two contexts in a row, the second over a smaller
flat space (the scratch keeps the first one's contents)."""
import numpy as np
import pytest

import synth
from gpu_util import assert_bits_equal, load_state, to_device_grad16

pytestmark = pytest.mark.gpu


def _drive(sess, p0, grads, bounds, lr, plain_after):
    """A window over `bounds` with the given gradients, then plain steps;
    the device state after every step, the records, the arena and the
    restored outputs."""
    n = p0.size
    K = len(bounds) - 1
    load_state(sess, p0)
    states = []
    sess.begin_window(bounds, late_plan=2)
    for s in range(K + plain_after):
        sess.backward_begin()
        to_device_grad16(sess, grads[s])
        sess.step(lr)
        states.append(sess.state_to_host())
        if s == K - 1:
            stats = sess.drain(blocking=True)
    recs = sess.records().copy()
    arena = tuple(a.copy() for a in sess.arena_state())
    outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.uint16))
    meta = sess.restore(nthreads=4, out=outs)
    return states, recs, arena, outs, meta, stats


@pytest.mark.parametrize("dynamic", [False, True])
def test_noalloc_context_matches_caller_workspace(dynamic):
    from paper_2511_07035_amd import Session

    for n, bounds, seed in ((300_017, [0, 8, 90_000, 200_000, 300_017], 91),
                            (40_009, [0, 16, 20_000, 40_009], 92)):
        print(f"[case] noalloc n={n} K={len(bounds) - 1} dynamic={dynamic}", flush=True)
        K = len(bounds) - 1
        steps = K + 2
        scale = 65536.0 if dynamic else 1.0
        p0 = synth.master_cpu(n, seed)
        grads = np.stack([synth.grads_cpu(n, seed, s, scale=scale, plant_inf=dynamic and s == 2)
                          for s in range(1, steps + 1)])
        res = []
        for noalloc in (False, True):
            sess = Session(n, ring_bytes=256 << 10, copy_bytes=32 << 10, dynamic_scale=dynamic, init_scale=scale,
                           noalloc=noalloc)
            try:
                res.append(_drive(sess, p0, grads, bounds, 1e-4, steps - K))
                assert sess.scaler() is not None
            finally:
                sess.close()
        (sa, ra, aa, oa, ma, ta), (sb, rb, ab, ob, mb, tb) = res
        for s, (x, y) in enumerate(zip(sa, sb)):
            for k, what in enumerate(("master", "exp_avg", "exp_avg_sq")):
                assert_bits_equal(y[k], x[k], f"n={n} step {s + 1}: {what}")
            assert np.array_equal(y[3], x[3]), f"n={n} step {s + 1}: bf16 weights"
        for f in ("t", "skip", "scale_used", "step_size", "sqrt_bc2", "decay", "inv_scale"):
            assert np.array_equal(rb[f], ra[f]), f"record field {f}"
        for k in range(3):
            assert_bits_equal(ab[k], aa[k], f"n={n}: arena array {k}")
            assert_bits_equal(ob[k], oa[k], f"n={n}: restored array {k}")
        assert np.array_equal(ob[3], oa[3])
        assert (mb.t, mb.scale, mb.tracker) == (ma.t, ma.scale, ma.tracker)
        if dynamic:
            assert ma.t == K - 1


def test_noalloc_rules():
    """One no-alloc context per device at a time; no caller workspace or
    staging with it."""
    from paper_2511_07035_amd import GockptError, Session

    a = Session(1024, ring_bytes=0, noalloc=True)
    try:
        with pytest.raises(GockptError, match="EBUSY"):
            Session(1024, ring_bytes=0, noalloc=True)
        with pytest.raises(GockptError, match="EINVAL"):
            Session(1024, ring_bytes=0, noalloc=True, staging_bytes=2 << 20, copy_bytes=1 << 20)
    finally:
        a.close()
    b = Session(2048, ring_bytes=0, noalloc=True)  # free again after destroy
    b.close()
