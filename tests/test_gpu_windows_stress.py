"""Many save windows on one context, back to back: random window lengths and
bounds, small rings that wrap and spill, every wait policy and ring plan,
copies queued by the step or deferred to the next call, pinned and pageable
arenas, loss-scale skips, and plain steps between the
windows.  Each window's restored checkpoint, and the device state throughout,
must equal the oracle's synchronous run bit for bit -- nothing may leak from
one window into the next (ring bookkeeping, event pools, staging slots,
replay batches)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bits_equal, load_state, to_device_grad16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("variant", ["bf16", "fp16_caller_flag"])
def test_back_to_back_windows_bitwise(variant):
    """bf16: the library's own overflow test and norm.  fp16_caller_flag: fp16
    gradients, the skip decisions from a caller-side found-inf flag and no
    norm, so no step runs a prepass."""
    import torch
    from paper_2511_07035_amd import Session

    rng = np.random.default_rng(2024)
    n = 120_011
    fp16 = variant == "fp16_caller_flag"
    gdt = "fp16" if fp16 else "bf16"
    cfg = oracle.AdamWConfig(dynamic_scale=True, init_scale=4096.0, growth_interval=5, grad_dtype=gdt)
    p0 = synth.master_cpu(n, 77)
    sync = oracle.State(p0, scale=4096.0)
    flag = torch.zeros(1, dtype=torch.float32, device="cuda") if fp16 else None
    sess = Session(n, dynamic_scale=True, init_scale=4096.0, growth_interval=5, ring_bytes=384 << 10,
                   copy_bytes=32 << 10, staging_bytes=6 * (32 << 10), copy_threads=3, timing=True,
                   grad_dtype=gdt, grad_norm=not fp16, found_inf=flag)
    gstep = 0

    def one_step(in_window: bool):
        nonlocal gstep
        gstep += 1
        bad = rng.random() < 0.12
        g = synth.grads_cpu(n, 77, gstep, scale=sync.scale, plant_inf=bad, dtype=gdt)
        sess.backward_begin()
        to_device_grad16(sess, g)
        if flag is not None:  # the caller's own test of the gradients
            with torch.cuda.stream(sess.compute):
                mask = 0x7C00 if fp16 else 0x7F80  # exponent field all ones: inf or NaN
                flag.fill_(float(np.any((g & mask) == mask)))
        sess.step(cfg.lr)
        oracle.adamw_step(sync, g, cfg)

    try:
        load_state(sess, p0, w=sync.w)
        for win in range(24):
            K = int(rng.integers(1, 10))
            cuts = np.sort(rng.choice(np.arange(1, n // 8), size=K - 1, replace=False)) * 8 if K > 1 else []
            bounds = [0, *map(int, cuts), n]
            policy = int(rng.integers(0, 3))
            pageable = bool(rng.random() < 0.4) and policy == 0
            replay_every = int(rng.integers(1, K)) if (K > 2 and rng.random() < 0.3) else 0
            late = int(rng.integers(0, 3))  # ring plan: QUERY, HOST_WAIT, DEVICE_WAIT
            ring_off = bool(rng.random() < 0.2)
            defer = bool(rng.random() < 0.5) and policy == 0  # copies queued at the next library call
            print(f"[case] window {win}: K={K} policy={policy} pageable={pageable} R={replay_every} late={late} "
                  f"ring_off={ring_off} defer={defer}", flush=True)
            for _ in range(int(rng.integers(0, 3))):
                one_step(False)
            sess.begin_window(bounds, replay_every=replay_every, pageable=pageable, wait_policy=policy,
                              ring_off=ring_off, late_plan=late, defer_copies=defer)
            for _ in range(K):
                one_step(True)
            st = sess.drain(blocking=True)
            assert st.steps_done == K
            times = sess.step_times()
            assert int(times[:, 3].sum()) == st.bytes_ring
            outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32),
                    np.empty(n, np.uint16))
            meta = sess.restore(nthreads=3, out=outs)
            assert_bits_equal(outs[0], sync.p, f"window {win}: restored master")
            assert_bits_equal(outs[1], sync.m, f"window {win}: restored exp_avg")
            assert_bits_equal(outs[2], sync.v, f"window {win}: restored exp_avg_sq")
            assert np.array_equal(outs[3], sync.w), f"window {win}: restored weights"
            assert (meta.t, meta.scale, meta.tracker) == (sync.t, sync.scale, sync.tracker), f"window {win}"
            p, m, v, w = sess.state_to_host()
            assert_bits_equal(p, sync.p, f"window {win}: device master")
            assert_bits_equal(v, sync.v, f"window {win}: device exp_avg_sq")
        assert sess.scaler() == (sync.t, sync.scale, sync.tracker)
    finally:
        sess.close()
