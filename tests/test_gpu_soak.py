"""Soak: random windows on several contexts, every checkpoint bitwise against
the oracle's synchronous run.  Each context draws its size (up to 3M
elements), copy size, ring (none to 1 MiB), staging slots, worker threads,
gradient format and timing; each window its length (1-11), bounds, wait
policy, pinned or pageable arena, in-window replay, ring plan, ring off,
deferred copies, whether the host queues the whole window ahead of the
device, and planted infs under dynamic loss scaling; plain steps run between
windows.  By default one seed, 2 contexts of 12 windows; GOCKPT_SOAK="A-B C W"
runs seeds A..B with C contexts of W windows each (a longer run took 10
seeds of 6 contexts of 60 windows, all bitwise)."""
import ctypes
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bits_equal, load_state, to_device_grad16

pytestmark = pytest.mark.gpu


def _plan():
    spec = os.environ.get("GOCKPT_SOAK", "").split()
    if not spec:
        return [(7, 2, 12)]
    a, _, b = spec[0].partition("-")
    seeds = range(int(a), int(b or a) + 1)
    return [(sd, int(spec[1]) if len(spec) > 1 else 4, int(spec[2]) if len(spec) > 2 else 30) for sd in seeds]


@pytest.mark.parametrize("seed0,n_ctx,n_win", _plan())
def test_random_windows_soak(seed0, n_ctx, n_win):
    import torch
    from paper_2511_07035_amd import BENCH_LIB_PATH, Session

    bl = ctypes.CDLL(BENCH_LIB_PATH)
    bl.gockpt_bench_spin.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_int]
    for ci in range(n_ctx):
        rng = np.random.default_rng(seed0 * 1000 + ci)
        n = int(rng.integers(20_000, 200_000)) if rng.random() < 0.7 else int(rng.integers(200_000, 3_000_000))
        copy_bytes = int(rng.choice([4096, 8192, 16384, 65536]))
        ring_bytes = int(rng.choice([0, 16, 64, 256, 1024])) * 1024
        slots = int(rng.integers(2, 9))
        fp16 = bool(rng.random() < 0.3)
        gdt = "fp16" if fp16 else "bf16"
        cfg = oracle.AdamWConfig(dynamic_scale=True, init_scale=4096.0, growth_interval=5, grad_dtype=gdt)
        p0 = synth.master_cpu(n, 500 + ci)
        sync = oracle.State(p0, scale=4096.0)
        print(f"[case] soak seed {seed0} ctx {ci}: n={n} copy={copy_bytes} ring={ring_bytes} slots={slots} "
              f"grads={gdt}", flush=True)
        sess = Session(n, dynamic_scale=True, init_scale=4096.0, growth_interval=5, ring_bytes=ring_bytes,
                       copy_bytes=copy_bytes, staging_bytes=slots * copy_bytes, copy_threads=int(rng.integers(1, 5)),
                       timing=bool(rng.random() < 0.5), grad_dtype=gdt)
        gstep = 0
        try:
            load_state(sess, p0, w=sync.w)
            for win in range(n_win):
                K = int(rng.integers(1, 12))
                cuts = np.sort(rng.choice(np.arange(1, n // 8), size=K - 1, replace=False)) * 8 if K > 1 else []
                bounds = [0, *map(int, cuts), n]
                policy = int(rng.integers(0, 3))
                pageable = bool(rng.random() < 0.4) and policy == 0
                R = int(rng.integers(1, K)) if (K > 2 and rng.random() < 0.3) else 0
                late = int(rng.integers(0, 3))
                ring_off = bool(rng.random() < 0.15)
                defer = bool(rng.random() < 0.4) and policy == 0
                ahead = bool(rng.random() < 0.3)
                for _ in range(int(rng.integers(0, 3))):  # plain steps between windows
                    gstep += 1
                    g = synth.grads_cpu(n, 500 + ci, gstep, scale=sync.scale, plant_inf=rng.random() < 0.1, dtype=gdt)
                    sess.backward_begin()
                    to_device_grad16(sess, g)
                    sess.step(cfg.lr)
                    oracle.adamw_step(sync, g, cfg)
                sess.begin_window(bounds, replay_every=R, pageable=pageable, wait_policy=policy, ring_off=ring_off,
                                  late_plan=late, defer_copies=defer)
                grads = []
                for s in range(K):
                    gstep += 1
                    grads.append(synth.grads_cpu(n, 500 + ci, gstep, scale=sync.scale, plant_inf=rng.random() < 0.1,
                                                 dtype=gdt))
                if ahead:  # every step queued while a 20 ms kernel holds the compute stream
                    dev = [torch.from_numpy(g.view(np.int16)).to("cuda") for g in grads]
                    torch.cuda.synchronize()
                    assert bl.gockpt_bench_spin(sess.compute.cuda_stream, 20.0, 1) == 0
                for s in range(K):
                    sess.backward_begin()
                    if ahead:
                        with torch.cuda.stream(sess.compute):
                            sess.grad.view(torch.int16).copy_(dev[s])
                    else:
                        to_device_grad16(sess, grads[s])
                    sess.step(cfg.lr)
                    oracle.adamw_step(sync, grads[s], cfg)
                st = sess.drain(blocking=True)
                assert st.steps_done == K
                outs = (np.empty(n, np.float32), np.empty(n, np.float32), np.empty(n, np.float32),
                        np.empty(n, np.uint16))
                meta = sess.restore(nthreads=int(rng.integers(1, 5)), out=outs)
                tag = (f"seed {seed0} ctx {ci} window {win} K={K} pol={policy} pg={pageable} R={R} late={late} "
                       f"off={ring_off} defer={defer} ahead={ahead}")
                assert_bits_equal(outs[0], sync.p, tag + " master")
                assert_bits_equal(outs[1], sync.m, tag + " m")
                assert_bits_equal(outs[2], sync.v, tag + " v")
                assert np.array_equal(outs[3], sync.w), tag + " w"
                assert (meta.t, meta.scale, meta.tracker) == (sync.t, sync.scale, sync.tracker), tag
            p, m, v, w = sess.state_to_host()
            assert_bits_equal(p, sync.p, f"ctx {ci}: device master")
        finally:
            sess.close()
