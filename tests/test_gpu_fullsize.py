"""Full-size parity on sampled elements, in the launch configuration bench.py
times (same bounds, ring, copy size).

The workloads run at their real sizes on device-generated inputs.  A sample of
element indices -- every part boundary with its neighbours, the first and
last elements, and ~32K random ones -- is gathered at every stage: the initial
state, each step's gradients, the device state after the window, what reached
the host arena (each part after its own step, and the gradient blocks), and
the replayed checkpoint.  The oracle recomputes those elements one by one
(each element's result depends only on its own inputs and on the step's skip
decision, which torch decides here from the whole gradient, independently of
the library) and everything is compared bit for bit.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_bits_equal

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _sample(n, bounds, count, seed):
    rng = np.random.default_rng(seed)
    parts = [rng.integers(0, n, count), np.arange(min(16, n)), np.arange(max(0, n - 16), n)]
    for b in bounds:
        parts.append(np.arange(max(0, b - 8), min(n, b + 8)))
    return np.unique(np.concatenate(parts).astype(np.int64))


def _nonfinite_any(torch, grad):
    """torch's own test of the whole gradient for inf/NaN (exponent field all
    ones), independent of the library."""
    mask = 0x7C00 if grad.dtype == torch.float16 else 0x7F80
    bits = grad.view(torch.int16)
    n = bits.numel()
    step = 1 << 28
    for a in range(0, n, step):
        x = bits[a:a + step]
        if bool(((x & mask) == mask).any()):
            return True
    return False


def run_fullsize(workload: str, seed: int = 0, count: int = 1 << 15, pageable: bool = False, replay_every: int = 0,
                 staging_bytes: int = 0, ring_bytes=None, grad_dtype: str = "bf16", caller_flag: bool = False):
    """caller_flag: the skip decisions come from a found-inf flag that torch's
    own test writes before each step, and no norm is computed (no prepass)."""
    import torch

    from paper_2511_07035_amd import GOCKPT_ALIGN_ELEMS, Session, gockpt_plan_bounds

    wl = synth.WORKLOADS[workload]
    layout = synth.LAYOUTS[wl["layout"]]()
    n = synth.numel(layout)
    K = wl["K"]
    if wl["partition"] == "tensors":
        bounds = gockpt_plan_bounds(K, n, synth.tensor_ends(layout))
    else:
        bounds = gockpt_plan_bounds(K, n, align=256 if wl["partition"] == "bytes" else GOCKPT_ALIGN_ELEMS)
    dyn = wl["dynamic"]
    scale0 = 65536.0 if dyn else 1.0
    sched = synth.DYNSCALE_SCHEDULE if dyn else {}
    torch.cuda.empty_cache()
    ring = wl["ring_bytes"] if ring_bytes is None else ring_bytes
    print(f"[fullsize] {workload}: n={n} K={K} ring={ring} pageable={pageable} replay_every={replay_every} "
          f"grads={grad_dtype} caller_flag={caller_flag}", flush=True)

    master = torch.empty(n, dtype=torch.float32, device="cuda")
    synth.master_dev_(master, seed)
    weight = master.to(torch.bfloat16)
    flag = torch.zeros(1, dtype=torch.float32, device="cuda") if caller_flag else None
    sess = Session(n, master=master, weight=weight, dynamic_scale=dyn, init_scale=scale0, ring_bytes=ring,
                   copy_bytes=64 << 20, staging_bytes=staging_bytes, copy_threads=8, grad_dtype=grad_dtype,
                   grad_norm=not caller_flag, found_inf=flag)
    try:
        idx = _sample(n, bounds, count, seed + 1)
        idx_t = torch.from_numpy(idx).cuda()
        torch.cuda.synchronize()
        p0 = master[idx_t].cpu().numpy()
        w0 = weight.view(torch.int16)[idx_t].cpu().numpy().view(np.uint16)
        grads = np.zeros((K, idx.size), dtype=np.uint16)  # raw 16-bit patterns
        nonfinite = np.zeros(K, dtype=np.int32)
        lrs = np.full(K, 1e-4, dtype=np.float32)
        sess.begin_window(bounds, replay_every=replay_every, pageable=pageable)
        for s in range(1, K + 1):
            sess.backward_begin()
            with torch.cuda.stream(sess.compute):
                synth.grads_dev_(sess.grad, seed, s, law=wl["grad"], scale=sched.get(s, 1.0) if dyn else 1.0,
                                 plant_inf=s in wl["inf_steps"])
                grads[s - 1] = sess.grad.view(torch.int16)[idx_t].cpu().numpy().view(np.uint16)
                nonfinite[s - 1] = int(_nonfinite_any(torch, sess.grad))
                if flag is not None:
                    flag.fill_(float(nonfinite[s - 1]))
            sess.step(float(lrs[s - 1]))
            if s % 4 == 0:
                print(f"[fullsize] {workload}: step {s} issued", flush=True)
        st = sess.drain(blocking=True)
        print(f"[fullsize] {workload}: drained {st.bytes_d2h / 1e9:.1f} GB ({st.bytes_spilled / 1e9:.1f} GB "
              f"straight from live buffers)", flush=True)
        recs = sess.records()
        dev_p = master[idx_t].cpu().numpy()
        dev_m = sess.exp_avg[idx_t].cpu().numpy()
        dev_v = sess.exp_avg_sq[idx_t].cpu().numpy()
        dev_w = weight.view(torch.int16)[idx_t].cpu().numpy().view(np.uint16)
        ap, am, av = sess.arena_state()
        snap = (ap[idx].copy(), am[idx].copy(), av[idx].copy())
        replayed = 0 < replay_every < K
        sent = {} if replayed else {s: sess.arena_grads(s)[idx[idx < bounds[s - 1]]].copy() for s in range(2, K + 1)}
        meta = sess.restore(nthreads=16)
        rest = (ap[idx].copy(), am[idx].copy(), av[idx].copy())
        print(f"[fullsize] {workload}: window done, restore {meta.restore_ms:.0f} ms", flush=True)
    finally:
        sess.close()

    cfg = oracle.AdamWConfig(dynamic_scale=dyn, init_scale=scale0, grad_dtype=grad_dtype)
    sb = np.searchsorted(idx, bounds).astype(np.int64)  # part bounds inside the sample
    ora = oracle.State(p0, w=w0, scale=scale0)
    cap = oracle.window_capture(ora, grads, sb, cfg, lrs=lrs, nonfinite=nonfinite)
    assert list(recs["skip"]) == list(cap.records["skip"])
    assert list(recs["t"]) == list(cap.records["t"])
    assert list(recs["scale_used"]) == list(cap.records["scale_used"])
    assert_bits_equal(dev_p, ora.p, f"{workload}: device master after the window")
    assert_bits_equal(dev_m, ora.m, f"{workload}: device exp_avg after the window")
    assert_bits_equal(dev_v, ora.v, f"{workload}: device exp_avg_sq after the window")
    assert np.array_equal(dev_w, ora.w), f"{workload}: device bf16 weights after the window"
    if replayed:
        # the in-window replay already brought every part to the last step
        assert_bits_equal(snap[0], ora.p, f"{workload}: arena master after the in-window replay")
        assert_bits_equal(snap[1], ora.m, f"{workload}: arena exp_avg after the in-window replay")
        assert_bits_equal(snap[2], ora.v, f"{workload}: arena exp_avg_sq after the in-window replay")
    else:
        assert_bits_equal(snap[0], cap.snap_p, f"{workload}: arena master")
        assert_bits_equal(snap[1], cap.snap_m, f"{workload}: arena exp_avg")
        assert_bits_equal(snap[2], cap.snap_v, f"{workload}: arena exp_avg_sq")
        offs = oracle.sent_offsets(sb)
        for s in range(2, K + 1):
            if cap.records["skip"][s - 1]:
                continue
            assert np.array_equal(sent[s], cap.sent[offs[s - 1]:offs[s]]), f"{workload}: gradient block of step {s}"
    assert_bits_equal(rest[0], ora.p, f"{workload}: restored master")
    assert_bits_equal(rest[1], ora.m, f"{workload}: restored exp_avg")
    assert_bits_equal(rest[2], ora.v, f"{workload}: restored exp_avg_sq")
    assert meta.t == ora.t and meta.scale == ora.scale
    return recs, meta


def test_gpt1p3b_k8_fullsize():
    recs, meta = run_fullsize("gpt1p3b_k8")
    assert meta.t == 8 and not recs["skip"].any()


def test_gpt1p3b_k8_dynscale_fullsize():
    recs, meta = run_fullsize("gpt1p3b_k8_dynscale")
    assert list(recs["skip"]) == [0, 0, 1, 0, 0, 0, 1, 0]
    assert meta.t == 6 and meta.scale == 16384.0 and meta.tracker == 1


def test_gpt1p3b_k8_dynscale_fp16_fullsize():
    """fp16 gradients at full size, with fp16 infinities at steps 3 and 7."""
    recs, meta = run_fullsize("gpt1p3b_k8_dynscale", grad_dtype="fp16")
    assert list(recs["skip"]) == [0, 0, 1, 0, 0, 0, 1, 0]
    assert meta.t == 6 and meta.scale == 16384.0


def test_gpt1p3b_k8_dynscale_caller_flag_fullsize():
    """The skip decisions from a caller-side found-inf flag, no norm: no
    prepass reads the 2.6 GB of gradients, the result is the same."""
    recs, meta = run_fullsize("gpt1p3b_k8_dynscale", caller_flag=True)
    assert list(recs["skip"]) == [0, 0, 1, 0, 0, 0, 1, 0]
    assert np.all(recs["gnorm2"] == -1.0)
    assert meta.t == 6 and meta.scale == 16384.0


def test_llama7b_k16_fullsize():
    """6.74e9 elements (108 GB of device state), 16 parts, a 256 MiB ring:
    most of each step's pack is copied straight from the live buffers.  The
    182 GB window does not fit the host's pinned-memory limit, so it lands in
    a pageable arena through 4 GiB of pinned staging."""
    recs, meta = run_fullsize("llama7b_k16", count=1 << 14, pageable=True, staging_bytes=4 << 30)
    assert meta.t == 16


def test_llama13b_k32_fullsize():
    """1.30e10 elements (208 GB of device state), 32 parts at tensor
    boundaries, Laplace gradients.  The 560 GB window cannot be held on the
    host, so the window replays every 2 landed steps onto the parts already
    received (2 gradient slots, 12 n + 4 bounds[31] = 208 GB pageable arena)."""
    recs, meta = run_fullsize("llama13b_k32", count=1 << 14, pageable=True, staging_bytes=4 << 30,
                              replay_every=2, ring_bytes=16 << 30)
    assert meta.t == 32
