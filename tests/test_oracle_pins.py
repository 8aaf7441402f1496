"""Pins of the CPU oracle against facts that do not come from the oracle.

The oracle (oracle/gockpt_oracle.c) is what the HIP path is compared with, so
it is pinned here first:
  * 16-bit rounding against torch's own float32 -> bfloat16 conversion and
    against exact nearest-neighbour arithmetic;
  * Adam's closed forms in exact rational arithmetic: one step from zero
    moments, a constant gradient for t steps, a zero gradient;
  * bias-correction powers against exact rational powers;
  * the loss-scaler sequence of the dynamic-scaling workload (hand-derived
    fixture) and brute-force skip semantics;
  * the window invariant of Sec. 4.3.1 -- replaying the captured parts gives
    the synchronous result -- over every composition of tiny spaces, random
    chunkings and random skip patterns, and the paper's three-part example
    (Sec. 4.2.1 / Sec. 4.3.1).
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def F(x) -> Fraction:
    return Fraction(float(x))


def ulp32(x) -> float:
    return float(np.spacing(np.float32(abs(float(x)))))


def bf16_value(bits) -> float:
    return float(np.array([int(bits) << 16], dtype=np.uint32).view(np.float32)[0])


# ---------------------------------------------------------------------------
# bf16 rounding
# ---------------------------------------------------------------------------

def _structured_f32_patterns():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x1234, 0xC001], dtype=np.uint32)
    return (hi[:, None] | lows[None, :]).reshape(-1)


def test_bf16_rne_matches_torch_conversion(oracle_lib):
    bits = _structured_f32_patterns()
    rng = np.random.default_rng(1)
    bits = np.concatenate([bits, rng.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32)])
    x = bits.view(np.float32)
    ours = oracle_lib.bf16_rne_array(x)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.all(ours[nan] == 0x7FC0)


def test_bf16_rne_is_nearest_even_exactly(oracle_lib):
    """Exact nearest-neighbour check, independent of any bit trick."""
    rng = np.random.default_rng(2)
    bits = np.concatenate([rng.integers(0, 1 << 32, 20000, dtype=np.uint64).astype(np.uint32),
                           np.array([0x7F7F8000, 0x7F7F7FFF, 0x7F7FFFFF, 0x00008000, 0x00018000,
                                     0x80008000, 0x3F808000, 0x3F818000], dtype=np.uint32)])
    for b in bits:
        x = float(np.array([b], dtype=np.uint32).view(np.float32)[0])
        if math.isnan(x):
            continue
        got = oracle_lib.bf16_rne(x)
        if math.isinf(x):
            assert got == (b >> 16)
            continue
        lo = int(b) & 0xFFFF0000
        lo_bits = lo >> 16
        hi_bits = lo_bits + 1
        lo_v = F(bf16_value(lo_bits))
        # the neighbour one step further from zero; past the largest finite
        # value it is 2^128 (unbounded exponent), which rounds to infinity
        hi_v = F(bf16_value(hi_bits)) if (hi_bits & 0x7F80) != 0x7F80 else Fraction(2 ** 128) * (
            -1 if x < 0 else 1)
        xv = F(x)
        dlo, dhi = abs(xv - lo_v), abs(hi_v - xv)
        if dlo < dhi:
            want = lo_bits
        elif dhi < dlo:
            want = hi_bits
        else:
            want = lo_bits if (lo_bits & 1) == 0 else hi_bits
        assert got == want, hex(b)


def test_bf16_to_f32_exact(oracle_lib):
    for b in [0x0000, 0x8000, 0x3F80, 0xBF80, 0x7F80, 0xFF80, 0x0001, 0x7F7F, 0x4049]:
        want = float(torch.tensor([b], dtype=torch.int16 if b < 0x8000 else torch.int32)
                     .to(torch.int16).view(torch.bfloat16).float()[0]) if b < 0x8000 else None
        got = oracle_lib.bf16_to_f32(b)
        assert np.float32(got).view(np.uint32) == (b << 16)
        if want is not None:
            assert got == want or (math.isnan(got) and math.isnan(want))


# ---------------------------------------------------------------------------
# bias-correction powers and per-step scalars
# ---------------------------------------------------------------------------

def test_powi_exact_for_half(oracle_lib):
    for t in range(0, 1100):
        assert oracle_lib.powi(0.5, t) == math.ldexp(1.0, -t)


@pytest.mark.parametrize("beta", [0.9, 0.999, 0.95, 0.5 + 1e-9])
def test_powi_close_to_exact_power(oracle_lib, beta):
    bd = F(beta)
    for t in list(range(1, 130)) + [257, 1000, 4097]:
        exact = bd ** t
        got = F(oracle_lib.powi(beta, t))
        # squaring doubles a relative error, so square-and-multiply is bounded
        # by about (t - 1) unit roundoffs, like t - 1 successive products
        tol = Fraction(t + 1) * Fraction(1, 2 ** 53) * exact
        if exact < Fraction(1, 2 ** 1000):  # outside the normal range: underflows
            assert got < Fraction(1, 2 ** 990), (beta, t)
            continue
        assert abs(got - exact) <= tol, (beta, t)


def test_step_scalars_against_mathematics(oracle_lib):
    cfg = oracle_lib.AdamWConfig()
    lr = np.float32(1e-4)
    s1 = oracle_lib.step_scalars(cfg, lr, 1, 1.0)
    # t = 1: lr / (1 - beta1) and sqrt(1 - beta2), each within one fp32 ulp
    assert abs(F(s1.step_size) - F(lr) / (1 - F(cfg.beta1))) <= F(ulp32(s1.step_size))
    assert abs(float(s1.sqrt_bc2) - math.sqrt(1 - cfg.beta2)) <= ulp32(s1.sqrt_bc2)
    assert abs(F(s1.decay) - (1 - F(lr) * F(cfg.weight_decay))) <= F(ulp32(s1.decay)) / 2
    assert abs(F(s1.omb1) - (1 - F(cfg.beta1))) <= F(ulp32(s1.omb1)) / 2
    assert abs(F(s1.omb2) - (1 - F(cfg.beta2))) <= F(ulp32(s1.omb2)) / 2
    assert s1.b1 == np.float32(cfg.beta1) and s1.b2 == np.float32(cfg.beta2)
    # far into training the bias corrections vanish exactly
    s_inf = oracle_lib.step_scalars(cfg, lr, 10 ** 6, 1.0)
    assert s_inf.step_size == lr and s_inf.sqrt_bc2 == 1.0
    # the loss-scale reciprocal is exact for powers of two
    for e in range(0, 30):
        assert oracle_lib.step_scalars(cfg, lr, 3, float(2 ** e)).inv_scale == 2.0 ** -e


# ---------------------------------------------------------------------------
# Adam closed forms
# ---------------------------------------------------------------------------

HP_SETS = [
    dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01),
    dict(lr=0.1, beta1=0.8, beta2=0.99, eps=1e-3, weight_decay=0.5),
    dict(lr=3e-3, beta1=0.95, beta2=0.98, eps=1e-6, weight_decay=0.0),
]


def _case_values():
    rng = np.random.default_rng(3)
    gs = np.concatenate([rng.normal(0, 1e-3, 40), rng.normal(0, 1e-6, 20), rng.normal(0, 1.0, 20),
                         [1e-8, -1e-8, 2e-3, -5.0]]).astype(np.float32)
    g_bits = synth._bf16_bits_cpu(gs)
    p0 = np.concatenate([rng.normal(0, 0.02, 60), rng.normal(0, 1e-4, 24)]).astype(np.float32)
    return p0, g_bits


@pytest.mark.parametrize("hp", HP_SETS)
@pytest.mark.parametrize("scale", [1.0, 1024.0])
def test_single_step_closed_form(oracle_lib, hp, scale):
    """t = 1 from m = v = 0: m = (1-b1) g, v = (1-b2) g^2, the bias-corrected
    ratio is g/(|g|+eps), so p1 = p0 (1 - lr wd) - lr g/(|g| + eps)."""
    cfg = oracle_lib.AdamWConfig(**hp, init_scale=scale)
    p0, g_bits = _case_values()
    # gradients carry the loss scale: multiply the drawn value by it
    g_scaled = synth._bf16_bits_cpu(np.array([bf16_value(b) * scale for b in g_bits], dtype=np.float32))
    st = oracle_lib.State(p0, scale=scale)
    oracle_lib.adamw_step(st, g_scaled, cfg)
    lr = F(np.float32(hp["lr"]))
    c = 1 - lr * F(hp["weight_decay"])
    for i in range(p0.size):
        g = F(bf16_value(g_scaled[i])) / F(scale)
        delta = lr * g / (abs(g) + F(hp["eps"]))
        want_p = F(p0[i]) * c - delta
        tol_p = 4 * max(ulp32(float(F(p0[i]) * c)), ulp32(float(delta)))
        assert abs(F(st.p[i]) - want_p) <= F(tol_p), (i, float(st.p[i]), float(want_p))
        want_m = (1 - F(hp["beta1"])) * g
        want_v = (1 - F(hp["beta2"])) * g * g
        assert abs(F(st.m[i]) - want_m) <= F(2 * ulp32(float(want_m))) + F(1e-45)
        assert abs(F(st.v[i]) - want_v) <= F(3 * ulp32(float(want_v))) + F(1e-45)
    assert st.t == 1


@pytest.mark.parametrize("hp", HP_SETS)
def test_constant_gradient_closed_form(oracle_lib, hp):
    """A constant gradient g for t steps from zero moments: the bias-corrected
    moments are exactly g and g^2 in real arithmetic, so each step subtracts
    lr g/(|g|+eps) after the decay: p_t = p0 c^t - lr s (1 + c + ... + c^{t-1})."""
    cfg = oracle_lib.AdamWConfig(**hp)
    T = 40
    p0 = np.array([0.02, -0.013, 1e-4, 0.5], dtype=np.float32)
    g_vals = np.array([1e-3, -2e-4, 3e-6, 0.25], dtype=np.float32)
    g_bits = synth._bf16_bits_cpu(g_vals)
    st = oracle_lib.State(p0)
    grads = np.tile(g_bits, (T, 1))
    oracle_lib.sync_run(st, grads, cfg)
    lr = F(np.float32(hp["lr"]))
    c = 1 - lr * F(hp["weight_decay"])
    for i in range(p0.size):
        g = F(bf16_value(g_bits[i]))
        s = g / (abs(g) + F(hp["eps"]))
        geo = sum(c ** k for k in range(T))
        want = F(p0[i]) * c ** T - lr * s * geo
        # rounding of p each step plus the contract's fp32 moment
        # coefficients (b + (1-b) differs from 1 by < 7e-8 per step)
        tol = 2 * T * max(ulp32(float(want)), ulp32(p0[i])) + 1e-5 * float(abs(lr * s * geo))
        assert abs(float(F(st.p[i]) - want)) <= tol, (i, hp)
        want_m = (1 - F(hp["beta1"]) ** T) * g
        want_v = (1 - F(hp["beta2"]) ** T) * g * g
        assert abs(float(F(st.m[i]) - want_m)) <= 1e-6 * abs(float(want_m)) + 4 * T * ulp32(float(want_m))
        assert abs(float(F(st.v[i]) - want_v)) <= 1e-5 * abs(float(want_v)) + 4 * T * ulp32(float(want_v))
    assert st.t == T


def test_zero_gradient_only_decays(oracle_lib):
    cfg = oracle_lib.AdamWConfig(lr=0.05, weight_decay=0.3)
    p0 = np.array([1.0, -0.75, 3e-3, 1e-30], dtype=np.float32)
    T = 25
    st = oracle_lib.State(p0)
    oracle_lib.sync_run(st, np.zeros((T, p0.size), dtype=np.uint16), cfg)
    decay = oracle_lib.step_scalars(cfg, np.float32(cfg.lr), 1, 1.0).decay
    assert np.all(st.m == 0) and np.all(st.v == 0)
    for i in range(p0.size):
        want = F(p0[i]) * F(decay) ** T
        assert abs(F(st.p[i]) - want) <= F(T * ulp32(float(want))) + F(1e-45)
    assert st.t == T


def test_bf16_weights_follow_master(oracle_lib):
    cfg = oracle_lib.AdamWConfig()
    n = 3000
    st = oracle_lib.State(synth.master_cpu(n, 5))
    oracle_lib.sync_run(st, np.stack([synth.grads_cpu(n, 5, s) for s in range(1, 4)]), cfg)
    ref = torch.from_numpy(st.p.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(st.w, ref)


def test_nonfinite_scan_and_norm_bruteforce(oracle_lib):
    n = 5000
    g = synth.grads_cpu(n, 9, 1)
    assert not oracle_lib.any_nonfinite(g)
    vals = torch.from_numpy(g.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    assert oracle_lib.grad_norm2(g, 1.0) == pytest.approx(float(np.sum(vals * vals)), rel=1e-12)
    for bad in (0x7F80, 0xFF80, 0x7FC0, 0x7F81, 0xFFFF):
        h = g.copy()
        h[1234] = bad
        assert oracle_lib.any_nonfinite(h)
    h = g.copy()
    h[77] = 0x7F7F  # largest finite
    assert not oracle_lib.any_nonfinite(h)


# ---------------------------------------------------------------------------
# fp16 gradients (Sec. 2.2 allows FP16 or BF16)
# ---------------------------------------------------------------------------

ALL16 = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)


def test_fp16_decode_matches_numpy_all_patterns(oracle_lib):
    """binary16 -> fp32 for every one of the 65536 patterns against numpy's
    float16 conversion (NaNs compared as NaN)."""
    ref = ALL16.view(np.float16).astype(np.float32)
    got = np.array([oracle_lib.fp16_to_f32(int(h)) for h in ALL16], dtype=np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan) and nan.sum() == 2 * 1023
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_fp16_nonfinite_and_norm(oracle_lib):
    """A gradient is non-finite exactly when numpy calls its float16 value inf
    or NaN; the norm is the fp64 sum of the exactly decoded squares."""
    finite = np.isfinite(ALL16.view(np.float16))
    for h in ALL16[::97]:  # a spread of patterns across every exponent
        assert oracle_lib.any_nonfinite(np.array([h], np.uint16), "fp16") == (not finite[h])
    for h in (0x7C00, 0xFC00, 0x7C01, 0x7E00, 0xFFFF):
        assert oracle_lib.any_nonfinite(np.array([0, h, 0], np.uint16), "fp16")
        assert not oracle_lib.any_nonfinite(np.array([0, h, 0], np.uint16), "bf16") or (h & 0x7F80) == 0x7F80
    assert not oracle_lib.any_nonfinite(np.array([0x7BFF, 0xFBFF, 0x0001, 0x8001], np.uint16), "fp16")
    g = synth.grads_cpu(5000, 9, 1, dtype="fp16")
    vals = g.view(np.float16).astype(np.float64)
    assert oracle_lib.grad_norm2(g, 0.5, "fp16") == pytest.approx(float(np.sum((vals * 0.5) ** 2)), rel=1e-12)


@pytest.mark.parametrize("hp", HP_SETS)
def test_fp16_single_step_closed_form(oracle_lib, hp):
    """The t = 1 closed form with fp16 gradients, including subnormal ones
    (below 2^-14) and the largest finite one (65504)."""
    cfg = oracle_lib.AdamWConfig(**hp, grad_dtype="fp16")
    rng = np.random.default_rng(11)
    gs = np.concatenate([rng.normal(0, 1e-3, 40), rng.normal(0, 1e-6, 12), [3e-8, -6e-8, 65504.0, -1.0]])
    g16 = gs.astype(np.float16).view(np.uint16)
    p0 = rng.normal(0, 0.02, g16.size).astype(np.float32)
    st = oracle_lib.State(p0)
    oracle_lib.adamw_step(st, g16, cfg)
    lr = F(np.float32(hp["lr"]))
    c = 1 - lr * F(hp["weight_decay"])
    for i in range(p0.size):
        g = F(float(g16[i:i + 1].view(np.float16)[0]))
        delta = lr * g / (abs(g) + F(hp["eps"]))
        want_p = F(p0[i]) * c - delta
        tol_p = 4 * max(ulp32(float(F(p0[i]) * c)), ulp32(float(delta)))
        assert abs(F(st.p[i]) - want_p) <= F(tol_p), (i, float(st.p[i]), float(want_p))
        want_m = (1 - F(hp["beta1"])) * g
        assert abs(F(st.m[i]) - want_m) <= F(2 * ulp32(float(want_m))) + F(1e-45)
    assert st.t == 1


def test_fp16_window_replay_equals_sync(oracle_lib):
    """The window invariant with fp16 gradients, dynamic scaling and planted
    fp16 infinities (0x7C00)."""
    rng = np.random.default_rng(17)
    for trial in range(20):
        n = int(rng.integers(8, 2000))
        K = min(int(rng.integers(1, 10)), n)
        cuts = np.sort(rng.choice(np.arange(1, n), size=K - 1, replace=False)) if K > 1 else []
        bounds = [0, *map(int, cuts), n]
        cfg = oracle_lib.AdamWConfig(dynamic_scale=True, init_scale=1024.0, growth_interval=int(rng.integers(1, 4)),
                                     grad_dtype="fp16")
        bad = rng.random(K) < 0.3
        grads = np.stack([synth.grads_cpu(n, 60 + trial, s, scale=1024.0, plant_inf=bool(bad[s - 1]), dtype="fp16")
                          for s in range(1, K + 1)])
        cap = _check_invariant(oracle_lib, n, bounds, grads, cfg, scale=1024.0)
        assert list(cap.records["skip"]) == [int(b) for b in bad]


# ---------------------------------------------------------------------------
# loss scaler
# ---------------------------------------------------------------------------

def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_dynamic_scale_window_sequence(oracle_lib):
    fx = _load("dynscale_k8.json")
    cfg = oracle_lib.AdamWConfig(dynamic_scale=True, init_scale=fx["init_scale"], growth_factor=2.0,
                                 backoff_factor=0.5, growth_interval=fx["growth_interval"])
    n = 4096
    K = len(fx["scale_used"])
    grads = np.stack([synth.grads_cpu(n, 11, s, scale=synth.DYNSCALE_SCHEDULE[s],
                                      plant_inf=s in fx["inf_steps"]) for s in range(1, K + 1)])
    st = oracle_lib.State(synth.master_cpu(n, 11), scale=fx["init_scale"])
    recs = oracle_lib.sync_run(st, grads, cfg)
    assert [float(r) for r in recs["scale_used"]] == fx["scale_used"]
    assert [int(r) for r in recs["t"]] == fx["t_after"]
    assert [int(r) for r in recs["skip"]] == fx["skip"]
    assert st.t == fx["final"]["t"] and st.scale == fx["final"]["scale"] and st.tracker == fx["final"]["tracker"]


def test_scaler_growth_and_backoff(oracle_lib):
    fx = _load("scaler_growth.json")
    cfg = oracle_lib.AdamWConfig(dynamic_scale=True, init_scale=fx["init_scale"], growth_factor=2.0,
                                 backoff_factor=0.5, growth_interval=fx["growth_interval"],
                                 min_scale=fx["min_scale"])
    n = 64
    seq = fx["nonfinite"]
    st = oracle_lib.State(np.zeros(n, dtype=np.float32), scale=fx["init_scale"])
    got_scale, got_tracker = [], []
    for k, bad in enumerate(seq):
        g = np.zeros(n, dtype=np.uint16)
        if bad:
            g[5] = 0x7F80
        oracle_lib.adamw_step(st, g, cfg)
        got_scale.append(float(st.scale))
        got_tracker.append(int(st.tracker))
    assert got_scale == fx["scale_after"]
    assert got_tracker == fx["tracker_after"]


def test_skipped_steps_are_noops(oracle_lib):
    """Brute force: a run with planted infs equals a run over only the clean
    steps, each with the loss scale it carried."""
    cfg = oracle_lib.AdamWConfig(dynamic_scale=True, init_scale=65536.0)
    n = 2000
    K = 8
    inf_steps = {3, 7}
    grads = np.stack([synth.grads_cpu(n, 12, s, scale=synth.DYNSCALE_SCHEDULE[s], plant_inf=s in inf_steps)
                      for s in range(1, K + 1)])
    a = oracle_lib.State(synth.master_cpu(n, 12), scale=65536.0)
    oracle_lib.sync_run(a, grads, cfg)
    b = oracle_lib.State(synth.master_cpu(n, 12), scale=65536.0)
    static = oracle_lib.AdamWConfig()
    for s in range(1, K + 1):
        if s in inf_steps:
            continue
        b.scaler.scale = synth.DYNSCALE_SCHEDULE[s]
        oracle_lib.adamw_step(b, grads[s - 1], static)
    assert np.array_equal(a.p, b.p) and np.array_equal(a.m, b.m) and np.array_equal(a.v, b.v)
    assert np.array_equal(a.w, b.w) and a.t == b.t == K - len(inf_steps)


def test_overflow_check_off_applies_every_step(oracle_lib):
    """With the overflow test off no step is skipped: the element holding
    +inf gets m = +inf, v = +inf and a NaN master weight (inf / inf in the Adam
    ratio), whose bf16 copy is the canonical 0x7FC0; the update is
    elementwise, so every other element equals a run in which that gradient
    was finite."""
    n = 3000
    cfg = oracle_lib.AdamWConfig(check_overflow=False)
    g = synth.grads_cpu(n, 13, 1, plant_inf=True)
    i = synth.inf_index(n, 13, 1)
    assert g[i] == 0x7F80
    a = oracle_lib.State(synth.master_cpu(n, 13))
    rec = oracle_lib.adamw_step(a, g, cfg)
    assert a.t == 1 and int(rec["skip"][0]) == 0 and np.isinf(rec["gnorm2"][0])
    assert np.isposinf(a.m[i]) and np.isposinf(a.v[i]) and np.isnan(a.p[i]) and a.w[i] == 0x7FC0
    g2 = g.copy()
    g2[i] = 0x3F80  # 1.0
    b = oracle_lib.State(synth.master_cpu(n, 13))
    oracle_lib.adamw_step(b, g2, cfg)
    keep = np.arange(n) != i
    for x, y in ((a.p, b.p), (a.m, b.m), (a.v, b.v), (a.w, b.w)):
        assert np.array_equal(x[keep], y[keep])
    # with the test on, the same gradients leave everything as it was
    c = oracle_lib.State(synth.master_cpu(n, 13))
    oracle_lib.adamw_step(c, g, oracle_lib.AdamWConfig())
    assert c.t == 0 and np.array_equal(c.p, synth.master_cpu(n, 13))


# ---------------------------------------------------------------------------
# the multi-step window (Sec. 4.2.1) and its reconstruction (Sec. 4.3.1)
# ---------------------------------------------------------------------------

def _compositions(n, k):
    for cuts in itertools.combinations(range(1, n), k - 1):
        yield [0, *cuts, n]


def _check_invariant(oracle_lib, n, bounds, grads, cfg, lrs=None, nonfinite=None, p0=None, scale=1.0):
    p0 = synth.master_cpu(n, 21) if p0 is None else p0
    sync = oracle_lib.State(p0, scale=scale)
    recs = oracle_lib.sync_run(sync, grads, cfg, lrs=lrs, nonfinite=nonfinite)
    win = oracle_lib.State(p0, scale=scale)
    cap = oracle_lib.window_capture(win, grads, bounds, cfg, lrs=lrs, nonfinite=nonfinite)
    assert np.array_equal(cap.records, recs)
    p, m, v, w = oracle_lib.replay_restore(cap, cfg)
    assert np.array_equal(p, sync.p) and np.array_equal(m, sync.m) and np.array_equal(v, sync.v)
    assert np.array_equal(w, sync.w)
    # the window itself leaves the live state at the synchronous state too
    assert np.array_equal(win.p, sync.p)
    return cap


def test_replay_equals_sync_all_compositions(oracle_lib):
    cfg = oracle_lib.AdamWConfig(lr=1e-2)
    count = 0
    for n in range(1, 11):
        for K in range(1, min(n, 8) + 1):
            grads = np.stack([synth.grads_cpu(n, 31, s) for s in range(1, K + 1)])
            for bounds in _compositions(n, K):
                _check_invariant(oracle_lib, n, bounds, grads, cfg)
                count += 1
    assert count > 900


def test_replay_equals_sync_random_windows(oracle_lib):
    rng = np.random.default_rng(7)
    for trial in range(60):
        n = int(rng.integers(8, 3000))
        K = int(rng.integers(1, 17))
        K = min(K, n)
        cuts = np.sort(rng.choice(np.arange(1, n), size=K - 1, replace=False)) if K > 1 else []
        bounds = [0, *map(int, cuts), n]
        dynamic = bool(trial % 2)
        cfg = oracle_lib.AdamWConfig(dynamic_scale=dynamic, init_scale=256.0 if dynamic else 1.0,
                                     growth_interval=int(rng.integers(1, 5)))
        lrs = rng.uniform(1e-5, 1e-2, K).astype(np.float32)
        bad = rng.random(K) < 0.25
        grads = np.stack([synth.grads_cpu(n, 40 + trial, s, scale=256.0 if dynamic else 1.0,
                                          plant_inf=bool(bad[s - 1])) for s in range(1, K + 1)])
        cap = _check_invariant(oracle_lib, n, bounds, grads, cfg, lrs=lrs, scale=256.0 if dynamic else 1.0)
        assert list(cap.records["skip"]) == [int(b) for b in bad]


def test_single_step_window_at_last_step(oracle_lib):
    """A window of one part taken at step K sends the whole state after step K;
    the K-step window reconstructs exactly that."""
    cfg = oracle_lib.AdamWConfig()
    n, K = 1000, 6
    grads = np.stack([synth.grads_cpu(n, 51, s) for s in range(1, K + 1)])
    a = oracle_lib.State(synth.master_cpu(n, 51))
    oracle_lib.sync_run(a, grads[:K - 1], cfg)
    cap1 = oracle_lib.window_capture(a, grads[K - 1:], [0, n], cfg)
    b = oracle_lib.State(synth.master_cpu(n, 51))
    capK = oracle_lib.window_capture(b, grads, [0, 100, 208, 400, 640, 896, n], cfg)
    p, m, v, w = oracle_lib.replay_restore(capK, cfg)
    assert np.array_equal(p, cap1.snap_p) and np.array_equal(m, cap1.snap_m) and np.array_equal(v, cap1.snap_v)


def test_paper_three_part_example(oracle_lib):
    """Sec. 4.2.1 / 4.3.1: parts A, B, C; A is sent first and needs the
    gradients of the next two updates, B those of the last update, C none; the
    result equals sending the final state directly."""
    fx = _load("paper_three_part.json")
    n = 24
    bounds = fx["bounds"]
    K = len(bounds) - 1
    cfg = oracle_lib.AdamWConfig(lr=1e-2)
    grads = np.stack([synth.grads_cpu(n, 61, s) for s in range(1, K + 1)])
    cap = _check_invariant(oracle_lib, n, bounds, grads, cfg)
    offs = oracle_lib.sent_offsets(bounds)
    for s in range(1, K + 1):
        parts = fx["grads_sent_at_step"][str(s)]
        covered = sum(bounds[j] - bounds[j - 1] for j in (fx["part_index"][p] for p in parts))
        assert offs[s] - offs[s - 1] == covered
        assert np.array_equal(cap.sent[offs[s - 1]:offs[s]], grads[s - 1][:covered])
    for part, steps in fx["replayed_steps"].items():
        j = fx["part_index"][part]
        assert steps == list(range(j + 1, K + 1))


def test_bf16_rne_exhaustive_all_fp32_patterns(oracle_lib):
    """The oracle's bf16 rounding (keep/drop comparison) against the integer
    form of round-to-nearest-even -- add 0x7FFF plus the lowest kept bit,
    shift right 16; NaN handled apart -- over every one of the 2^32 fp32
    patterns."""
    chunk = 1 << 26
    idx = np.arange(chunk, dtype=np.uint32)
    x = np.empty(chunk, np.uint32)
    t = np.empty(chunk, np.uint32)
    got = np.empty(chunk, np.uint16)
    lib = oracle_lib.lib()
    for base in range(0, 1 << 32, chunk):
        np.add(idx, np.uint32(base), out=x)
        lib.oracle_bf16_rne_array(chunk, x.ctypes.data, got.ctypes.data)
        np.right_shift(x, 16, out=t)
        np.bitwise_and(t, 1, out=t)
        np.add(t, x, out=t)
        np.add(t, np.uint32(0x7FFF), out=t)
        np.right_shift(t, 16, out=t)
        want = t.astype(np.uint16)
        np.bitwise_and(x, np.uint32(0x7FFFFFFF), out=t)
        want[t > np.uint32(0x7F800000)] = 0x7FC0
        if not np.array_equal(got, want):
            i = int(np.flatnonzero(got != want)[0])
            raise AssertionError(f"pattern {int(x[i]):#010x}: got {int(got[i]):#06x} want {int(want[i]):#06x}")
