"""Window planner (Sec. 4.2.3): the event model of a window checked against the
paper's stall formulas and against brute force, and the planner's search.

Host-only library functions; no GPU.
"""
import itertools

import numpy as np
import pytest

from paper_2511_07035_amd import GockptError, gockpt_plan_window, gockpt_simulate_window

T = 100.0  # ms per plain step in the formula cases: forward 40 + backward 60, free update
PAPER = dict(align=8, state_bytes=14, grad_bytes=2, copy_bytes=1 << 30)  # the paper's 14 B / 2 B accounting


def _link_for(part_bytes: float, ms: float) -> float:
    """GB/s at which part_bytes take ms."""
    return part_bytes / (ms * 1e-3) / 1e9


@pytest.mark.parametrize("N", range(1, 11))
def test_gockpt_explicit_wait_formula(N):
    """Sec. 4.2.3: with one part's state taking one step to transfer and the
    gradients waited for, the stall is sum_i i/7 T_step = N(N-1)/14 T_step."""
    n = 8 * N * 1000
    link = _link_for(14 * n / N, T)
    b = np.arange(N + 1) * (n // N)
    r, per = gockpt_simulate_window(b, n, 40.0, 60.0, 0.0, link, wait_policy=1, **PAPER)
    assert r.stall_ms == pytest.approx(N * (N - 1) / 14 * T, rel=1e-9, abs=1e-9)
    # step s waits for the gradients of s-1 parts: (s-1)/7 T_step
    assert per[:N] == pytest.approx([(s - 1) / 7 * T for s in range(1, N + 1)], abs=1e-9)
    assert per[N] == pytest.approx(0.0, abs=1e-9)


@pytest.mark.parametrize("N", [1.0, 1.5, 2.0, 3.25, 7.0])
def test_async_formulas(N):
    """Sec. 4.2.3: a transfer of N steps costs (N-1) T_step when it overlaps one
    step (Async-O) and N T_step when it blocks (Async)."""
    n = 56_000
    link = _link_for(14 * n, N * T)
    r_o, _ = gockpt_simulate_window([0, n], n, 40.0, 60.0, 0.0, link, wait_policy=0, **PAPER)
    r_a, _ = gockpt_simulate_window([0, n], n, 40.0, 60.0, 0.0, link, wait_policy=2, **PAPER)
    assert r_o.stall_ms == pytest.approx(max(0.0, N - 1) * T, rel=1e-9, abs=1e-9)
    assert r_a.stall_ms == pytest.approx(N * T, rel=1e-9)


def test_printed_delta_is_async_o_minus_gockpt():
    """The printed (-N^2 + 15N - 14)/14 T_step equals T_Async-O - T_GoCkpt (the
    paper labels it the other way round); over whole N it peaks at 3 T_step,
    at N = 7 and N = 8."""
    deltas = {}
    for N in range(1, 15):
        n = 8 * N * 1000
        link = _link_for(14 * n / N, T)
        b = np.arange(N + 1) * (n // N)
        g, _ = gockpt_simulate_window(b, n, 40.0, 60.0, 0.0, link, wait_policy=1, **PAPER)
        a, _ = gockpt_simulate_window([0, n], n, 40.0, 60.0, 0.0, link, wait_policy=0, **PAPER)
        deltas[N] = a.stall_ms - g.stall_ms
        assert deltas[N] == pytest.approx((-N * N + 15 * N - 14) / 14 * T, rel=1e-9, abs=1e-9)
    top = max(deltas.values())
    assert top == pytest.approx(3.0 * T)
    assert sorted(N for N, d in deltas.items() if d == pytest.approx(top)) == [7, 8]


def test_per_step_delays_add_up():
    n = 1 << 20
    b = [0, 200_000, 500_000, 800_000, n]
    for pol in (0, 1, 2):
        for ring in (0, 1 << 20, 8 << 20):
            r, per = gockpt_simulate_window(b, n, 3.0, 5.0, 1.0, 2.0, wait_policy=pol, ring_bytes=ring,
                                            copy_bytes=1 << 18)
            assert per.sum() == pytest.approx(r.stall_ms, abs=1e-9)
            assert r.d2h_bytes == 12 * n + 2 * sum(b[:-1])


def test_ring_holding_the_window_hides_it():
    """A ring that holds the whole window: under the lazy rule nothing is waited
    for; the explicit gradient wait still costs the gradient transfers."""
    n = 1 << 20
    b = [0, 262_144, 524_288, 786_432, n]
    window = 12 * n + 2 * sum(b[:-1])
    ring = (window // 256 + 64) * 256
    lazy, _ = gockpt_simulate_window(b, n, 3.0, 5.0, 1.0, 1.0, ring_bytes=ring)
    assert lazy.stall_ms == pytest.approx(0.0, abs=1e-12) and lazy.spilled_bytes == 0
    grads, _ = gockpt_simulate_window(b, n, 3.0, 5.0, 1.0, 1.0, ring_bytes=ring, wait_policy=1)
    assert grads.stall_ms == pytest.approx(2 * sum(b[:-1]) / 1e6, rel=1e-9)  # 1 GB/s = 1e6 B/ms
    none, _ = gockpt_simulate_window(b, n, 3.0, 5.0, 1.0, 0.2)  # copies no longer fit behind a step
    assert none.spilled_bytes == window and none.stall_ms > 0


def test_planner_takes_the_hbm_snapshot_when_the_ring_holds_it():
    """With room for the whole state in the ring, one step that packs it all is
    free under the lazy rule and moves the fewest bytes: K = 1."""
    n = 1 << 22
    b, r = gockpt_plan_window(n, 10.0, 20.0, 1.0, 1.0, ring_bytes=(12 * n // 256 + 1) * 256)
    assert r.K == 1 and list(b) == [0, n]
    assert r.stall_ms == pytest.approx(0.0, abs=1e-9) and r.d2h_bytes == 12 * n


@pytest.mark.parametrize("seed", range(40))
def test_planner_matches_brute_force(seed):
    """Tiny spaces: the planner's stall equals the best over every K <= 4 and
    every choice of bounds (to its 1 us tie threshold)."""
    rng = np.random.default_rng(seed)
    n = 96
    kw = dict(align=8, copy_bytes=256, ring_bytes=int(rng.choice([0, 256, 512, 1024])),
              wait_policy=int(rng.integers(0, 3)), ring_plan=int(rng.integers(0, 3)),
              staging_bytes=int(rng.choice([0, 256, 1024])), host_gbs=float(rng.uniform(0.0, 2.0)) * 1.152e-3)
    tf, tb, tu = rng.uniform(0, 2, 3)
    link = float(rng.uniform(0.2, 3.0)) * 1.152e-3
    best = min(gockpt_simulate_window([0, *cut, n], n, tf, tb, tu, link, **kw)[0].stall_ms
               for K in range(1, 5) for cut in itertools.combinations(range(8, n, 8), K - 1))
    b, r = gockpt_plan_window(n, tf, tb, tu, link, max_K=4, **kw)
    assert 1 <= r.K <= 4 and len(b) == r.K + 1
    assert r.stall_ms <= best + 1e-3
    again, _ = gockpt_simulate_window(b, n, tf, tb, tu, link, **kw)
    assert again.stall_ms == r.stall_ms


def test_planner_beats_equal_parts_on_a_spilling_window():
    """Llama-7B-like: a 256 MiB ring, a link that cannot hide the window behind
    the forward pass.  The plan must not be worse than equal parts at any K up
    to the cap, and stays within the 7-step cap of Sec. 4.2.3."""
    n = 6_738_415_616
    args = (n, 110.4, 278.0, 30.3, 56.3)
    kw = dict(ring_bytes=256 << 20, copy_bytes=64 << 20)
    b, r = gockpt_plan_window(*args, **kw)
    assert 1 <= r.K <= 7 and b[0] == 0 and b[-1] == n and np.all(np.diff(b) > 0) and np.all(b[1:-1] % 256 == 0)
    for K in range(1, 8):
        eq = (np.arange(K + 1) * n // K) // 256 * 256
        eq[-1] = n
        assert r.stall_ms <= gockpt_simulate_window(eq, *args, **kw)[0].stall_ms + 1e-6
    eq16 = (np.arange(17) * n // 16) // 256 * 256
    eq16[-1] = n
    assert r.stall_ms < 0.5 * gockpt_simulate_window(eq16, *args, **kw)[0].stall_ms


def test_planner_tensor_bounds():
    ends = np.cumsum([1000, 24, 4096, 4096, 333, 8192, 8192, 16, 12_000, 5000])
    n = int(ends[-1])
    b, r = gockpt_plan_window(n, 1.0, 2.0, 0.1, 0.05, tensor_ends=ends, max_K=5)
    inner = set(int(x) for x in ends[:-1] if x % 8 == 0)
    assert b[0] == 0 and b[-1] == n and all(int(x) in inner for x in b[1:-1])
    assert np.all(np.diff(b) > 0)


def test_planner_respects_the_cap():
    n = 1 << 24
    for cap in (1, 2, 3, 9):
        b, r = gockpt_plan_window(n, 1.0, 1.0, 0.1, 1.0, max_K=cap)
        assert r.K <= cap and len(b) == r.K + 1


@pytest.mark.parametrize("bad", [dict(link_gbs=0.0), dict(t_fwd_ms=-1.0), dict(wait_policy=3), dict(ring_bytes=100),
                                 dict(max_K=300), dict(align=12), dict(copy_bytes=1000)])
def test_planner_rejects_bad_parameters(bad):
    args = dict(n=1 << 20, t_fwd_ms=1.0, t_bwd_ms=1.0, t_upd_ms=0.1, link_gbs=1.0)
    args.update(bad)
    n, tf, tb, tu, link = args.pop("n"), args.pop("t_fwd_ms"), args.pop("t_bwd_ms"), args.pop("t_upd_ms"), \
        args.pop("link_gbs")
    with pytest.raises(GockptError):
        gockpt_plan_window(n, tf, tb, tu, link, **args)


def test_simulate_rejects_bad_bounds():
    with pytest.raises(GockptError):
        gockpt_simulate_window([0, 12, 64], 64, 1.0, 1.0, 0.1, 1.0)  # interior bound not a multiple of 8
    with pytest.raises(GockptError):
        gockpt_simulate_window([0, 64, 32], 64, 1.0, 1.0, 0.1, 1.0)


def test_bad_ring_plan_or_staging_refused():
    """An unknown ring plan, staging smaller than one copy piece and a
    non-finite host rate are refused."""
    import ctypes

    from paper_2511_07035_amd import _plan_params, gockpt_plan_result, lib

    b = np.array([0, 4000, 8000], dtype=np.int64)
    out = gockpt_plan_result()
    per = np.zeros(3)
    for kw, rc in ((dict(), 0), (dict(ring_plan=2), 0), (dict(ring_plan=3), -1), (dict(ring_plan=-1), -1),
                   (dict(copy_bytes=1024, staging_bytes=512), -1), (dict(copy_bytes=1024, staging_bytes=2048), 0),
                   (dict(copy_bytes=1024, staging_bytes=2048, host_gbs=float("inf")), -1)):
        p, _ = _plan_params(8000, 40.0, 60.0, 0.0, 50.0, **kw)
        assert lib().gockpt_simulate_window(ctypes.byref(p), 2, b.ctypes.data, ctypes.byref(out),
                                            per.ctypes.data) == rc, kw


# ---- ring plans and staged windows -------------------------------------------

def test_device_wait_holds_the_update_for_the_ring_bytes_it_overwrites():
    """K = 2, parts of m elements, a ring of 14m bytes: step 1 packs its 12m
    state bytes at [0, 12m); step 2 packs 2m of gradients and 12m of state at
    [12m, 26m), overwriting [0, 12m), so under DEVICE_WAIT its update waits
    for step 1's copy: the stall is max(0, 12m / link - forward - backward),
    and nothing spills.  The late plans find only 2m free instead: step 2's
    state goes straight from the live buffers."""
    m = 1 << 20
    n, b = 2 * m, [0, m, 2 * m]
    link = 12 * m / 50e-3 / 1e9  # step 1's state takes 50 ms
    kw = dict(ring_bytes=14 * m, copy_bytes=1 << 20)
    dev, per = gockpt_simulate_window(b, n, 10.0, 20.0, 1.0, link, ring_plan=2, **kw)
    assert dev.stall_ms == pytest.approx(50.0 - 30.0, rel=1e-9)
    assert per[1] == pytest.approx(20.0, rel=1e-9) and per[0] == 0.0 and per[2] == 0.0
    assert dev.spilled_bytes == 0 and dev.d2h_bytes == 12 * n + 2 * m
    for plan in (0, 1):
        late, _ = gockpt_simulate_window(b, n, 10.0, 20.0, 1.0, link, ring_plan=plan, **kw)
        assert late.spilled_bytes == 12 * m
    # a fast link: step 1's copy is done before step 2's update starts
    fast, _ = gockpt_simulate_window(b, n, 10.0, 20.0, 1.0, link * 2, ring_plan=2, **kw)
    assert fast.stall_ms == pytest.approx(0.0, abs=1e-12)


def test_device_wait_with_a_ring_holding_the_window_waits_for_nothing():
    n = 1 << 20
    b = [0, 262_144, 524_288, 786_432, n]
    ring = ((12 * n + 2 * sum(b[:-1])) // 256 + 64) * 256
    r, per = gockpt_simulate_window(b, n, 3.0, 5.0, 1.0, 0.01, ring_bytes=ring, ring_plan=2)
    assert r.stall_ms == pytest.approx(0.0, abs=1e-12) and r.spilled_bytes == 0


@pytest.mark.parametrize("seed", range(12))
def test_staging_with_room_and_an_instant_host_is_the_pinned_window(seed):
    """Enough slots for every copy and host copies that take no time: the
    staged model is the pinned one."""
    rng = np.random.default_rng(seed)
    n = 1 << 16
    b = [0, *sorted(int(x) * 8 for x in rng.choice(n // 8 - 1, 3, replace=False) + 1), n]
    kw = dict(ring_bytes=int(rng.choice([0, 1 << 16, 1 << 18])), copy_bytes=4096, ring_plan=int(rng.integers(0, 3)),
              wait_policy=int(rng.integers(0, 3)))
    args = (b, n, *rng.uniform(0.1, 2.0, 3), float(rng.uniform(0.0005, 0.01)))
    pinned, pp = gockpt_simulate_window(*args, **kw)
    staged, ps = gockpt_simulate_window(*args, staging_bytes=1 << 30, **kw)
    assert staged.stall_ms == pytest.approx(pinned.stall_ms, abs=1e-9)
    assert staged.latency_ms == pytest.approx(pinned.latency_ms, abs=1e-9)
    assert np.allclose(pp, ps, atol=1e-9)


def test_staged_async_closed_forms():
    """K = 1, no ring: the 12n bytes of state go after the update in m pieces
    of c bytes.  With a slot per piece and a host slower than the link, the
    host finishes c/link + 12n/host after the update; with one slot every
    piece waits for the previous one to be emptied: 12n/link + 12n/host, and
    the step after the window waits for the last piece to land,
    12n/link + (m - 1) c/host after the update."""
    n = 1 << 20
    c = 1 << 20
    B = 12 * n
    m = B // c
    tf, tb, tu = 5.0, 7.0, 1.0
    link, host = 1.0, 0.25  # GB/s: 1e6 and 2.5e5 bytes per ms
    L, H = link * 1e6, host * 1e6
    wide, _ = gockpt_simulate_window([0, n], n, tf, tb, tu, link, copy_bytes=c, staging_bytes=(m + 1) * c,
                                     host_gbs=host)
    assert wide.latency_ms == pytest.approx(tf + tb + tu + c / L + B / H, rel=1e-12)
    one, per = gockpt_simulate_window([0, n], n, tf, tb, tu, link, copy_bytes=c, staging_bytes=c, host_gbs=host)
    assert one.latency_ms == pytest.approx(tf + tb + tu + B / L + B / H, rel=1e-12)
    land = B / L + (m - 1) * c / H
    assert one.stall_ms == pytest.approx(max(0.0, land - tf - tb), rel=1e-12)
    assert per[1] == pytest.approx(one.stall_ms, rel=1e-12)
    pinned, _ = gockpt_simulate_window([0, n], n, tf, tb, tu, link, copy_bytes=c)
    assert pinned.stall_ms == pytest.approx(max(0.0, B / L - tf - tb), rel=1e-12)
