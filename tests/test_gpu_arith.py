"""The device's fp32 division and square root, built with the library's
flags, against the host's IEEE operations (numpy float32, i.e. SSE divss and
sqrtss, correctly rounded, subnormals kept), bit for bit: 2^24 random pairs
over the whole exponent range plus edge values.  With these two and the
contract's fixed operation order, every bit of the update is fixed."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _edges():
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, -1.0, 2.0, 0.5, 3.0,
                         np.finfo(np.float32).max, -np.finfo(np.float32).max,
                         np.finfo(np.float32).tiny, np.float32(1e-45), np.float32(-1e-45),
                         np.float32(1e-40), np.float32(1.17e-38), np.float32(3.4e38), np.float32(1e-30)],
                        dtype=np.float32)
    a, b = np.meshgrid(specials, specials)
    return a.ravel(), b.ravel()


def test_device_div_sqrt_match_host_ieee():
    import torch

    import bench as bench_mod

    B = bench_mod.bench_lib()
    rng = np.random.default_rng(31)
    n = 1 << 24
    bits = rng.integers(0, 1 << 32, size=(2, n), dtype=np.uint64).astype(np.uint32)
    a = bits[0].view(np.float32)
    b = bits[1].view(np.float32)
    ea, eb = _edges()
    # subnormal quotients and near-overflow quotients
    c = rng.uniform(1, 2, 4096).astype(np.float32)
    ea = np.concatenate([ea, c * np.float32(1e-38), c * np.float32(1.5e38)]).astype(np.float32)
    eb = np.concatenate([eb, c * np.float32(1e2), c * np.float32(0.5)]).astype(np.float32)
    a = np.concatenate([a, ea])
    b = np.concatenate([b, eb])
    m = a.size
    with np.errstate(all="ignore"):
        q_ref = a / b
        r_ref = np.sqrt(a)
    print(f"[case] div/sqrt m={m}", flush=True)
    da = torch.from_numpy(a).cuda()
    db = torch.from_numpy(b).cuda()
    dq = torch.empty_like(da)
    dr = torch.empty_like(da)
    s = torch.cuda.current_stream()
    assert B.gockpt_bench_divsqrt(da.data_ptr(), db.data_ptr(), dq.data_ptr(), dr.data_ptr(), m, s.cuda_stream) == 0
    torch.cuda.synchronize()
    q = dq.cpu().numpy()
    r = dr.cpu().numpy()
    for got, want, what in ((q, q_ref, "a/b"), (r, r_ref, "sqrt(a)")):
        nan = np.isnan(want)
        assert np.array_equal(np.isnan(got), nan), what
        bad = np.flatnonzero(got[~nan].view(np.uint32) != want[~nan].view(np.uint32))
        assert bad.size == 0, f"{what}: {bad.size} of {m} differ"


def test_device_bf16_rounding_all_fp32_patterns():
    """The contract's fp32 -> bf16 rounding as compiled for the device (the
    function the update kernel inlines for the bf16 weights), over all 2^32
    fp32 bit patterns: every non-NaN pattern against torch's CPU conversion
    (round to nearest even) bit for bit; every NaN to the contract's 0x7FC0
    (torch's vectorised conversion gives other NaN patterns)."""
    import torch

    import bench as bench_mod

    B = bench_mod.bench_lib()
    chunk = 1 << 28
    out = torch.empty(chunk, dtype=torch.int16, device="cuda")
    s = torch.cuda.current_stream()
    for base in range(0, 1 << 32, chunk):
        print(f"[case] bf16 rounding of patterns {base:#x}..{base + chunk - 1:#x}", flush=True)
        assert B.gockpt_bench_convert(0, base, chunk, out.data_ptr(), s.cuda_stream) == 0
        got = out.cpu().numpy().view(np.uint16)
        pats = np.arange(chunk, dtype=np.uint32) + np.uint32(base)
        want = torch.from_numpy(pats.view(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        nan = (pats & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
        assert np.all(got[nan] == 0x7FC0), "NaN patterns must give 0x7FC0"
        assert np.all((want[nan] & 0x7F80) == 0x7F80) and np.all(want[nan] & 0x7F), "torch: NaN in, NaN out"
        bad = np.flatnonzero((got != want) & ~nan)
        assert bad.size == 0, (f"{bad.size} patterns differ; first {int(pats[bad[0]]):#010x}: "
                               f"device {int(got[bad[0]]):#06x}, torch {int(want[bad[0]]):#06x}")


def test_device_widening_all_16bit_patterns():
    """bf16 -> fp32 and fp16 -> fp32 as compiled for the device, over all
    65536 patterns each, against torch's and numpy's CPU conversions.  bf16
    widening moves the bits up, NaN payloads included, so every pattern must
    match; fp16 NaNs become quiet NaNs with the sign kept (the contract), the
    rest must match bit for bit."""
    import torch

    import bench as bench_mod

    B = bench_mod.bench_lib()
    out = torch.empty(1 << 16, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream()
    pats = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    refs = {1: torch.from_numpy(pats.view(np.int16)).view(torch.bfloat16).float().numpy(),
            2: pats.view(np.float16).astype(np.float32)}
    for mode, want in refs.items():
        assert B.gockpt_bench_convert(mode, 0, 1 << 16, out.data_ptr(), s.cuda_stream) == 0
        got = out.cpu().numpy().view(np.float32)
        nan = np.isnan(want)
        assert np.array_equal(np.isnan(got), nan), f"mode {mode}: NaN positions"
        assert np.array_equal(got[~nan].view(np.uint32), want[~nan].view(np.uint32)), f"mode {mode}"
        gb, wb = got[nan].view(np.uint32), want[nan].view(np.uint32)
        if mode == 1:
            assert np.array_equal(gb, wb), "bf16 NaN patterns widen bit for bit"
        else:
            assert np.array_equal(gb >> 31, wb >> 31) and np.all(gb & 0x00400000), "fp16 NaN: sign kept, quiet"
