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
