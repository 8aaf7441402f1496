"""The C ABI used from plain C: tests/c/window_c.c includes only gockpt.h and
the HIP runtime API (no Python, no torch).  On the CPU it must compile as
C11 against the header; on the GPU it runs a window whose restored checkpoint
must equal the oracle's synchronous state, bit for bit."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2511_07035_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build(out_dir) -> str:
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = os.path.join(str(out_dir), "window_c")
    cmd = [cc, "-std=c11", "-O2", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
           f"-I{ROOT}/include", os.path.join(ROOT, "tests", "c", "window_c.c"), "-o", exe, f"-L{PKG}", "-lgockpt",
           f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{PKG}", f"-Wl,-rpath,{ROCM}/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def test_c_consumer_compiles_against_the_header(tmp_path):
    _build(tmp_path)


@pytest.mark.gpu
def test_c_consumer_window_matches_oracle(tmp_path):
    exe = _build(tmp_path)
    n, K, seed = 100_003, 3, 60
    bounds = np.array([0, 8, 40_000, n], dtype=np.int64)
    p0 = synth.master_cpu(n, seed)
    grads = np.stack([synth.grads_cpu(n, seed, s) for s in range(1, K + 1)])
    inp, out = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    with open(inp, "wb") as f:
        f.write(np.array([n, K], np.int64).tobytes())
        f.write(bounds.tobytes())
        f.write(p0.tobytes())
        f.write(grads.astype(np.uint16).tobytes())
    print(f"[case] C consumer n={n} K={K}", flush=True)
    r = subprocess.run([exe, inp, out], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    raw = open(out, "rb").read()
    off = 0

    def take(dtype, count):
        nonlocal off
        a = np.frombuffer(raw, dtype=dtype, count=count, offset=off)
        off += a.nbytes
        return a

    p, m, v = take(np.float32, n), take(np.float32, n), take(np.float32, n)
    w, p_dev = take(np.uint16, n), take(np.float32, n)
    t = int(take(np.int64, 1)[0])
    ref = oracle.State(p0)
    oracle.sync_run(ref, grads, oracle.AdamWConfig())
    for got, want in ((p, ref.p), (m, ref.m), (v, ref.v), (p_dev, ref.p)):
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    assert np.array_equal(w, ref.w) and t == ref.t == K


@pytest.mark.parametrize("lang", ["c99", "c++11"])
def test_header_alone_is_strict_c_and_cpp(tmp_path, lang):
    """gockpt.h on its own (no HIP headers) under -pedantic -Werror, as C99
    and as C++11."""
    cc = shutil.which("g++" if lang.startswith("c++") else "gcc")
    if cc is None:
        pytest.skip("no compiler")
    src = tmp_path / "h.c"
    src.write_text('#include "gockpt.h"\nint main(void) { return (int)sizeof(gockpt_config) == 0; }\n')
    cmd = [cc, f"-std={lang}", "-Wall", "-Wextra", "-pedantic", "-Werror", f"-I{ROOT}/include"]
    if lang.startswith("c++"):
        cmd += ["-x", "c++"]
    r = subprocess.run(cmd + ["-c", str(src), "-o", str(tmp_path / "h.o")], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
