"""The library's host-only C++ (window planner, bounds and arena layout,
checkpoint writer/reader, multithreaded replay) built with g++ under
AddressSanitizer + UndefinedBehaviorSanitizer and under ThreadSanitizer and
driven by tests/host/sanitize_driver.cpp.  CPU only; no HIP runtime."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2511_07035_amd", "csrc")
SOURCES = [os.path.join(ROOT, "tests", "host", "sanitize_driver.cpp")] + [
    os.path.join(CSRC, f) for f in ("gockpt_plan.cpp", "gockpt_planner.cpp", "gockpt_restore.cpp",
                                    "gockpt_persist.cpp")]


@pytest.mark.parametrize("sanitizer", ["address,undefined", "thread"])
def test_host_code_under_sanitizers(tmp_path, sanitizer):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no g++")
    exe = str(tmp_path / "driver")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", f"-fsanitize={sanitizer}",
           "-fno-sanitize-recover=all", "-ffp-contract=off", "-mavx2", "-msse4.2", f"-I{ROOT}/include", f"-I{CSRC}",
           *SOURCES, "-o", exe, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, str(tmp_path / "ck")], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "ok" in r.stdout, (r.stdout + r.stderr)[-4000:]
    assert "Sanitizer" not in r.stderr, r.stderr[-4000:]
