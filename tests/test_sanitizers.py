"""The library's host code (cache, read accounting, storage tier) under
AddressSanitizer and ThreadSanitizer.

Each driver in tests/sanitize/ is linked with every library source, the
sanitizer applied to host code only (``-Xarch_host -fsanitize=...``), and run
on the CPU.  Building takes about a minute per sanitizer, so these run only
when CKV_SANITIZE=1.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2601_13631_amd", "csrc")
SRC = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))

pytestmark = pytest.mark.skipif(os.environ.get("CKV_SANITIZE") != "1",
                                reason="sanitizer builds run with CKV_SANITIZE=1")


@pytest.mark.parametrize("sanitizer", ["address", "thread"])
@pytest.mark.parametrize("driver", ["cache_io_drive.cpp", "store_drive.cpp"])
def test_host_code_under_sanitizer(tmp_path, sanitizer, driver):
    exe = str(tmp_path / "drive")
    cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xarch_host", f"-fsanitize={sanitizer}",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "sanitize", driver),
           *SRC, "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe], cwd=str(tmp_path), capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "drive ok" in r.stdout
    assert "WARNING: ThreadSanitizer" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
