"""Host-only check of the clustering code (Alg. 1) under AddressSanitizer and
UndefinedBehaviorSanitizer: the library's clustering source is compiled for
the host alone (no device code) with the randomised driver in
tests/host/assign_fuzz.cpp, which runs every rule on random client
populations and the invalid-argument paths."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SAN = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=undefined"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_assign_under_host_sanitizers(tmp_path):
    src = os.path.join(ROOT, "paper_2609_29395_amd", "csrc", "assign.cpp")
    drv = os.path.join(ROOT, "tests", "host", "assign_fuzz.cpp")
    exe = str(tmp_path / "assign_fuzz")
    flags = ["-std=c++17", "-O1", "-g"] + SAN.split()
    steps = [
        [HIPCC, *flags, "-x", "hip", "--cuda-host-only", "--offload-arch=gfx950", "-c", src,
         "-o", str(tmp_path / "assign.o")],
        [HIPCC, *flags, "-c", drv, "-o", str(tmp_path / "drv.o")],
        [HIPCC, *SAN.split(), str(tmp_path / "drv.o"), str(tmp_path / "assign.o"), "-o", exe],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
        assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe, "160", "96", "11"], capture_output=True, text=True, timeout=600, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and "runtime error" not in out and "ERROR: AddressSanitizer" not in out, out[-3000:]
    assert "bad 0" in r.stdout
