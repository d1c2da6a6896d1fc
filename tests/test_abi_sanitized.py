"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer: a build of
libtt with the sanitizers on the host side only (the gfx950 device code is built as usual and
never runs here), driven by tests/abi_sanitize_driver.c through the calls that need no GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None, reason="hipcc not available")
def test_host_library_is_clean_under_sanitizers(tmp_path):
    import glob

    hipcc = HIPCC if os.path.exists(HIPCC) else shutil.which("hipcc")
    csrc = os.path.join(ROOT, "paper_2510_15545_amd", "csrc")
    lib = str(tmp_path / "libtt_san.so")
    host_san = ["-Xarch_host", "-fsanitize=address",
                "-Xarch_host", "-fsanitize=undefined"]
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
                    "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san,
                    "-I", os.path.join(ROOT, "include"), "-I", csrc, *sorted(glob.glob(os.path.join(csrc, "*.hip"))),
                    "-o", lib], check=True, capture_output=True, text=True)
    exe = str(tmp_path / "abi_driver")
    subprocess.run([hipcc, "-x", "c", "-O1", "-g", *host_san, "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "abi_sanitize_driver.c"), "-o", exe, "-L", str(tmp_path),
                    "-ltt_san", "-Wl,-rpath," + str(tmp_path)], check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out
    assert "runtime error" not in out and "AddressSanitizer" not in out, out
    assert "done" in run.stdout, out
