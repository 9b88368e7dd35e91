"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

The oracle (oracle/svm_oracle.c) is compiled together with a driver that calls every entry
point -- training with the full Gram and with the least-recently-used row cache, the working-set
rounds at q = 2, 8 and q > n, the selection, kernel rows, f from alpha and decision values --
and the host-side checkers of the kernels' index and bit arithmetic are compiled with the
sanitizers on their host code.  Any out-of-bounds access, leak or undefined operation aborts the
program and fails the test.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2311_14908_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1",
           OMP_NUM_THREADS="2")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_san"
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", *SAN, os.path.join(ROOT, "oracle", "svm_oracle.c"),
                    os.path.join(HERE, "oracle_sanitize_driver.c"), "-o", str(exe), "-lm"], check=True,
                   capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok"
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
@pytest.mark.parametrize("src", ["tile_order_check.cpp", "xchg_record_check.cpp", "ws_record_check.cpp"])
def test_host_checkers_under_sanitizers(src, tmp_path):
    exe = tmp_path / os.path.splitext(src)[0]
    host_san = [f for flag in SAN for f in ("-Xarch_host", flag)]
    subprocess.run([HIPCC, "-O1", "-g", "-x", "hip", "--offload-arch=gfx950", *host_san, "-I", CSRC,
                    os.path.join(HERE, src), "-o", str(exe)], check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok")
