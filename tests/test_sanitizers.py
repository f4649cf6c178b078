"""CPU: the host code under AddressSanitizer and UndefinedBehaviorSanitizer.

- The fp64 oracle (oracle.c, ln_linear.c), built with gcc -fsanitize and run
  on tiny seeded problems of both nodes, masks, row and query subsets
  (tests/san/oracle_driver.c).
- The C ABI's host paths (argument checks, workspace sizing and layout),
  built with hipcc with the sanitizers on the host side only (device code is
  built as usual and never launched) and run without a GPU: every
  workspace-size call over a sweep of shapes up to the largest accepted, and
  the argument errors of every entry point (tests/san/abi_driver.cpp).

A sanitizer report makes the run fail (-fno-sanitize-recover).
"""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "san")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=600)
    text = r.stdout + r.stderr
    assert r.returncode == 0, text[-4000:]
    assert "runtime error" not in text and "AddressSanitizer" not in text, text[-4000:]
    return text


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    srcs = [os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "oracle", "ln_linear.c"),
            os.path.join(SAN, "oracle_driver.c")]
    subprocess.run(["gcc", "-O1", "-g", "-fopenmp", "-std=c11", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", *srcs, "-o", exe,
                    "-lm"], check=True)
    assert "0 non-finite" in _run(exe)


HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_abi_host_paths_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_san")
    csrc = os.path.join(ROOT, "paper_2506_20686_amd", "csrc")
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
                "-fno-omit-frame-pointer"]
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san,
           "-I", os.path.join(ROOT, "include"), "-I", csrc,
           *sorted(glob.glob(os.path.join(csrc, "*.hip"))), os.path.join(SAN, "abi_driver.cpp"),
           "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "0 failures" in _run(exe)
