"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

- The oracle (plain C) is built with gcc's sanitizers and every routine runs
  on small, ragged, empty and S = 64 shapes, with special fp16 inputs.
- The C ABI's argument checks (host side of libcdt) are built with the
  sanitizers on the host pass only (hipcc -Xarch_host) and fed bad and
  edge-case arguments; none of these calls reaches the GPU.
Either run aborts with the sanitizer's report on an out-of-bounds access,
use after free, integer overflow or other undefined behaviour.
"""
import glob
import os
import subprocess

import pytest

from tests.conftest import ROOT

HERE = os.path.join(ROOT, "tests", "sanitize")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "drive_oracle")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(HERE, "drive_oracle.c"),
                    "-o", exe, "-lm"], check=True, capture_output=True)
    r = subprocess.run([exe], env=SAN_ENV, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr, r.stderr[-4000:]


def test_abi_checks_under_sanitizers(tmp_path):
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "drive_abi")
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2607_19490_amd", "csrc", "*.hip")))
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-ffp-contract=off",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), *srcs, os.path.join(HERE, "drive_abi.hip"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, timeout=900)
    r = subprocess.run([exe], env=SAN_ENV, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr, r.stderr[-4000:]
