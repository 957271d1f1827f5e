"""Build the test-side device checks (HIP programs compiled with the
library's own flags and headers; run by the GPU tests)."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "t3_arith.hip")
EXE = os.path.join(HERE, "t3_arith")


def build(verbose=False):
    sys.path.insert(0, ROOT)
    from paper_2607_19490_amd import build as lib_build
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    flags = [f for f in lib_build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    tmp = EXE + ".tmp"
    cmd = [hipcc, *flags, "-I", os.path.join(ROOT, "include"), "-I", lib_build.CSRC, SRC,
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
