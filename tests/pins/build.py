"""Build the test-only library pins (host code, g++): rocRAND's Philox."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
PHILOX_SRC = os.path.join(HERE, "rocrand_philox_pin.cpp")
PHILOX_LIB = os.path.join(HERE, "libpin_philox.so")
ROCM_INCLUDE = os.environ.get("ROCM_PATH", "/opt/rocm") + "/include"


def build(verbose=False):
    tmp = PHILOX_LIB + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
           "-I" + ROCM_INCLUDE, PHILOX_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, PHILOX_LIB)
    return PHILOX_LIB


if __name__ == "__main__":
    print(build(verbose=True))
