"""Build the C program that drives libcdt through include/cdt.h alone (host
code, gcc, linked against the built libcdt.so and the HIP runtime)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "detect.c")
EXE = os.path.join(HERE, "detect")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(verbose=False):
    lib_dir = os.path.join(ROOT, "paper_2607_19490_amd")
    tmp = EXE + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC,
           "-o", tmp, "-L", lib_dir, "-l:libcdt.so", "-L", os.path.join(ROCM, "lib"),
           "-lamdhip64", "-Wl,-rpath,$ORIGIN/../../paper_2607_19490_amd",
           "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
