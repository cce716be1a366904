"""Compile the plain C11 consumer of the library (test infrastructure) next to
this file: gcc -std=c11 -pedantic with warnings as errors against
include/relaxkv.h, linked to the in-tree librelaxkv.so and the HIP runtime."""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2609_33503_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SRC = os.path.join(HERE, "relaxkv_c_consumer.c")
OUT = os.path.join(HERE, "relaxkv_c_consumer")


def command(out=OUT):
    return ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-pedantic",
            "-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include"),
            "-I", os.path.join(ROOT, "include"), SRC, "-o", out,
            "-L", PKG, "-lrelaxkv", "-Wl,-rpath," + PKG,
            "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")]


def build(out=OUT):
    r = subprocess.run(command(out), capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("C consumer build failed:\n" + r.stderr)
    return out


if __name__ == "__main__":
    print("built", build())
    sys.exit(0)
