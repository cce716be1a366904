"""Build the library's host side with AddressSanitizer and UndefinedBehavior-
Sanitizer (device code is compiled as usual) and the host-stress driver
against it, into a directory of the caller's (test infrastructure)."""

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2609_33503_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
# Host-only sanitizer flags: each -fsanitize= directly after -Xarch_host.
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        err = "\n".join(x for x in r.stderr.splitlines() if "packed-fp32-ops" not in x)
        raise RuntimeError(f"{' '.join(cmd[:3])} ... failed:\n{err}")


def _asan_rt_dir():
    r = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True)
    return os.path.dirname(r.stdout.strip())


def build(out_dir):
    rt = _asan_rt_dir()
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))

    def obj(src):
        o = os.path.join(out_dir, os.path.basename(src) + ".o")
        _run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-Wno-unused-command-line-argument", *HOST_SAN,
              f"-I{INCLUDE}", f"-I{CSRC}", "-x", "hip", "-c", src, "-o", o])
        return o

    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(obj, srcs))
    lib = os.path.join(out_dir, "librelaxkv.so")
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libasan", *HOST_SAN,
          "-Wl,-rpath," + rt, "-o", lib, *objs])
    exe = os.path.join(out_dir, "host_stress")
    _run([CLANG, "-std=c11", "-O1", "-g", "-Wall", "-Wextra", "-Werror", "-pedantic",
          "-shared-libasan", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include"),
          f"-I{INCLUDE}", os.path.join(HERE, "host_stress.c"), "-o", exe,
          "-L", out_dir, "-lrelaxkv", "-Wl,-rpath," + out_dir, "-Wl,-rpath," + rt,
          "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"),
          "-lm"])
    return exe
