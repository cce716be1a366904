"""Build the HIP library ``librelaxkv.so`` in-tree for gfx950.

Every source under ``csrc/`` is compiled by hipcc (one process per file, in
parallel) and linked into ``paper_2609_33503_amd/librelaxkv.so``.  All device
code is compiled with packed-fp32 instructions disabled.
Run as ``python -m paper_2609_33503_amd.build``.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "librelaxkv.so")
BUILD_DIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument", f"-I{INCLUDE}", f"-I{CSRC}"]


def _hipcc():
    h = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(h):
        raise RuntimeError("hipcc not found")
    return h


# The attention and scoring kernels never see NaN (masked logits are -inf):
# without NaN semantics fmaxf needs no operand canonicalisation.  The sparse
# attention is scheduled with the backend's max-ILP strategy (about 2% faster on
# the 32K workload than the default; the same instructions, reordered).
PER_FILE = {"attn.hip": ["-fno-honor-nans", "-mllvm", "-amdgpu-sched-strategy=max-ilp"],
            "score.hip": ["-fno-honor-nans"],
            "query_attn.hip": ["-fno-honor-nans"]}


def _compile(src):
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    extra = PER_FILE.get(os.path.basename(src), [])
    cmd = [_hipcc(), *COMMON, *extra, "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature; that is harmless.
    err = "\n".join(x for x in r.stderr.splitlines() if "packed-fp32-ops" not in x)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    return obj


def build(verbose=False):
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                  if f.endswith((".hip", ".cpp")))
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = OUT + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
