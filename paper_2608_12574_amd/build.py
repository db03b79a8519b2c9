"""Build ``libtam.so`` (host C++ + HIP kernels for gfx950) in-tree with hipcc.

    python -m paper_2608_12574_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libtam.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", "-pthread", "-Wall", "-Wno-unused-result", f"-I{ROOT}/include"]
# The packed-FP32 VALU forms are switched off for every GPU compile.
GPU = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".cpp", ".hip")))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *COMMON, *GPU, "-c", src, "-o", obj]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    objs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        futs = {ex.submit(_compile, s): s for s in srcs}
        for f in cf.as_completed(futs):
            try:
                objs.append(f.result())
            except subprocess.CalledProcessError as e:
                sys.stderr.write(e.stdout + e.stderr)
                raise RuntimeError(f"hipcc failed on {futs[f]}") from e
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *GPU, "-shared", "-fPIC", "-pthread", "-o", tmp, *sorted(objs)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc link failed")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
