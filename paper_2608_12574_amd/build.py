"""Build ``libtam.so`` (host C++ + HIP kernels for gfx950) in-tree with hipcc.

    python -m paper_2608_12574_amd.build               # the library
    python -m paper_2608_12574_amd.build --sanitize    # a host-sanitized copy

The sanitized copy (``_build/sanitize/libtam.so``) instruments the host code
only (trie and vocabulary builds, the worker pool, the C ABI) with
AddressSanitizer and UndefinedBehaviorSanitizer; the GPU code is built as
usual.  It is for CPU runs of the host tests.  Python itself is not
instrumented, so the sanitizer runtime is preloaded into that one process:

    RT=$(/opt/rocm/bin/hipcc -print-file-name=libclang_rt.asan-x86_64.so)
    LD_PRELOAD="$RT${LD_PRELOAD:+:$LD_PRELOAD}" ASAN_OPTIONS=detect_leaks=0 \
    TAM_LIBRARY=_build/sanitize/libtam.so python -m pytest -m "not gpu" \
        tests/test_abi_host.py tests/test_layout_host.py
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


# Host-side sanitizers: every -fsanitize= applies to the host pass only.
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
SANITIZE_DIR = os.path.join(BUILD, "sanitize")


def _compile(src: str, out_dir: str, extra: list) -> str:
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *COMMON, *extra, *GPU, "-c", src, "-o", obj]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    out_dir = SANITIZE_DIR if sanitize else BUILD
    lib = os.path.join(SANITIZE_DIR, "libtam.so") if sanitize else LIB
    extra = ["-O1", *SANITIZE] if sanitize else []
    os.makedirs(out_dir, exist_ok=True)
    srcs = sources()
    objs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        futs = {ex.submit(_compile, s, out_dir, extra): s for s in srcs}
        for f in cf.as_completed(futs):
            try:
                objs.append(f.result())
            except subprocess.CalledProcessError as e:
                sys.stderr.write(e.stdout + e.stderr)
                raise RuntimeError(f"hipcc failed on {futs[f]}") from e
    tmp = lib + ".tmp"
    link_extra = []
    if sanitize:  # the shared sanitizer runtime, found through the library's rpath
        rt = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                            text=True).stdout.strip().splitlines()[-1]
        link_extra = ["-shared-libsan", *SANITIZE, f"-Wl,-rpath,{os.path.dirname(rt)}"]
    cmd = [HIPCC, *GPU, *link_extra, "-shared", "-fPIC", "-pthread", "-o", tmp, *sorted(objs)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc link failed")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv[1:])
