"""Build libdsv.so (the HIP library behind include/dsv.h) for gfx950, in-tree.

    python -m paper_2607_28848_amd.build              # the library
    python -m paper_2607_28848_amd.build --host-asan  # + host-sanitized variant

The host-sanitized variant compiles the host code (plan.cpp, api.cpp: segment
table validation, plan packing, argument checks) with g++ and
AddressSanitizer + UndefinedBehaviorSanitizer, and the device code exactly as
the library does.  It lands in _build/host_asan/libdsv.so; the binding loads it
when DSV_LIBRARY names it, in a process started with gcc's libasan loaded
first.  It is for CPU-only runs of the host-side tests.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libdsv.so")
SOURCES = ["plan.cpp", "api.cpp", "gemm_bf16.hip", "kernels_bf16.hip", "kernels_f32.hip", "optim.hip", "dropout.hip", "scratch.hip"]
HOST_SOURCES = [s for s in SOURCES if s.endswith(".cpp")]
ASAN_DIR = os.path.join(PKG, "_build", "host_asan")
ASAN_LIB = os.path.join(ASAN_DIR, "libdsv.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HOST_SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                 "-fno-omit-frame-pointer"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    # no packed fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def build(verbose: bool = False) -> str:
    """Compile every source into libdsv.so (always recompiles)."""
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, cwd=PKG, capture_output=True, text=True)
    out = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + out)
    if verbose and out.strip():
        print(out, flush=True)
    os.replace(tmp, LIB)
    return LIB


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, cwd=PKG, capture_output=True, text=True)
    out = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("%s failed:\n%s" % (cmd[0], out))
    return out


def build_host_asan(verbose: bool = False) -> str:
    """Build _build/host_asan/libdsv.so: host code under g++ with ASan + UBSan,
    device sources compiled by hipcc as in build() (no sanitizer reaches them)."""
    os.makedirs(ASAN_DIR, exist_ok=True)
    dev_flags = [f for f in FLAGS if f != "-shared"]
    jobs = []
    for src in SOURCES:
        obj = os.path.join(ASAN_DIR, src + ".o")
        path = os.path.join(CSRC, src)
        if src in HOST_SOURCES:
            cmd = (["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-Wall", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include")]
                   + HOST_SANITIZE + ["-c", path, "-o", obj])
        else:
            cmd = [HIPCC] + dev_flags + ["-c", path, "-o", obj]
        jobs.append((cmd, obj))
    with ThreadPoolExecutor(max_workers=min(len(jobs), 8)) as ex:
        list(ex.map(lambda j: _run(j[0], verbose), jobs))
    tmp = ASAN_LIB + ".tmp%d" % os.getpid()
    _run(["g++", "-shared"] + HOST_SANITIZE + ["-o", tmp] + [o for _, o in jobs]
         + ["-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")],
         verbose)
    os.replace(tmp, ASAN_LIB)
    return ASAN_LIB


if __name__ == "__main__":
    build(verbose=True)
    print("built", LIB)
    if "--host-asan" in sys.argv[1:]:
        build_host_asan(verbose=True)
        print("built", ASAN_LIB)
    sys.exit(0)
