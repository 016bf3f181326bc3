"""Builds the HIP train-step library (libbmlp.so) for gfx950, in place.

Every source under csrc/ is compiled by hipcc into one shared library next to
this file.  The C ABI is declared in include/bmlp.h at the repository root.
"""
from __future__ import annotations

import glob
import hashlib
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libbmlp.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
ARCH = "gfx950"

COMMON_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
                "-Wall", "-Wno-unused-function"]
# Device pass only: keep packed-fp32 instructions out of device code.  The
# host pass would not know the feature, so each source is compiled twice,
# device code first, then the host code with that device code embedded, under
# one compilation-unit id so that both passes name static device variables
# alike.
# MFMA accumulators in ordinary VGPRs instead of AGPRs: the epilogues read
# every accumulator with VALU instructions (ballots, keys, argmax), which
# otherwise copy each one out of the AGPRs first (v_accvgpr_read).  Wave
# priority raised until a wave's first memory loads are issued (s_setprio),
# so that the update kernel's six waves per SIMD start their loads early.
DEVICE_FLAGS = ["--offload-device-only", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-kernarg-preload-count=16", "-mllvm", "-amdgpu-mfma-vgpr-form",
                "-mllvm", "-amdgpu-set-wave-priority"]
HOST_FLAGS = ["--offload-host-only"]


def kernel_fingerprint(src: str) -> str:
    """SHA-256 of a kernel source and of the flags its device code is
    compiled with: a counter profile taken from another build of the kernel no
    longer describes it."""
    h = hashlib.sha256()
    with open(src, "rb") as f:
        h.update(f.read())
    h.update(b"\0" + " ".join(COMMON_FLAGS + DEVICE_FLAGS).encode())
    return h.hexdigest()


def hipcc() -> str:
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return exe


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def host_sources():
    """Plain C++ sources (the host planning code): compiled for the host only."""
    return sorted(glob.glob(os.path.join(CSRC, "*.cpp")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd)}")
    if res.stderr.strip():
        sys.stderr.write(res.stderr)


def _compile(src: str, objdir: str, verbose: bool) -> str:
    name = os.path.splitext(os.path.basename(src))[0]
    if src.endswith(".cpp"):
        obj = os.path.join(objdir, name + ".o")
        _run([hipcc(), "-x", "c++", "-O3", "-std=c++17", "-fPIC", "-Wall", f"-I{INCLUDE}", f"-I{CSRC}",
              "-c", src, "-o", obj], verbose)
        return obj
    inc = [f"-I{INCLUDE}", f"-I{CSRC}", f"-cuid=bmlp_{name}"]
    dev = os.path.join(objdir, name + ".dev")
    obj = os.path.join(objdir, name + ".o")
    _run([hipcc(), *COMMON_FLAGS, *DEVICE_FLAGS, *inc, "-c", src, "-o", dev], verbose)
    _run([hipcc(), *COMMON_FLAGS, *HOST_FLAGS, *inc, "-Xclang", "-fcuda-include-gpubinary", "-Xclang", dev,
          "-c", src, "-o", obj], verbose)
    return obj


def build(verbose: bool = False) -> str:
    """Compile libbmlp.so; returns its path.  Raises on a compile error."""
    import concurrent.futures
    import tempfile
    with tempfile.TemporaryDirectory(prefix="bmlp_build_") as objdir:
        srcs = sources() + host_sources()
        workers = max(1, min(len(srcs), len(os.sched_getaffinity(0)), 16))
        with concurrent.futures.ThreadPoolExecutor(workers) as pool:
            objs = list(pool.map(lambda f: _compile(f, objdir, verbose), srcs))
        tmp = LIB_PATH + ".tmp"
        _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
