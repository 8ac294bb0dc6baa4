"""Builds libarckv.so in-tree: host C++ with g++, HIP kernels with hipcc for gfx950.

    python -m paper_2606_21238_amd.build          # or __graft_entry__.build()

Output: paper_2606_21238_amd/lib/libarckv.so (objects under paper_2606_21238_amd/_build/).
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
BUILD = os.path.join(PKG, "_build")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libarckv.so")
ARCH = "gfx950"

HOST_SRC = ["host/blockhash.cpp", "host/cache.cpp", "host/attn_plan.cpp", "host/prepare.cpp", "host/errors.cpp"]
HIP_SRC = ["kernels/kv_scatter.hip", "kernels/prefill_attn.hip", "kernels/qkv_rope.hip"]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm toolchain required to build libarckv)")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass does not know the device-only feature flag below; that note is noise
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed: {' '.join(cmd)}\n{out}")
    return out


SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
ASAN_BUILD = os.path.join(PKG, "_build_sanitize")
ASAN_LIB = os.path.join(LIBDIR, "libarckv_sanitize.so")
CHECKED_BUILD = os.path.join(PKG, "_build_checked")
CHECKED_LIB = os.path.join(LIBDIR, "libarckv_checked.so")


def build(verbose: bool = False, sanitize: bool = False, checked: bool = False) -> str:
    """sanitize: the host C++ (hashing, cache, planner, batch preparation) instrumented with
    AddressSanitizer and UndefinedBehaviorSanitizer, into lib/libarckv_sanitize.so, for CPU tests
    (load it with ARCKV_LIBRARY and the sanitizer runtimes preloaded).  The HIP sources are
    built as usual, with no sanitizer: device code is never instrumented.
    checked: the kernels with device checks (ARCKV_DEVICE_CHECKS: out-of-range indices they
    clamp or skip are recorded, see arckv_device_checks), into lib/libarckv_checked.so."""
    assert not (sanitize and checked)
    build_dir = ASAN_BUILD if sanitize else CHECKED_BUILD if checked else BUILD
    out_lib = ASAN_LIB if sanitize else CHECKED_LIB if checked else LIB
    os.makedirs(build_dir, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    hipcc = _hipcc()
    common = ["-O3", "-fPIC", "-std=c++17", "-Wall", f"-I{INCLUDE}", f"-I{os.path.join(CSRC, 'host')}"]
    host_flags = ["-O1", "-g", *SANITIZE] if sanitize else []
    jobs = []
    objs = []
    for src in HOST_SRC:
        obj = os.path.join(build_dir, os.path.basename(src) + ".o")
        jobs.append(["g++", *common, *host_flags, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HIP_SRC:
        obj = os.path.join(build_dir, os.path.basename(src) + ".o")
        jobs.append([hipcc, f"--offload-arch={ARCH}", *common, *(["-DARCKV_DEVICE_CHECKS"] if checked else []),
                     # no packed fp32 VALU ops are ever generated: some of their forms have given wrong results on gfx950
                     "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                     "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        outs = list(ex.map(_run, jobs))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = out_lib + ".tmp"
    if sanitize:
        # linked by g++ (no HIP source on this line), with the sanitizer runtimes
        _run(["g++", "-shared", "-fPIC", *SANITIZE, *objs, "-L/opt/rocm/lib", "-lamdhip64",
              f"-Wl,-rpath,/opt/rocm/lib", "-o", tmp])
    else:
        _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, out_lib)
    return out_lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv, checked="--checked" in sys.argv))
