"""Builds the gfx950 HIP library ``libalp.so`` in-tree with hipcc.

Every source is compiled to an object in parallel, then the objects are linked into one shared
library.  The kernels contain no cross-file device calls, so no relocatable device code is
needed.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libalp.so")
SOURCES = ["alp_api.hip", "alp_kernels.hip", "alp_split.hip", "alp_pruned.hip", "alp_stats.hip",
           "alp_place.hip", "alp_static.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMPILE_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # No packed fp32 instructions in the device code.  clang cannot forward -Xclang options to
    # the device pass alone (-Xarch_device rejects options that take an argument), so the host
    # pass sees the feature too and reports that x86 does not know it; that report is dropped
    # from the build output below.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]
# What the host pass prints for the device-only feature above.
_HOST_FEATURE_NOTE = "'-packed-fp32-ops' is not a recognized feature for this target"


def _run(cmd):
    p = subprocess.run(cmd, capture_output=True, text=True)
    lines = [ln for ln in (p.stdout + p.stderr).splitlines() if _HOST_FEATURE_NOTE not in ln]
    if lines:
        print("\n".join(lines), file=sys.stderr)
    if p.returncode != 0:
        raise subprocess.CalledProcessError(p.returncode, cmd)


def build(extra_flags=(), out: str = LIB) -> str:
    """Compiles every source into ``out`` (always rebuilds)."""
    with tempfile.TemporaryDirectory(prefix="alp_build_") as tmp:
        objs = [os.path.join(tmp, s + ".o") for s in SOURCES]
        cmds = [[HIPCC, *COMPILE_FLAGS, *extra_flags, "-c", os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
        workers = min(len(cmds), max(1, len(os.sched_getaffinity(0))))
        with ThreadPoolExecutor(workers) as pool:
            for f in [pool.submit(_run, c) for c in cmds]:
                f.result()
        tmp_lib = out + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp_lib,
              "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx"])
        os.replace(tmp_lib, out)
    return out


if __name__ == "__main__":
    print(build())
