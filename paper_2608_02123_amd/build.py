"""Build ``libpctree.so`` (the C-ABI library and its gfx950 kernels) in-tree."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpctree.so")
SOURCES = ["pctree_api.hip", "pctree_kernels.hip", "pctree_profile.hip", "pctree_verify.hip",
           "pctree_attention.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libpctree.so)")


def compile_flags() -> list[str]:
    return [
        f"--offload-arch={ARCH}",
        "-O3",
        "-std=c++17",
        "-fPIC",
        # no packed-fp32 VALU ops in device code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # (the wide head stage loads LDS through M0 in inline assembly on purpose)
        "-Wno-inline-asm",
        f"-I{INCLUDE}",
        f"-I{CSRC}",
    ]


# AddressSanitizer on the host code only (the device code is built as usual):
# the checking build of the C ABI, loaded with the sanitizer runtime preloaded
ASAN_LIB = os.path.join(PKG, "libpctree_asan.so")
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]

# The stage-timeline build (include/pctree_profile.h): the kernels compiled
# with their wall-clock stamps, linked with the other objects of the default
# build into a library of its own
TIMELINE_LIB = os.path.join(PKG, "libpctree_timeline.so")
TIMELINE_SOURCE = "pctree_kernels.hip"


def _link(cc, objs, out, extra, verbose):
    tmp = out + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)


def build(verbose: bool = False, asan: bool = False, timeline: bool = True) -> str:
    """Compile every HIP source for gfx950 and link ``libpctree.so`` and, with
    ``timeline``, ``libpctree_timeline.so`` (or, with ``asan``,
    ``libpctree_asan.so`` with host-side AddressSanitizer); returns the path
    of the main library."""
    cc = hipcc()
    extra = ASAN_FLAGS if asan else []
    timeline = timeline and not asan
    jobs = [(src, os.path.join(CSRC, src.replace(".hip", "_asan.o" if asan else ".o")), [])
            for src in SOURCES]
    if timeline:
        jobs.append((TIMELINE_SOURCE, os.path.join(CSRC, "pctree_kernels_timeline.o"),
                     ["-DPCTREE_TIMELINE"]))
    procs = []
    for src, obj, defs in jobs:  # the sources compile side by side
        cmd = [cc, *compile_flags(), *extra, *defs, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stderr=None if verbose else subprocess.DEVNULL)))
    for cmd, proc in procs:
        if proc.wait() != 0:
            raise subprocess.CalledProcessError(proc.returncode, cmd)
    objs = [obj for src, obj, defs in jobs if not defs]
    out = ASAN_LIB if asan else LIB
    _link(cc, objs, out, extra, verbose)
    if timeline:
        tobjs = [obj if src != TIMELINE_SOURCE else jobs[-1][1] for src, obj, defs in jobs
                 if not defs]
        _link(cc, tobjs, TIMELINE_LIB, extra, verbose)
    for _, obj, _ in jobs:
        os.remove(obj)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, asan="--asan" in sys.argv,
                timeline="--no-timeline" not in sys.argv))
