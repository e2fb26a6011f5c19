"""Compile libblockserve.so (the HIP kernels and the C ABI) for gfx950 in-tree."""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libblockserve.so")


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


# Sources whose MFMA accumulators may live in AGPRs (none at present). The
# others keep their accumulators in ordinary VGPRs: the attention loop
# rescales them under a branch, which with AGPR accumulators costs copies
# every tile.
AGPR_SOURCES: set[str] = set()


def _compile(src: str, obj: str) -> subprocess.CompletedProcess:
    cmd = [hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-c",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    if os.path.basename(src) not in AGPR_SOURCES:
        cmd += ["-mllvm", "-amdgpu-mfma-vgpr-form"]
    cmd += ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
            "-Wno-unused-command-line-argument", "-o", obj, src]
    return subprocess.run(cmd, capture_output=True, text=True)


def build(verbose: bool = False) -> str:
    """Always recompiles every source (one object each, in parallel, then one
    link); returns the library path."""
    import tempfile
    from concurrent.futures import ThreadPoolExecutor

    srcs = sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory(prefix="bs_build_") as td:
        objs = [os.path.join(td, os.path.basename(s) + ".o") for s in srcs]
        with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
            results = list(ex.map(_compile, srcs, objs))
        for src, r in zip(srcs, results):
            if verbose:
                print("compiled", os.path.basename(src), flush=True)
            if r.returncode != 0:
                sys.stderr.write(r.stdout + r.stderr)
                raise RuntimeError(f"hipcc failed compiling {os.path.basename(src)}")
        link = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
        r = subprocess.run(link, capture_output=True, text=True)
        if r.returncode != 0:
            sys.stderr.write(r.stdout + r.stderr)
            raise RuntimeError("hipcc failed linking libblockserve.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
