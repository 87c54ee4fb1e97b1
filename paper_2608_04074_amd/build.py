"""Build libnovakv.so (gfx950) in-tree with hipcc: every source compiled to an
object in parallel (some with flags of their own), then linked."""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
import time
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libnovakv.so")
SOURCES = ["api.hip", "decode.hip", "decode_lut.hip", "decode_lut64.hip", "encode.hip", "host_checks.cpp"]
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from forming packed-fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]

# Flags of single sources.  The encoders: their min/max reductions see no NaN
# (IEEE mode off, so min/max need no canonicalizing moves), and the fp64
# matrix products write their results to VGPRs, where the VALU reads them.
SOURCE_FLAGS = {
    "encode.hip": ["-fno-honor-nans", "-mno-amdgpu-ieee", "-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = True, extra=(), csrc: str = CSRC, out: str = LIB) -> str:
    """Compile the library; `extra` flags go to every source (e.g. -D options)."""
    t = time.time()
    cc = hipcc()
    with tempfile.TemporaryDirectory(prefix="novakv_build_") as tmpdir:
        def compile_one(src):
            obj = os.path.join(tmpdir, src + ".o")
            cmd = [cc, *HIPCC_FLAGS, *SOURCE_FLAGS.get(src, []), *extra, "-c", os.path.join(csrc, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.run(cmd, check=True)
            return obj

        workers = max(1, min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
        with ThreadPoolExecutor(max_workers=workers) as pool:
            objs = list(pool.map(compile_one, SOURCES))
        tmp = out + ".tmp"
        cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    if verbose:
        print(f"built {out} in {time.time() - t:.1f}s", flush=True)
    return out


if __name__ == "__main__":
    build()
    sys.exit(0)
