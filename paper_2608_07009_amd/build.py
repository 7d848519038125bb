"""Build libhisparse.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2608_07009_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB_DIR = os.path.join(PKG, "lib")
LIB_PATH = os.path.join(LIB_DIR, "libhisparse.so")
SOURCES = ["api.hip", "resolve.hip", "attention.hip"]
ARCH = "gfx950"

# Packed fp32 instructions stay off: only plain fp32 VALU code is generated.
HIPCC_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Wall", "-Wno-unused-result",
               "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


PHASE_STAMPS_LIB_PATH = os.path.join(LIB_DIR, "libhisparse_phase_stamps.so")


def build(verbose: bool = False, phase_stamps: bool = False) -> str:
    """Compile and link the library. phase_stamps: the phase-timing variant (the resolve kernel
    records its phase boundaries; hisparse_debug_resolve_phases reads them), written beside the
    normal library as libhisparse_phase_stamps.so."""
    tag = "obj_phase_stamps" if phase_stamps else "obj"
    out = PHASE_STAMPS_LIB_PATH if phase_stamps else LIB_PATH
    extra = ["-DHISPARSE_PHASE_STAMPS"] if phase_stamps else []
    os.makedirs(os.path.join(LIB_DIR, tag), exist_ok=True)
    cc = hipcc()

    def compile_one(src: str) -> str:
        obj = os.path.join(LIB_DIR, tag, src.replace(".hip", ".o"))
        cmd = [cc, *HIPCC_FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        if verbose and (r.stdout or r.stderr):
            print(r.stdout, r.stderr, file=sys.stderr)
        return obj

    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, "-ldl"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True, phase_stamps="--phase-stamps" in sys.argv[1:]))
