"""Build the HIP library (gfx950) of the fingerprint forward pass.

Compiles every translation unit under csrc/ with hipcc for gfx950 and links
``libfp_mi355x.so`` next to this file.  Always recompiles (the build check
runs where no GPU is present: hipcc cross-compiles).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libfp_mi355x.so")
BUILD_DIR = os.path.join(HERE, "_build")

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str, hipcc: str, build_dir: str, extra: list) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [hipcc, *COMMON, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, out: str | None = None, defines: dict | None = None) -> str:
    """Compile and link.  ``out`` overrides the library path and ``defines`` adds -D
    macros (tuning constants such as SKINNY_NS or FP_TARGET_WG)."""
    hipcc = _hipcc()
    lib = out or LIB
    extra = [f"-D{k}={v}" for k, v in (defines or {}).items()]
    build_dir = BUILD_DIR if not extra else os.path.join(BUILD_DIR, "v_" + "_".join(f"{k}{v}" for k, v in sorted(defines.items())))
    os.makedirs(build_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, hipcc, build_dir, extra), srcs))
    LIB_ = lib
    tmp = LIB_ + ".tmp"
    # -z defs: an unresolved symbol (e.g. a kernel whose host stub was not emitted) fails the
    # link instead of the first load
    cmd = [hipcc, "-shared", f"--offload-arch={ARCH}", "-fPIC", "-Wl,-z,defs", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB_)
    if verbose:
        print("built", LIB_)
    return LIB_


if __name__ == "__main__":
    build(verbose=True)
