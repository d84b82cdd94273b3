"""Build libvideomla.so in-tree with hipcc for gfx950.

Every HIP/C++ source under csrc/ is compiled to an object under _build/ (in parallel) and
linked into paper_2605_30351_amd/libvideomla.so. The diagnostic variant, the same sources
compiled with VMLA_PHASE_STAMPS (include/videomla_stamps.h), goes to libvideomla_stamps.so.
Run as `python paper_2605_30351_amd/build.py [--stamps | --all]` (it does not import the
package, whose binding needs the built library).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libvideomla.so")
STAMPS_LIB = os.path.join(PKG, "libvideomla_stamps.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 VALU ops are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def _sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def _compile(src: str, extra: list[str], build_dir: str) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *COMMON, *extra, *lang, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, extra: list[str] | None = None, stamps: bool = False) -> str:
    """Compile every source and link the shared library (the diagnostic variant with
    stamps=True); returns its path."""
    build_dir = os.path.join(BUILD, "stamps") if stamps else BUILD
    lib = STAMPS_LIB if stamps else LIB
    os.makedirs(build_dir, exist_ok=True)
    extra = list(extra or []) + (["-DVMLA_PHASE_STAMPS"] if stamps else [])
    srcs = _sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, extra, build_dir), srcs))
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib} from {len(srcs)} sources")
    return lib


def build_all(verbose: bool = False) -> list[str]:
    """Both libraries, built side by side."""
    with cf.ThreadPoolExecutor(max_workers=2) as ex:
        futs = [ex.submit(build, verbose, None, st) for st in (False, True)]
        return [f.result() for f in futs]


if __name__ == "__main__":
    args = sys.argv[1:]
    if "--all" in args:
        build_all(verbose=True)
    else:
        build(verbose=True, extra=[x for x in args if x != "--stamps"], stamps="--stamps" in args)
