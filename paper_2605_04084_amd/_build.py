"""Compile libfasq.so (HIP, gfx950) in-tree with hipcc.

Every source under ``csrc/`` is compiled to an object in ``_build/`` and the
objects are linked into ``libfasq.so`` next to this file.  The build always
recompiles (it is the "does it build" check); it is cheap enough to run per
change.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
from typing import List, Optional, Sequence

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
REPO_DIR = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
BUILD_DIR = os.path.join(REPO_DIR, "_build")
LIB_PATH = os.path.join(PKG_DIR, "libfasq.so")
ARCH = "gfx950"

COMMON_FLAGS = [
    "-O3",
    "-std=c++17",
    "-fPIC",
    f"--offload-arch={ARCH}",
    "-I", os.path.join(REPO_DIR, "include"),
    "-Wall",
    "-Wno-unused-function",
    # keep the compiler from forming packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: a ROCm toolchain is required to build libfasq")
    return path


def sources() -> List[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _compile(src: str, verbose: bool, build_dir: str = BUILD_DIR, defines: Sequence[str] = ()) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [hipcc(), *COMMON_FLAGS, *(f"-D{d}" for d in defines), "-c", src, "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)}:\n{errs}")
    if verbose and errs.strip():
        print(errs, file=sys.stderr)
    return obj


def build(verbose: bool = False, jobs: Optional[int] = None, defines: Sequence[str] = (),
          lib_path: str = LIB_PATH) -> str:
    """Compile every source and link ``libfasq.so``; returns the library path.

    ``defines`` (``NAME=VALUE`` strings) select compile-time variants, for
    example ``FASQ_DECODE_DOT=0`` (the one- and two-token decode kernels on
    the diagonal MFMA); such builds go to ``lib_path`` with their objects in
    a build directory of their own."""
    build_dir = BUILD_DIR if not defines else os.path.join(BUILD_DIR, "variant_" + "_".join(defines).replace("=", "-"))
    os.makedirs(build_dir, exist_ok=True)
    os.makedirs(os.path.dirname(os.path.abspath(lib_path)), exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, build_dir, defines), srcs))
    tmp = lib_path + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking libfasq.so failed:\n{r.stderr}")
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    import argparse

    ap = argparse.ArgumentParser(description="build libfasq.so for gfx950")
    ap.add_argument("-v", "--verbose", action="store_true")
    ap.add_argument("-D", dest="defines", action="append", default=[], metavar="NAME=VALUE",
                    help="compile-time variant (needs --out)")
    ap.add_argument("--out", default=LIB_PATH, help="library path (default: the in-tree libfasq.so)")
    a = ap.parse_args()
    if a.defines and os.path.abspath(a.out) == os.path.abspath(LIB_PATH):
        ap.error("a variant build needs --out: the in-tree library is the default build")
    print(build(verbose=a.verbose, defines=a.defines, lib_path=a.out))
