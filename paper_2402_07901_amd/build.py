"""Builds libfastmax.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_2402_07901_amd.build   (or build() from Python)
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libfastmax.so")
OBJDIR = os.path.join(HERE, "_build")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics",
    "-Wall", "-Wno-unused-function",
    f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
]


def sources():
    out = []
    for name in sorted(os.listdir(CSRC)):
        if name.endswith(".hip") or name.endswith(".cpp"):
            out.append(os.path.join(CSRC, name))
    return out


# Per-source extra compiler flags (none needed at present).
EXTRA = {}


# Sanitizer build (tests/test_sanitize.py): AddressSanitizer and UBSan on the
# host code only (argument validation, workspace plans, dispatch); the GPU
# code is built as usual.  Linked by clang++ against the HIP runtime.
LIB_ASAN = os.path.join(HERE, "libfastmax_asan.so")
OBJDIR_ASAN = os.path.join(HERE, "_build_asan")
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host",
                 "-fno-omit-frame-pointer", "-Xarch_host", "-g"]
CLANGXX = os.environ.get("CLANGXX", "/opt/rocm/llvm/bin/clang++")


def _compile(src: str, sanitize: bool = False) -> str:
    objdir = OBJDIR_ASAN if sanitize else OBJDIR
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    extra = HOST_SANITIZE if sanitize else []
    cmd = [HIPCC, *COMMON, *EXTRA.get(os.path.basename(src), []), *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compiles every source in csrc/ and links libfastmax.so (with
    ``sanitize``: libfastmax_asan.so, host code under ASan/UBSan).  Returns
    its path."""
    objdir = OBJDIR_ASAN if sanitize else OBJDIR
    lib = LIB_ASAN if sanitize else LIB
    os.makedirs(objdir, exist_ok=True)
    srcs = sources()
    jobs = min(len(srcs), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(lambda s: _compile(s, sanitize), srcs))
    tmp = lib + ".tmp"
    if sanitize:
        rocm = os.path.dirname(os.path.dirname(HIPCC))
        cmd = [CLANGXX, "-shared", "-fPIC", "-fsanitize=address,undefined", "-o", tmp, *objs,
               f"-L{os.path.join(rocm, 'lib')}", "-lamdhip64"]
    else:
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
