"""Build the gfx950 shared library ``_lib/libchunkattn.so`` in-tree with hipcc.

Usage: ``python -m paper_2402_15220_amd.build`` (or ``build()`` from Python).
Every HIP source is compiled for gfx950 only, with packed-fp32 instruction
generation disabled. ``build(sanitize=True, lib=path)`` builds the same
sources with AddressSanitizer and UndefinedBehaviorSanitizer on the host code
only (device code is compiled as usual) into another file, for host-side
tests; load it with ``CA_LIBRARY=path`` and the clang ASan runtime preloaded.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libchunkattn.so")
INCLUDE = os.path.join(os.path.dirname(PKG), "include")

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}",
]

# host-only sanitizer flags (each -fsanitize= right after -Xarch_host, so the
# device code is built without them)
SANITIZE = ("-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
            "-Xarch_host -fno-omit-frame-pointer -Xarch_host -g -shared-libasan").split()

SOURCES = ["tree.cpp", "tables.cpp", "capi.cpp", "kernels.hip", "prefill.hip", "fill.hip",
           "scratch.hip"]


def _compile(src: str, objdir: str, extra: list) -> str:
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC] + COMMON + extra + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False, lib: str | None = None) -> str:
    """Compile every source and link the library; always rebuilds. With
    `sanitize`, host code carries ASan and UBSan and the library goes to
    `lib` (required: the in-tree library stays the plain build)."""
    if sanitize and not lib:
        raise ValueError("a sanitized build needs its own output path")
    out = lib or LIB
    extra = SANITIZE if sanitize else []
    objdir = out + ".obj"
    os.makedirs(objdir, exist_ok=True)
    os.makedirs(os.path.dirname(out), exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, objdir, extra), SOURCES))
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + extra + objs + [
        f"-Wl,-rpath,{ROCM}/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    shutil.rmtree(objdir, ignore_errors=True)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
