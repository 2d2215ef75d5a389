"""Build of ``libmfsgd.so`` (HIP, gfx950) in the package directory.

Every translation unit is compiled with hipcc for gfx950 only, with the packed
FP32 instructions disabled, then linked into one shared library.  Object files
go to ``_build/`` beside the sources; the library lands next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import hashlib
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmfsgd.so")
SOURCES = ["mfsgd_api.hip", "mfsgd_aux.hip", "mfsgd_table.hip", "mfsgd_kernels_f32.hip", "mfsgd_kernels_f16.hip"]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def _inputs_digest(src: str) -> str:
    """Digest of everything an object is built from: the source, every header
    beside it and the public headers (taken before compiling, so an edit made
    while the compiler runs leaves the object marked stale)."""
    h = hashlib.sha256()
    deps = [os.path.join(CSRC, src)] + sorted(os.path.join(CSRC, x) for x in os.listdir(CSRC) if x.endswith(".hpp"))
    deps += sorted(os.path.join(INCLUDE, x) for x in os.listdir(INCLUDE))
    for d in deps:
        with open(d, "rb") as f:
            h.update(os.path.basename(d).encode())
            h.update(f.read())
    h.update(" ".join(CFLAGS).encode())
    return h.hexdigest()


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    digest = _inputs_digest(src)
    cmd = [HIPCC, *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    with open(obj + ".inputs", "w") as f:
        f.write(digest + "\n")
    return obj


def _stale(src: str) -> bool:
    """Whether the object of `src` was built from other inputs than the
    current ones (or not at all)."""
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    try:
        with open(obj + ".inputs") as f:
            built = f.read().strip()
    except OSError:
        return True
    return not os.path.exists(obj) or built != _inputs_digest(src)


def build(jobs: int = 4, changed_only: bool = False) -> str:
    """Compile every HIP source (changed_only: those whose object is older than
    its inputs) and link libmfsgd.so; returns its path."""
    os.makedirs(OBJDIR, exist_ok=True)
    todo = [s for s in SOURCES if not changed_only or _stale(s)]
    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(SOURCES)))) as ex:
        list(ex.map(_compile, todo))
    objs = [os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    import sys
    print(build(changed_only="--changed" in sys.argv))
