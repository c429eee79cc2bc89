"""Build libknnlm.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import concurrent.futures
import glob
import hashlib
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libknnlm.so")
# Hash of the sources a library was built from, written next to it by build().
LIB_HASH = LIB + ".srchash"
OBJDIR = os.path.join(ROOT, "_build", "obj")

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 VALU ops are kept out of the device code on purpose.
CFLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", INCLUDE, "-I", CSRC]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return obj


def _deps():
    return sorted(sources() + glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(INCLUDE, "*.h")))


def source_hash() -> str:
    """sha256 over the names and contents of the HIP sources and headers the library is built from."""
    h = hashlib.sha256()
    for p in _deps():
        h.update(os.path.relpath(p, ROOT).encode() + b"\0")
        with open(p, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()


def build(verbose: bool = False) -> str:
    """Compile every csrc/*.hip and link libknnlm.so next to this file."""
    os.makedirs(OBJDIR, exist_ok=True)
    digest = source_hash()
    srcs = sources()
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    with open(LIB_HASH + ".tmp", "w") as f:
        f.write(digest + "\n")
    os.replace(LIB_HASH + ".tmp", LIB_HASH)
    if verbose:
        print(f"built {LIB}")
    return LIB


def stale() -> bool:
    """True if libknnlm.so is missing or was not built from the sources as they are now."""
    if not os.path.exists(LIB) or not os.path.exists(LIB_HASH):
        return True
    with open(LIB_HASH) as f:
        return f.read().strip() != source_hash()


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
