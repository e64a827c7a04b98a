"""Build the CLEAR-MoE HIP library for gfx950 (in-tree ``libclearmoe.so``).

Every translation unit under ``csrc/`` is compiled with hipcc for gfx950
only, in parallel, then linked into one shared library next to this file.
Packed-FP32 instruction selection is disabled for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libclearmoe.so")
BUILD_DIR = os.path.join(ROOT, "_build", "clearmoe")
SOURCES = ["api.cpp", "route.hip", "dispatch.hip", "gemm.hip", "fused.hip", "fused_split.hip",
           "fused_cls.hip", "class_ffn.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# The library carries the digest of the sources it was built from after this
# marker, so that a stale binary is recognised without loading it.
DIGEST_MARKER = b"CLEARMOE-SOURCE-DIGEST="
DIGEST_LEN = 16
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", f"-I{INCLUDE}", f"-I{CSRC}"]


def source_digest() -> str:
    """SHA-256 (first 16 hex digits) over every file under csrc/ and the
    public header, names included."""
    h = hashlib.sha256()
    files = [(n, os.path.join(CSRC, n)) for n in sorted(os.listdir(CSRC))]
    files.append(("clearmoe.h", os.path.join(INCLUDE, "clearmoe.h")))
    for name, path in files:
        if not os.path.isfile(path):
            continue
        with open(path, "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:DIGEST_LEN]


def built_digest(path: str = LIB) -> str:
    """The source digest a built library carries ("" if none or no library)."""
    if not os.path.exists(path):
        return ""
    with open(path, "rb") as f:
        data = f.read()
    i = data.find(DIGEST_MARKER)
    if i < 0:
        return ""
    return data[i + len(DIGEST_MARKER): i + len(DIGEST_MARKER) + DIGEST_LEN].decode("ascii", "replace")


# Translation units whose device assembly is kept beside the objects (with
# the source digest), for the CPU check of the fused kernel's counted waits.
KEEP_ASM = ("fused.hip", "fused_split.hip", "fused_cls.hip")


def device_asm(src: str) -> str:
    """Path of the kept gfx950 assembly of a translation unit."""
    return os.path.join(BUILD_DIR, os.path.splitext(src)[0] + f"-hip-amdgcn-amd-amdhsa-{ARCH}.s")


def _compile(src: str, digest: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    keep = ["-save-temps=obj"] if src in KEEP_ASM else []
    cmd = [HIPCC, "-x", "hip", *FLAGS, *keep, f'-DCLEARMOE_SOURCE_DIGEST="{digest}"', "-c",
           os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=BUILD_DIR)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    if keep:
        with open(device_asm(src) + ".digest", "w") as f:
            f.write(digest)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link ``libclearmoe.so``.  Returns its path."""
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD_DIR, exist_ok=True)
    digest = source_digest()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, digest), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


def clean() -> None:
    shutil.rmtree(BUILD_DIR, ignore_errors=True)
    if os.path.exists(LIB):
        os.remove(LIB)


if __name__ == "__main__":
    build(verbose=True)
