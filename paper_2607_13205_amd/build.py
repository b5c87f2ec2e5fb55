"""Build libkve.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2607_13205_amd.build

compiles every source of csrc/ to an object under _build/ (in parallel) and
links paper_2607_13205_amd/libkve.so.  Every HIP compile disables the packed
fp32 instructions (v_pk_*_f32), which must not be emitted on this platform.
"""

from __future__ import annotations

import concurrent.futures as cf
import hashlib
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libkve.so")
HASH_FILE = LIB + ".sha256"  # hash of the sources the library was built from
ARCH = "gfx950"

SOURCES = ["kve_api.cpp", "snapkv.hip", "h2o.hip", "topk.hip", "decode.hip", "quest.hip", "probe.hip",
           "ceiling.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC,
          "-Wall", "-Wno-unused-result"]
HIP_ONLY = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-munsafe-fp-atomics"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def source_hash() -> str:
    """SHA-256 over every file of csrc/ and include/ (names and contents) and
    the build flags with the checkout's own paths taken out, so that the same
    sources give the same hash in any checkout."""
    h = hashlib.sha256()
    for d in (CSRC, os.path.join(ROOT, "include")):
        for name in sorted(os.listdir(d)):
            path = os.path.join(d, name)
            if os.path.isfile(path):
                h.update(os.path.relpath(path, ROOT).encode() + b"\0")
                with open(path, "rb") as f:
                    h.update(f.read())
                h.update(b"\0")
    flags = [f.replace(ROOT, "<root>") for f in COMMON + HIP_ONLY + SOURCES]
    h.update("\0".join(flags).encode())
    return h.hexdigest()


def built_hash() -> str | None:
    """Hash recorded when the present libkve.so was built (None if unknown)."""
    try:
        with open(HASH_FILE) as f:
            return f.read().strip() or None
    except OSError:
        return None


def _compile(src: str, digest: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [hipcc()] + COMMON + (HIP_ONLY if src.endswith(".hip") else ["-x", "hip"] + HIP_ONLY)
    if src == "kve_api.cpp":  # the library reports the hash of its sources
        cmd += [f'-DKVE_SOURCE_HASH="{digest}"']
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build_library(verbose: bool = False) -> str:
    """Compile and link libkve.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    digest = source_hash()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, digest), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    with open(HASH_FILE + ".tmp", "w") as f:
        f.write(digest + "\n")
    os.replace(HASH_FILE + ".tmp", HASH_FILE)
    if verbose:
        print(f"built {LIB} (sources {digest[:16]})")
    return LIB


def ensure_built() -> str:
    """Path of libkve.so, (re)building it first when it is missing or was
    built from other sources than the present csrc/ and include/."""
    if not os.path.exists(LIB) or built_hash() != source_hash():
        build_library()
    return LIB


if __name__ == "__main__":
    build_library(verbose=True)
    sys.exit(0)
