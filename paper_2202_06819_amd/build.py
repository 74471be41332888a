"""Build libqconv.so (HIP kernels + C ABI) for gfx950, in-tree.

    python -m paper_2202_06819_amd.build

Every HIP source is compiled with hipcc for gfx950 only, with packed-FP32
instruction selection disabled, and linked into
``paper_2202_06819_amd/libqconv.so`` next to this file.

The library carries the digest of the sources and flags it was built from
(``qconv_build_digest()``; also a plain marker string in the file), so a
caller can tell a stale binary from a current one: :func:`ensure_built`
rebuilds when they differ.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libqconv.so")
ARCH = "gfx950"

CFLAGS = [
    "-x", "hip", f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC",
    "-Wall", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.isabs(cand) and os.path.exists(cand) or not os.path.isabs(cand)):
            return cand
    raise RuntimeError("hipcc not found")


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


DIGEST_MARKER = b"QCONV_SOURCE_DIGEST="


def source_digest() -> str:
    """sha256 (16 hex digits) of every source, header and compile flag the library is built from."""
    h = hashlib.sha256(" ".join(CFLAGS[:-2]).encode())
    files = sorted(glob.glob(os.path.join(CSRC, "*")) + [os.path.join(INCLUDE, "qconv.h")])
    for f in files:
        if os.path.isfile(f):
            h.update(os.path.basename(f).encode() + b"\0")
            with open(f, "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def built_digest(path: str = LIB) -> str | None:
    """The source digest recorded in a built library (read from the file, nothing is loaded), or None."""
    try:
        with open(path, "rb") as fh:
            data = fh.read()
    except OSError:
        return None
    i = data.find(DIGEST_MARKER)
    if i < 0:
        return None
    d = data[i + len(DIGEST_MARKER): i + len(DIGEST_MARKER) + 16]
    return d.decode("ascii", "replace")


def ensure_built(verbose: bool = False) -> str:
    """Build libqconv.so unless it exists and was built from the current sources."""
    if built_digest() != source_digest():
        build(verbose=verbose)
    return LIB


def _compile(src: str, verbose: bool, digest: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [_hipcc(), *CFLAGS, f"-DQCONV_SOURCE_DIGEST=\"{digest}\"", "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (res.stderr or "").splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return obj


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every HIP source and link libqconv.so; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    digest = source_digest()
    jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, digest), srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    if built_digest(tmp) != digest:
        raise RuntimeError(f"{tmp} does not carry the source digest {digest}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
