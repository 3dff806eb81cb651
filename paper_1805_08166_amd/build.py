"""Builds libautotensor.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import glob
import hashlib
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libautotensor.so")
# digest of the sources the library was built from, written beside it
DIGEST = os.path.join(HERE, "libautotensor.srchash")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # fp32 sums must stay single IEEE adds (no contraction into FMAs)
    "-ffp-contract=off",
    "-fno-fast-math",
    # no packed-fp32 instructions in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.cpp")) + glob.glob(os.path.join(CSRC, "*.hip")))


OBJ_DIR = os.path.join(HERE, "_build")


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source under csrc/ (one hipcc per file, in parallel)
    and link them into one shared library."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    inc = ["-I", os.path.join(HERE, "..", "include")]
    objs = []
    cmds = []
    for src in sources():
        obj = os.path.join(OBJ_DIR, os.path.basename(src) + ".o")
        objs.append(obj)
        cmds.append(["hipcc", *HIPCC_FLAGS, *inc, "-c", "-o", obj, src])

    def run(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)

    with ThreadPoolExecutor(max_workers=max(1, jobs)) as pool:
        for f in [pool.submit(run, c) for c in cmds]:
            f.result()
    digest = source_digest()
    tmp = LIB + ".tmp"
    run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    with open(DIGEST, "w") as f:
        f.write(digest + "\n")
    return LIB


def inputs():
    """Every file the library is built from: sources, headers, the C ABI."""
    return sorted(sources() + glob.glob(os.path.join(CSRC, "*.h"))) + [
        os.path.join(HERE, "..", "include", "autotensor.h")]


def source_digest() -> str:
    h = hashlib.sha256()
    for p in inputs():
        h.update(os.path.basename(p).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def stale() -> bool:
    """True when the library is missing or was built from other sources."""
    if not os.path.exists(LIB) or not os.path.exists(DIGEST):
        return True
    with open(DIGEST) as f:
        return f.read().strip() != source_digest()


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
