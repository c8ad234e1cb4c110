"""Build ``libpackserve.so`` (the C-ABI window scorer) for gfx950 with hipcc.

Always recompiles.  Flags:
  * ``--offload-arch=gfx950``: CDNA4 only, no other targets.
  * ``-ffp-contract=off``: every fp32 expression is evaluated as written, so
    the same candidate always yields bit-identical latencies wherever the
    kernel evaluates it (filters and the reported values of the choice).
  * ``-Xclang -target-feature -Xclang -packed-fp32-ops``: no packed fp32
    instructions are generated.
  * ``-DPS_SOURCE_HASH``: :func:`source_hash` of the sources, returned by
    ``ps_build_id()``, so a stale library is told apart from a fresh one.
"""
from __future__ import annotations

import hashlib
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "libpackserve.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("ps_kernels.hip", "ps_sequential.hip", "ps_index.hip",
                                                   "ps_api.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def source_hash() -> str:
    """First 16 hex digits of the SHA-256 of the csrc files (in name order)
    followed by the C header: what ``ps_build_id()`` of a fresh build returns."""
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(f.read())
    with open(os.path.join(ROOT, "include", "packserve.h"), "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:16]


def build(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wall", "-Wno-unused-function", f'-DPS_SOURCE_HASH="{source_hash()}"',
           "-I", os.path.join(ROOT, "include"), "-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
