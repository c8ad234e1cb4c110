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
  * ``-Rpass-analysis=kernel-resource-usage``: the compiler's register
    report of every kernel; the build fails if any kernel spills vector
    registers to scratch.  The kernels read other lanes' registers (ballots,
    DPP row reductions, readlane, shuffles), and a spilled register that is
    reloaded while some lanes are inactive keeps stale values in those lanes:
    a build of the four-requests-per-wave scorer forced to spill returned
    wrong decisions.
"""
from __future__ import annotations

import hashlib
import os
import re
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


def vgpr_spills(remarks: str) -> dict:
    """{kernel: vector registers spilled} from the compiler's
    kernel-resource-usage remarks."""
    out, cur = {}, None
    for line in remarks.splitlines():
        m = re.search(r"remark:\s+Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            continue
        m = re.search(r"remark:\s+VGPRs Spill: (\d+)", line)
        if m and cur is not None:
            out[cur] = int(m.group(1))
    return out


def build(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wall", "-Wno-unused-function", "-Rpass-analysis=kernel-resource-usage",
           f'-DPS_SOURCE_HASH="{source_hash()}"',
           "-I", os.path.join(ROOT, "include"), "-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # compiler diagnostics other than the register report (whose remarks
    # come with a source snippet each) and the host pass's note on the
    # packed-fp32 feature
    keep, skip = [], False
    for line in r.stderr.splitlines():
        if "remark:" in line or "packed-fp32-ops" in line:
            skip = True
            continue
        if re.search(r": (warning|error|note):", line):
            skip = False
        if not skip:
            keep.append(line)
    diag = "\n".join(keep)
    if diag.strip():
        print(diag, file=sys.stderr, flush=True)
    if r.returncode != 0:
        raise subprocess.CalledProcessError(r.returncode, cmd)
    spills = {k: v for k, v in vgpr_spills(r.stderr).items() if v}
    if not vgpr_spills(r.stderr):
        raise RuntimeError("no kernel resource report in the compiler output")
    if spills:
        os.remove(tmp)
        raise RuntimeError(f"kernels spill vector registers: {spills}")
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
