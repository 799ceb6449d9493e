"""Build the native library libcs.so in-tree for gfx950.

    python -m paper_2112_13896_amd.build

Compiles the HIP kernels and C ABI (csrc/cs_api.hip) and the host pack
routine (csrc/cs_pack.cpp) with hipcc, once as the product library and once
with the product counter compiled in (libcs_count.so, used by tests).  Packed-fp32 instruction generation is
switched off for all device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libcs.so")
COUNT_LIB = os.path.join(HERE, "libcs_count.so")
STAMP_LIB = os.path.join(HERE, "libcs_stamps.so")
ARCH = "gfx950"

DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources() -> list:
    return [os.path.join(CSRC, "cs_api.hip"), os.path.join(CSRC, "cs_pack.cpp")]


def source_digest() -> str:
    """SHA-256 over every native source and header the library is built from."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                   if f.endswith((".hip", ".cpp", ".h")))
    files.append(os.path.join(INCLUDE, "cs.h"))
    for f in files:
        h.update(os.path.basename(f).encode())
        h.update(open(f, "rb").read())
    return h.hexdigest()


def _cmd(out: str, extra: list) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Wall", "-Wno-unused-command-line-argument", *DEVICE_FLAGS, "-I", INCLUDE, "-I", CSRC,
            *extra, "-o", out, *sources()]


def build(verbose: bool = False, extra: list | None = None, counting: bool = True) -> str:
    """Compile libcs.so (always recompiles) and, with `counting`, the two
    instrumented builds: libcs_count.so (every multiply-route-sum kernel counts
    the products it forms; tests only) and libcs_stamps.so (phase stamps; the
    benchmark's phase report), the compilations side by side.  Returns the
    path of libcs.so."""
    jobs = [(LIB, list(extra or []))]
    if counting:
        jobs.append((COUNT_LIB, list(extra or []) + ["-DCS_COUNT_PRODUCTS"]))
        jobs.append((STAMP_LIB, list(extra or []) + ["-DCS_PHASE_STAMPS"]))
    procs = []
    for out, ex in jobs:
        cmd = _cmd(out + ".tmp", ex)
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((out, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                            text=True)))
    failed = None
    noise = "is not a recognized feature for this target"
    for out, p in procs:
        text = p.communicate()[0]
        if p.returncode != 0:
            sys.stderr.write(text)
            failed = failed or f"hipcc failed with exit code {p.returncode} ({os.path.basename(out)})"
            continue
        msgs = [ln for ln in text.splitlines() if noise not in ln and ln.strip()]
        if msgs and verbose:
            print("\n".join(msgs))
    if failed:
        raise RuntimeError(failed)
    for out, _ in procs:
        os.replace(out + ".tmp", out)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
