"""Build step: compile the HIP library for gfx950, in tree.

``python -m paper_2512_05831_amd.build`` (or ``build_library()``) runs hipcc on
``csrc/eb.hip`` (with ``csrc/eb_gather.h``), ``csrc/eb_gather_weighted.hip``,
``csrc/eb_gather_narrow.hip``, ``csrc/eb_gather_narrow_weighted.hip``,
``csrc/eb_exchange.hip`` and ``csrc/eb_ceiling.hip`` (the bandwidth probe the
benchmark uses) and writes ``libeb.so`` next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(HERE, "csrc", f)
        for f in ("eb.hip", "eb_gather_weighted.hip", "eb_gather_narrow.hip",
                  "eb_gather_narrow_weighted.hip", "eb_exchange.hip", "eb_ceiling.hip")]
LIB = os.path.join(HERE, "libeb.so")
ARCH = "gfx950"

# Packed fp32 instructions are disabled for all device code.
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def build_library(verbose: bool = False) -> str:
    """Compile libeb.so (always recompiles) and return its path.  The sources
    are compiled to objects in parallel, then linked."""
    import tempfile

    with tempfile.TemporaryDirectory(prefix="ebbuild") as tmpdir:
        procs = []
        for src in SRCS:
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            cmd = [hipcc(), *HIPCC_FLAGS, "-c", src, "-o", obj]
            procs.append((cmd, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                     stderr=subprocess.PIPE, text=True)))
        objs = []
        for cmd, obj, proc in procs:
            _, err = proc.communicate()
            if proc.returncode != 0:
                raise RuntimeError(f"hipcc failed ({proc.returncode}):\n{' '.join(cmd)}\n{err}")
            if verbose and err:
                sys.stderr.write(err)
            objs.append(obj)
        tmp = LIB + ".tmp"
        cmd = [hipcc(), *HIPCC_FLAGS, "-shared", *objs, "-o", tmp]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc link failed ({res.returncode}):\n{' '.join(cmd)}\n{res.stderr}")
        os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
