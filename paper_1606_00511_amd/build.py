"""Build the HIP library ``libhf.so`` in-tree for gfx950.

Usage: ``python -m paper_1606_00511_amd.build`` (or ``build_library()``).
Every source in ``csrc/`` is compiled by hipcc (in parallel, one object per
source under ``_build/``) and linked into one shared object next to this file;
the Python binding loads it from there.  The library carries the SHA-256 of
the sources it was built from (``hf_build_id``), and the binding refuses a
library whose hash does not match the sources beside it.
"""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

from paper_1606_00511_amd.buildid import CSRC, SOURCES, source_hash

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libhf.so")
OBJDIR = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in res.stderr.splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    return res.returncode, errs


def build_library(verbose=False, out=LIB, extra=(), host_extra=(), objdir=OBJDIR):
    """Compile every source and link ``out``.  ``extra`` is added to every
    hipcc line; ``host_extra`` only to the host-only source (hf_api.cpp)."""
    os.makedirs(objdir, exist_ok=True)
    bid = source_hash()
    defs = ["-DHF_BUILD_ID=\"%s\"" % bid]
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    jobs = []
    for s in SOURCES:
        obj = os.path.join(objdir, s + ".o")
        cmd = [HIPCC] + FLAGS + list(extra) + defs + inc + ["-c", "-o", obj,
                                                         os.path.join(CSRC, s)]
        if s.endswith(".cpp"):
            cmd[1:1] = list(host_extra)
        jobs.append((cmd, obj))
    if verbose:
        for cmd, _ in jobs:
            print(" ".join(cmd), flush=True)
    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 4)) as ex:
        results = list(ex.map(lambda j: _run(j[0]), jobs))
    for (cmd, _), (rc, errs) in zip(jobs, results):
        if rc != 0:
            raise RuntimeError("hipcc failed (%d): %s\n%s" % (rc, cmd[-1], errs))
        if verbose and errs:
            print(errs, file=sys.stderr)
    tmp = out + ".tmp"
    link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + list(extra) + \
        list(host_extra) + ["-o", tmp] + [o for _, o in jobs]
    if verbose:
        print(" ".join(link), flush=True)
    rc, errs = _run(link)
    if rc != 0:
        raise RuntimeError("link failed (%d):\n%s" % (rc, errs))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build_library(verbose=True))
