"""Identity of a build of ``libhf.so``: the SHA-256 of the sources it is
compiled from (every file of ``csrc/`` and the public header, in name order).

The build passes it to the compiler; the library returns it from
``hf_build_id()``, and the binding compares it with the sources on disk so
that a stale library is never loaded.
"""

import hashlib
import os

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
HEADER = os.path.join(os.path.dirname(HERE), "include", "hf.h")
SOURCES = ["hf_api.cpp", "gemm.hip", "gemm_bf16.hip", "rowops.hip", "cgvec.hip",
           "noalloc.hip", "narrow.hip"]


def source_files():
    files = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC))
             if f.endswith((".cpp", ".hip", ".h"))]
    return files + [HEADER]


def source_hash():
    h = hashlib.sha256()
    for path in source_files():
        h.update(os.path.basename(path).encode() + b"\0")
        with open(path, "rb") as fh:
            h.update(fh.read())
        h.update(b"\0")
    return h.hexdigest()
