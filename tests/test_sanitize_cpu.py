"""Host AddressSanitizer and UndefinedBehaviorSanitizer run of the C ABI.

Builds a copy of libhf.so whose host code (argument validation, workspace
layout, the solvers' host loops) is instrumented with ASan and UBSan, and
runs the CPU tests of the ABI (tests/test_abi_cpu.py) against it in a child
process with the sanitizer runtime preloaded.  The device code is built as
usual; nothing here touches a GPU.  Any report of either sanitizer fails the
child, and with it this test.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host",
       "-fno-sanitize-recover=undefined", "-Xarch_host", "-shared-libsan",
       "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime():
    out = subprocess.run(["/opt/rocm/llvm/bin/clang",
                          "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True)
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(600)
def test_abi_under_host_sanitizers():
    rt = asan_runtime()
    if rt is None:
        pytest.skip("no ASan runtime in this toolchain")
    from paper_1606_00511_amd.build import OBJDIR, build_library
    lib = os.path.join(OBJDIR, "asan", "libhf_asan.so")
    build_library(out=lib, host_extra=SAN, objdir=os.path.join(OBJDIR, "asan"))
    env = dict(os.environ)
    env.update(HF_LIB_PATH=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=23",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True)
    tail = (res.stdout + res.stderr)[-4000:]
    assert res.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
    assert " passed" in res.stdout
