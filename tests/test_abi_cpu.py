"""Host-side checks of the C ABI that need no GPU: the library loads, every
symbol include/hf.h declares is exported, and argument validation rejects
bad input before any device call."""

import ctypes
import os
import re

import pytest

from paper_1606_00511_amd import hf as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(H.LIB_PATH):
        from paper_1606_00511_amd.build import build_library
        build_library()
    return H.lib()


def declared_functions():
    txt = open(os.path.join(ROOT, "include", "hf.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    names = re.findall(r"\b(hf_[a-z_]+)\s*\(", txt)
    return sorted(set(names))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(H.EXPORTS)


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def create(L, dims, act=H.HF_SIGMOID, prec=H.HF_FP32, max_batch=16):
    arr = (ctypes.c_int32 * len(dims))(*dims)
    h = ctypes.c_void_p()
    rc = L.hf_create(arr, len(dims), act, prec, max_batch, None, ctypes.byref(h))
    return rc, h


def test_create_validates(L):
    assert create(L, [4])[0] == H.HF_EINVAL                 # need L >= 1
    assert create(L, [4, 0, 3])[0] == H.HF_EINVAL           # zero width
    assert create(L, [4, -2, 3])[0] == H.HF_EINVAL
    assert create(L, [4, 3], act=7)[0] == H.HF_EINVAL       # unknown act
    assert create(L, [4, 3], prec=3)[0] == H.HF_EINVAL      # unknown precision
    rc, h = create(L, [4, 3], prec=H.HF_BF16_INPUTS)       # bf16 GEMM inputs
    assert rc == H.HF_OK and L.hf_destroy(h) == H.HF_OK
    assert create(L, [4, 3], max_batch=0)[0] == H.HF_EINVAL
    assert create(L, [4, 5000])[0] == H.HF_EINVAL           # > HF_MAX_CLASSES
    assert create(L, [2] * 18)[0] == H.HF_EINVAL            # > HF_MAX_LAYERS
    assert create(L, [1 << 20, 4096], max_batch=4096)[0] == H.HF_EINVAL  # 2^31
    assert L.hf_create(None, 2, 0, 0, 4, None, None) == H.HF_EINVAL
    arr = (ctypes.c_int32 * 2)(4, 3)
    assert L.hf_create(arr, 2, 0, 0, 4, None, None) == H.HF_EINVAL  # no out


@pytest.mark.parametrize("dims", [(784, 100, 10), (784, 500, 500, 500, 10),
                                  (440, 2048, 2048, 2048, 2048, 1973), (3, 1)])
def test_num_params_and_workspace(L, dims):
    rc, h = create(L, list(dims), max_batch=64)
    assert rc == H.HF_OK
    n = sum(dims[l] * (dims[l - 1] + 1) for l in range(1, len(dims)))
    assert L.hf_num_params(h) == n
    ws = L.hf_workspace_bytes(h, 0)
    assert ws > 4 * 3 * n  # at least the CG vectors
    assert L.hf_workspace_bytes(h, 64) == ws
    # the bytes grow with the batch the workspace serves
    sizes = [L.hf_workspace_bytes(h, b) for b in (1, 2, 17, 63, 64)]
    assert all(a <= b for a, b in zip(sizes, sizes[1:])) and sizes[0] > 4 * 3 * n
    assert L.hf_workspace_bytes(h, 65) == 0
    assert L.hf_destroy(h) == H.HF_OK
    rc, h = create(L, list(dims), prec=H.HF_BF16_INPUTS, max_batch=64)
    assert rc == H.HF_OK and L.hf_num_params(h) == n
    assert L.hf_workspace_bytes(h, 0) > 4 * 3 * n
    assert L.hf_workspace_bytes(h, 1) <= L.hf_workspace_bytes(h, 64)
    assert L.hf_destroy(h) == H.HF_OK


def test_calls_without_workspace_or_with_bad_args(L):
    rc, h = create(L, [8, 6, 4])
    assert rc == H.HF_OK
    n = L.hf_num_params(h)
    fake = ctypes.c_void_p(1 << 20)   # never dereferenced: validation fails first
    rc = L.hf_loss_grad(h, fake, fake, fake, 4, fake, fake)
    assert rc == H.HF_EWORKSPACE
    assert b"workspace" in L.hf_last_error(h)
    # workspace argument checks happen before any device call
    assert L.hf_set_workspace(h, None, 1 << 30) == H.HF_EINVAL
    assert L.hf_set_workspace(h, ctypes.c_void_p(4096 + 16), 1 << 30) == H.HF_EINVAL
    assert b"256-byte" in L.hf_last_error(h)
    assert L.hf_set_workspace(h, ctypes.c_void_p(4096), 16) == H.HF_EWORKSPACE
    info = H.hf_cg_info()
    assert L.hf_cg(h, fake, fake, fake, 4, fake, 0.01, 5, 0.0, 0, fake, fake,
                   ctypes.byref(info)) == H.HF_EWORKSPACE
    assert L.hf_bicgstab(h, fake, fake, fake, 4, fake, 0.01, 5, 0.0, 0, fake,
                         fake, ctypes.byref(info)) == H.HF_EWORKSPACE
    assert L.hf_pcg(h, fake, fake, fake, 4, fake, 0.01, 5, 0.0, 0, fake, fake,
                    fake, ctypes.byref(info)) == H.HF_EWORKSPACE
    assert L.hf_pbicgstab(h, fake, fake, fake, 4, fake, 0.01, 5, 0.0, 0, fake,
                          fake, fake, ctypes.byref(info)) == H.HF_EWORKSPACE
    assert L.hf_fisher_diag(h, fake, fake, fake, 4, fake) == H.HF_EWORKSPACE
    assert L.hf_loss(h, fake, fake, fake, 4, fake) == H.HF_EWORKSPACE
    prm = H.hf_iter_params(0, 0, 0.01, 5, 0.0, 0.0, 1e-4, 0.5, 10)
    hs = ctypes.c_int32(0)
    it = H.hf_iter_info()
    assert L.hf_iterate(h, fake, fake, fake, 4, fake, fake, 4, ctypes.byref(prm),
                        ctypes.byref(hs), fake, ctypes.byref(it)) == H.HF_EWORKSPACE
    assert L.hf_destroy(h) == H.HF_OK
    assert n == 6 * 9 + 4 * 7


def test_null_context(L):
    assert L.hf_num_params(None) == -1
    assert L.hf_workspace_bytes(None, 0) == 0
    assert L.hf_set_trace(None, None, 0) == H.HF_EINVAL
    assert L.hf_destroy(None) == H.HF_OK
    assert L.hf_last_error(None) == b"null context"
    assert L.hf_strerror(H.HF_ELABEL) == b"HF_ELABEL"
    assert L.hf_set_stream(None, None) == H.HF_EINVAL
    assert L.hf_check(None) == H.HF_EINVAL
    assert L.hf_prof_count(None) == 0


def test_trace_arguments(L):
    """hf_set_trace validates before any device call."""
    rc, h = create(L, [8, 6, 4])
    assert rc == H.HF_OK
    assert L.hf_set_trace(h, None, -1) == H.HF_EINVAL
    assert L.hf_set_trace(h, None, 3) == H.HF_EINVAL
    assert L.hf_set_trace(h, ctypes.c_void_p(4096 + 4), 3) == H.HF_EINVAL
    assert b"16-byte" in L.hf_last_error(h)
    assert L.hf_set_trace(h, ctypes.c_void_p(4096), 3) == H.HF_OK  # not touched
    assert L.hf_set_trace(h, None, 0) == H.HF_OK
    assert L.hf_destroy(h) == H.HF_OK


def test_build_id_matches_sources(L):
    """The library reports the hash of the sources it was built from, and
    the binding refuses a library whose hash differs from the sources on
    disk."""
    from paper_1606_00511_amd import buildid
    assert L.hf_build_id().decode() == buildid.source_hash()
    saved = H._lib
    try:
        H._lib = None
        real = H.source_hash
        H.source_hash = lambda: "0" * 64
        with pytest.raises(RuntimeError, match="other sources"):
            H.lib()
    finally:
        H.source_hash = real
        H._lib = saved


def test_noalloc_rejections_before_device_work(L):
    """hf_hvp_noalloc validates its arguments and the scratch size on the
    host: a NULL context, a batch outside [1, max_batch], a misaligned
    pointer, and a batch whose product layout exceeds the static scratch."""
    fake = ctypes.c_void_p(1 << 20)
    assert L.hf_hvp_noalloc(None, fake, fake, fake, 4, fake, 0, fake, None) == H.HF_EINVAL
    rc, h = create(L, [440, 2048, 2048, 2048, 2048, 1973], max_batch=16384)
    assert rc == H.HF_OK
    assert L.hf_hvp_noalloc(h, fake, fake, fake, 0, fake, 0, fake, None) == H.HF_EINVAL
    assert L.hf_hvp_noalloc(h, fake, fake, fake, 16385, fake, 0, fake, None) == H.HF_EINVAL
    assert L.hf_hvp_noalloc(h, ctypes.c_void_p((1 << 20) + 4), fake, fake, 4, fake, 0,
                            fake, None) == H.HF_EINVAL
    assert L.hf_hvp_noalloc(h, fake, fake, fake, 4, fake, 0, fake,
                            ctypes.c_void_p((1 << 20) + 2)) == H.HF_EINVAL
    assert L.hf_hvp_noalloc(h, fake, fake, fake, 16384, fake, 0, fake, None) == \
        H.HF_EWORKSPACE
    assert b"scratch" in L.hf_last_error(h)
    assert L.hf_destroy(h) == H.HF_OK
