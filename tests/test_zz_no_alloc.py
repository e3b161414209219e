"""The entry point that allocates nothing (hf_hvp_noalloc), through the C ABI,
against the existing entry point it varies (hf_hvp) on the same inputs: the
fp32 bar (rel-L2 <= 1e-4; the two share their kernels and their layout for
the same batch, so the results are in fact bit-identical) and the bf16-operand
bar (2e-2).  Two calls in a row, the second with fewer rows, both modes; a
second context between two calls of the first (the scratch is shared); the
label flag; and the rejection of a batch whose layout exceeds the scratch,
before any device work.
"""

import ctypes

import numpy as np
import pytest

from paper_1606_00511_amd import workloads as WL
from tests.parity_util import rel

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def noalloc(net, W, X, y, v, mode, out, flag=None):
    """hf_hvp_noalloc on torch's current stream; returns the C return code."""
    import torch
    from paper_1606_00511_amd import hf as H
    L = H.lib()
    net._stream()
    B = int(X.shape[0])
    rc = L.hf_hvp_noalloc(net._h, W.data_ptr(), X.data_ptr(),
                          y.data_ptr() if y is not None else None, B, v.data_ptr(),
                          H.MODES[mode], out.data_ptr(),
                          flag.data_ptr() if flag is not None else None)
    del torch
    return rc


CASES = [
    ((100, 200, 150, 37), "tanh", 300, 77, "fp32", 1e-4),
    ((784, 100, 10), "sigmoid", 1000, 512, "fp32", 1e-4),
    ((256, 2048, 2048, 10), "relu", 256, 100, "fp32", 1e-4),
    ((100, 200, 150, 37), "sigmoid", 300, 77, "bf16", 2e-2),
]


@pytest.mark.parametrize("case", CASES, ids=["tanh", "digit", "split", "bf16"])
def test_noalloc_matches_hf_hvp(case):
    import torch
    from paper_1606_00511_amd import hf as H
    dims, act, B, B2, prec, tol = case
    p = WL.make_small(dims, act, B, seed=5100 + B)
    net = H.HFNet(dims, act, B, prec=prec)
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    flag = torch.full((1,), 9, dtype=torch.int32, device="cuda")
    for rows in (B, B2):            # two calls in a row, the second smaller
        for mode in ("hessian", "gauss_newton"):
            ref = host(net.hf_hvp(W, X[:rows], y[:rows], v, mode))
            out = torch.full((net.n,), float("nan"), device="cuda")
            rc = noalloc(net, W, X[:rows], y[:rows], v, mode, out, flag)
            assert rc == H.HF_OK, H.lib().hf_last_error(net._h)
            got = host(out)
            err = rel(got, ref)
            print("%s %s rows %d: rel %.2e, identical %s" % (
                case[1], mode, rows, err, np.array_equal(got, ref)), flush=True)
            assert np.isfinite(got).all() and err <= tol
            assert int(host(flag)[0]) == 0
    net.hf_check()
    net.close()


def test_noalloc_shared_scratch_and_label_flag():
    """Two contexts take turns on the one scratch; a bad label sets the flag
    and the next good call clears it; no workspace is needed."""
    import torch
    from paper_1606_00511_amd import hf as H
    a = WL.make_small((100, 200, 150, 37), "tanh", 300, seed=5201)
    b = WL.make_small((64, 96, 10), "sigmoid", 500, seed=5202)
    na = H.HFNet((100, 200, 150, 37), "tanh", 300)
    nb = H.HFNet((64, 96, 10), "sigmoid", 500)
    Wa, Xa, ya, va = dev(a["theta"]), dev(a["X"]), dev(a["y"]), dev(a["v"])
    Wb, Xb, yb, vb = dev(b["theta"]), dev(b["X"]), dev(b["y"]), dev(b["v"])
    ra = host(na.hf_hvp(Wa, Xa, ya, va, "hessian"))
    rb = host(nb.hf_hvp(Wb, Xb, yb, vb, "hessian"))
    oa = torch.empty(na.n, device="cuda")
    ob = torch.empty(nb.n, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert noalloc(na, Wa, Xa, ya, va, "hessian", oa, flag) == H.HF_OK
    first = host(oa)
    assert noalloc(nb, Wb, Xb, yb, vb, "hessian", ob, flag) == H.HF_OK
    assert rel(host(ob), rb) <= 1e-4
    assert noalloc(na, Wa, Xa, ya, va, "hessian", oa, flag) == H.HF_OK
    assert np.array_equal(host(oa), first) and rel(first, ra) <= 1e-4
    ybad = ya.clone()
    ybad[5] = 37                    # outside [0, 37)
    assert noalloc(na, Wa, Xa, ybad, va, "hessian", oa, flag) == H.HF_OK
    assert int(host(flag)[0]) == 1
    assert noalloc(na, Wa, Xa, ya, va, "hessian", oa, flag) == H.HF_OK
    assert int(host(flag)[0]) == 0
    # Gauss-Newton needs no labels; NULL flag is allowed
    assert noalloc(na, Wa, Xa, None, va, "gauss_newton", oa) == H.HF_OK
    assert rel(host(oa), host(na.hf_hvp(Wa, Xa, None, va, "gauss_newton"))) <= 1e-4
    na.close()
    nb.close()


def test_noalloc_rejects_a_batch_beyond_the_scratch():
    """The speech net's layout at 16,384 rows needs far more than the scratch:
    HF_EWORKSPACE before any device work, output untouched."""
    import torch
    from paper_1606_00511_amd import hf as H
    dims = (440, 2048, 2048, 2048, 2048, 1973)
    L = H.lib()
    arr = (ctypes.c_int32 * len(dims))(*dims)
    h = ctypes.c_void_p()
    assert L.hf_create(arr, len(dims), H.HF_SIGMOID, H.HF_FP32, 16384, None,
                       ctypes.byref(h)) == H.HF_OK
    assert L.hf_workspace_bytes(h, 16384) > H.lib().hf_workspace_bytes(h, 1)
    n = L.hf_num_params(h)
    out = torch.full((n,), 7.0, device="cuda")
    W = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    X = torch.zeros((16384, 440), device="cuda")
    y = torch.zeros(16384, dtype=torch.int32, device="cuda")
    rc = L.hf_hvp_noalloc(h, W.data_ptr(), X.data_ptr(), y.data_ptr(), 16384,
                          v.data_ptr(), H.HF_HESSIAN, out.data_ptr(), None)
    assert rc == H.HF_EWORKSPACE
    assert b"scratch" in L.hf_last_error(h)
    assert bool((out == 7.0).all())
    assert L.hf_destroy(h) == H.HF_OK
