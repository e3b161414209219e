"""Edge cases of the C ABI on the GPU: arguments that must be rejected before
anything is launched, and parity at the largest shapes hf_create accepts
(HF_MAX_CLASSES output classes, HF_MAX_LAYERS weight layers).

Rejections: an empty batch (the batch-mean objective of Sec. 2.1 is not
defined for zero rows), a negative batch, a batch above max_batch, a pointer
that is not 16-byte aligned and a NULL operand all return HF_EINVAL, set a
message, and leave every output untouched.

Parity bar as in the other GPU tests: rel-L2 <= 1e-4 (fp32) and <= 2e-2
(bf16 GEMM operands) against the fp64 oracle on the same seeded inputs.
"""

import ctypes

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests.parity_util import check, rel, relu_margins

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def test_rejected_arguments_leave_outputs_untouched():
    import torch
    from paper_1606_00511_amd import hf as H
    dims, act, B = (37, 45, 13), "sigmoid", 20
    p = WL.make_small(dims, act, B, seed=4)
    h = H.HFNet(dims, act, B)
    L = H.lib()
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    n = h.n
    loss = torch.full((1,), 7.0, device="cuda")
    grad = torch.full((n,), 7.0, device="cuda")
    out = torch.full((n,), 7.0, device="cuda")
    step = torch.full((n,), 7.0, device="cuda")
    nd = torch.full((n,), 7.0, device="cuda")
    info = H.hf_cg_info()
    w, x, yy, vv = W.data_ptr(), X.data_ptr(), y.data_ptr(), v.data_ptr()

    def expect(rc, words):
        assert rc == H.HF_EINVAL
        msg = L.hf_last_error(h._h).decode()
        assert any(wd in msg for wd in words), msg

    for bad in (0, -1, B + 1):
        expect(L.hf_loss_grad(h._h, w, x, yy, bad, loss.data_ptr(), grad.data_ptr()),
               ["batch"])
        expect(L.hf_loss(h._h, w, x, yy, bad, loss.data_ptr()), ["batch"])
        expect(L.hf_hvp(h._h, w, x, yy, bad, vv, H.HF_HESSIAN, out.data_ptr()),
               ["batch"])
        expect(L.hf_cg(h._h, w, x, yy, bad, grad.data_ptr(), 0.01, 5, 0.0,
                       H.HF_GAUSS_NEWTON, step.data_ptr(), nd.data_ptr(),
                       ctypes.byref(info)), ["batch"])
        expect(L.hf_bicgstab(h._h, w, x, yy, bad, grad.data_ptr(), 0.01, 5, 0.0,
                             H.HF_GAUSS_NEWTON, step.data_ptr(), nd.data_ptr(),
                             ctypes.byref(info)), ["batch"])
    expect(L.hf_loss_grad(h._h, w, x + 4, yy, B, loss.data_ptr(), grad.data_ptr()),
           ["aligned"])
    expect(L.hf_hvp(h._h, w, x, yy, B, vv + 8, H.HF_HESSIAN, out.data_ptr()),
           ["aligned"])
    expect(L.hf_loss_grad(h._h, None, x, yy, B, loss.data_ptr(), grad.data_ptr()),
           ["NULL"])
    expect(L.hf_hvp(h._h, w, x, None, B, vv, H.HF_HESSIAN, out.data_ptr()),
           ["NULL", "label"])
    h.hf_check()
    for t in (loss, grad, out, step, nd):
        assert bool((t == 7.0).all())
    # the context still works after the rejections
    f, g = h.hf_loss_grad(W, X, y)
    f_o, g_o = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    assert abs(float(host(f)[0]) - f_o) <= 1e-4 * abs(f_o)
    assert rel(host(g), g_o) <= 1e-4


MAXC = [((40, 64, 4096), "tanh", 150, "fp32", 1e-4),
        ((40, 64, 4096), "sigmoid", 150, "bf16", 2e-2)]


@pytest.mark.parametrize("case", MAXC, ids=["fp32", "bf16"])
def test_max_classes(case):
    """4,096 classes: the softmax rows (16 KB each) fill the row kernels'
    LDS allowance."""
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B, prec, tol = case
    p = WL.make_small(dims, act, B, seed=77)
    h = HFNet(dims, act, B, prec=prec)
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    f, g = h.hf_loss_grad(W, X, y)
    f_o, g_o = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    assert abs(float(host(f)[0]) - f_o) <= tol * abs(f_o)
    check(host(g), g_o, act, tol=tol)
    for mode in ("hessian", "gauss_newton"):
        out = h.hf_hvp(W, X, y, v, mode)
        ref = O.curvature(dims, act, p["theta"], p["X"], p["y"], p["v"], mode)
        err, _ = check(host(out), ref, act, tol=tol)
        print("%s %s rel %.2e" % (prec, mode, err))
    h.hf_check()


@pytest.mark.parametrize("act", ["sigmoid", "tanh", "relu"])
def test_max_layers(act):
    """16 weight layers (the most hf_create accepts): loss, gradient, Hv, Gv
    and a CG solve's counts and signs."""
    from paper_1606_00511_amd.hf import HFNet
    dims = (24,) + (20,) * 15 + (7,)
    assert len(dims) - 1 == 16
    B = 90
    p = WL.make_small(dims, act, B, seed=16)
    h = HFNet(dims, act, B)
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    f, g = h.hf_loss_grad(W, X, y)
    f_o, g_o = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    assert abs(float(host(f)[0]) - f_o) <= 1e-4 * abs(f_o)
    mg = relu_margins(dims, act, p["theta"], p["X"])
    check(host(g), g_o, act, lambda k: O.loss_grad(dims, act, p["theta"], p["X"],
                                                    p["y"], kink=k)[1], margins=mg)
    for mode in ("hessian", "gauss_newton"):
        out = h.hf_hvp(W, X, y, v, mode)
        ref = O.curvature(dims, act, p["theta"], p["X"], p["y"], p["v"], mode)
        check(host(out), ref, act, lambda k: O.curvature(
            dims, act, p["theta"], p["X"], p["y"], p["v"], mode, kink=k),
            margins=mg)
    g32 = g_o.astype(np.float32)
    for mode in ("hessian", "gauss_newton"):
        _, _, gi = h.hf_cg(W, X, y, dev(g32), 1e-2, 6, mode)
        oi = O.cg_network(dims, act, p["theta"], p["X"], p["y"],
                          g32.astype(np.float64), 1e-2, 6, mode)
        assert (gi["iters"], gi["products"], gi["neg_curv"], gi["neg_iter"]) == \
            (oi["iters"], oi["products"], oi["neg_curv"], oi["neg_iter"])
        if oi["neg_curv"]:
            assert np.sign(gi["pBp"]) == np.sign(oi["pBp"])


@pytest.mark.parametrize("solver", ["hf_cg", "hf_bicgstab"])
def test_non_finite_scalars_are_reported(solver):
    """A NaN in g makes |g|^2 non-finite: the solve stops before its first
    product and returns HF_ENUMERIC with info.status set.  An Inf weight
    makes the first product, hence p^T B p, non-finite: the solve stops
    after that product with HF_ENUMERIC.  These are numeric outcomes, not
    faults; the context then solves a clean system as before."""
    from paper_1606_00511_amd import hf as H
    dims, act, B = (37, 45, 13), "tanh", 40
    p = WL.make_small(dims, act, B, seed=5)
    h = H.HFNet(dims, act, B)
    L = H.lib()
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = h.hf_loss_grad(W, X, y)
    ref_step, _, ref_info = getattr(h, solver)(W, X, y, g, 1e-2, 4, "gauss_newton")
    ref_step = host(ref_step)
    step, nd = g.clone(), g.clone()

    def call(Wt, gt):
        info = H.hf_cg_info()
        rc = getattr(L, solver)(h._h, Wt.data_ptr(), X.data_ptr(), y.data_ptr(), B,
                                gt.data_ptr(), 1e-2, 4, 0.0, H.HF_GAUSS_NEWTON,
                                step.data_ptr(), nd.data_ptr(), ctypes.byref(info))
        return rc, info

    g_nan = g.clone()
    g_nan[7] = float("nan")
    rc, info = call(W, g_nan)
    assert rc == H.HF_ENUMERIC and info.status == H.HF_ENUMERIC
    assert info.products == 0 and info.iters == 0
    assert b"non-finite" in L.hf_last_error(h._h)
    W_inf = W.clone()
    W_inf[h.n - 20] = float("inf")     # a weight of the output layer
    rc, info = call(W_inf, g)
    assert rc == H.HF_ENUMERIC and info.status == H.HF_ENUMERIC
    assert info.products >= 1 and info.iters == 0
    s2, _, i2 = getattr(h, solver)(W, X, y, g, 1e-2, 4, "gauss_newton")
    assert i2 == ref_info
    assert np.array_equal(host(s2), ref_step)


def test_workspace_for_fewer_rows():
    """A workspace laid out for b < max_batch rows serves calls up to b rows
    with the results of a full-size one, and rejects more rows with
    HF_EWORKSPACE, leaving the output untouched."""
    import torch
    from paper_1606_00511_amd import hf as H
    dims, act, B = (100, 200, 150, 37), "sigmoid", 300
    p = WL.make_small(dims, act, B, seed=6)
    full = H.HFNet(dims, act, B)
    part = H.HFNet(dims, act, B, ws_batch=120)
    assert part.workspace.numel() < full.workspace.numel()
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    for mode in ("hessian", "gauss_newton"):
        a = host(full.hf_hvp(W, X[:120], y[:120], v, mode))
        b = host(part.hf_hvp(W, X[:120], y[:120], v, mode))
        assert np.array_equal(a, b)
    out = torch.full((part.n,), 7.0, device="cuda")
    with pytest.raises(H.HFError) as e:
        part.hf_hvp(W, X[:121], y[:121], v, "hessian", out=out)
    assert e.value.code == H.HF_EWORKSPACE
    assert bool((out == 7.0).all())
    f1, g1 = full.hf_loss_grad(W, X[:120], y[:120])
    f2, g2 = part.hf_loss_grad(W, X[:120], y[:120])
    assert np.array_equal(host(g1), host(g2)) and float(host(f1)[0]) == float(host(f2)[0])
