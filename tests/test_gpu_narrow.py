"""GPU parity of the narrow-net product (one launch up to the weight
gradients: 4 or 16 batch rows per workgroup, every hidden unit of those rows
in LDS), through the C ABI, against the fp64 oracle.

The kernel serves nets with 2 to 4 weight layers, hidden layers at most 128
wide and at most 64 classes, at batches where the first layer's GEMM would
take 64 x 64 tiles.  It runs inside every cached product there: the CG
solves and the stateless products of such nets.  Bars as for the other
fp32 products: rel-L2 <= 1e-4 (ReLU with the per-unit bracket), CG counts,
the detection iteration and the sign of kappa exact.  Shapes: the widest
admitted layers (128 hidden, 64 classes), widths and batches that are not
multiples of 16 (the kernel's row and column blocks), one row, and 2, 3 and
4 weight layers.  Batches up to 1,024 rows take the layer-1 tiles and the
4-row kernel, larger ones the 16-row kernel; the profiler confirms which
ran.
"""

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests.parity_util import check, relu_margins

pytestmark = pytest.mark.gpu

TOL = 1e-4

CASES = [
    ((784, 100, 10), "sigmoid", 1000),
    ((64, 128, 64), "tanh", 333),
    ((96, 40, 30, 17), "relu", 77),
    ((32, 128, 128, 128, 64), "tanh", 50),
    ((20, 16, 12, 5), "sigmoid", 1),
    ((48, 100, 3), "relu", 130),
    ((64, 100, 10), "sigmoid", 4100),
    ((96, 40, 30, 17), "tanh", 1100),
]
CG_CASES = CASES[:4] + CASES[-2:]


def kernel_for(B):
    return "hf_narrow_product4" if (B + 15) // 16 <= 64 else "hf_narrow_product"


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def sid(c):
    return "%s-%s-b%d" % ("x".join(map(str, c[0])), c[1], c[2])


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", CASES, ids=[sid(c) for c in CASES])
def test_narrow_product(case, mode):
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=6100 + B + len(dims))
    net = HFNet(dims, act, B)
    net.prof_enable(True)
    net.prof_reset()
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    out = host(net.hf_hvp(W, X, y, v, mode))
    stats = net.prof_stats()
    net.prof_enable(False)
    assert kernel_for(B) in stats, sorted(stats)
    # the solve's cache is built by the narrow kernels as well
    assert "hf_narrow_forward4" in stats, sorted(stats)
    ref = O.curvature(dims, act, p["theta"], p["X"], p["y"], p["v"], mode)
    err, bound = check(out, ref, act, lambda k: O.curvature(
        dims, act, p["theta"], p["X"], p["y"], p["v"], mode, kink=k),
        margins=relu_margins(dims, act, p["theta"], p["X"]))
    print("%s %s: rel %.2e (bound %.2e)" % (sid(case), mode, err, bound))
    net.close()


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", CG_CASES, ids=[sid(c) for c in CG_CASES])
def test_narrow_cg(case, mode):
    """CG on the narrow product: counts, detection and kappa's sign exact;
    the lock-step trace compares every product with the oracle's A p_j."""
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=6200 + B)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, X, y)
    g_np = host(g).astype(np.float64)
    cap = 6
    buf = net.set_trace(cap)
    _, _, gi = net.hf_cg(W, X, y, g, 1e-2, cap, mode)
    net.set_trace(0)
    tr = host(buf)
    oi = O.cg_network(dims, act, p["theta"], p["X"], p["y"], g_np, 1e-2, cap, mode)
    print(sid(case), mode, {k: gi[k] for k in ("iters", "products", "neg_curv",
                                               "neg_iter")},
          oi["iters"], oi["products"], oi["neg_iter"])
    assert (gi["iters"], gi["products"], gi["neg_curv"], gi["neg_iter"]) == \
        (oi["iters"], oi["products"], oi["neg_curv"], oi["neg_iter"])
    if oi["neg_curv"]:
        assert np.sign(gi["pBp"]) == np.sign(oi["pBp"])
    margins = relu_margins(dims, act, p["theta"], p["X"])
    for k in range(min(cap, gi["products"])):
        v64 = tr[2 * k].astype(np.float64)
        ref = O.curvature(dims, act, p["theta"], p["X"], p["y"], v64, mode)
        err, bound = check(tr[2 * k + 1], ref, act, lambda kink: O.curvature(
            dims, act, p["theta"], p["X"], p["y"], v64, mode, kink=kink),
            margins=margins)
    net.close()


def test_narrow_not_taken_outside_its_shapes():
    """Wider hidden layers, more classes, one weight layer or a first-layer
    width that is not a multiple of 4 keep the GEMM path."""
    from paper_1606_00511_amd.hf import HFNet
    for dims in ((64, 129, 10), (64, 100, 65), (64, 10), (37, 45, 13)):
        p = WL.make_small(dims, "tanh", 40, seed=6300)
        net = HFNet(dims, "tanh", 40)
        net.prof_enable(True)
        net.prof_reset()
        out = net.hf_hvp(dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"]),
                         "hessian")
        host(out)
        assert not any(k.startswith("hf_narrow_product") for k in net.prof_stats()), dims
        net.prof_enable(False)
        net.close()


@pytest.mark.parametrize("case", CASES, ids=[sid(c) for c in CASES])
def test_narrow_loss_grad(case):
    """The gradient through the narrow kernels (the forward and backward
    pass in two launches, then one GEMM over the concatenated columns)
    against the oracle: loss to 1e-5 relative, gradient rel-L2 <= 1e-4 (ReLU
    with the bracket)."""
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=6500 + B + len(dims))
    net = HFNet(dims, act, B)
    net.prof_enable(True)
    net.prof_reset()
    f, g = net.hf_loss_grad(dev(p["theta"]), dev(p["X"]), dev(p["y"]))
    g = host(g)
    stats = net.prof_stats()
    net.prof_enable(False)
    assert "hf_narrow_forward4" in stats, sorted(stats)
    f_o, g_o = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    assert abs(float(host(f)[0]) - f_o) <= 1e-5 * abs(f_o)
    err, bound = check(g, g_o, act, lambda k: O.loss_grad(
        dims, act, p["theta"], p["X"], p["y"], kink=k)[1],
        margins=relu_margins(dims, act, p["theta"], p["X"]))
    print("%s gradient: rel %.2e (bound %.2e)" % (sid(case), err, bound))
    net.close()


@pytest.mark.parametrize("case", CASES, ids=[sid(c) for c in CASES])
def test_narrow_loss_only(case):
    """The loss-only forward of the line search (hf_loss) through the narrow
    kernels: f within 1e-5 relative of the oracle's, and no forward GEMM."""
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=6600 + B + len(dims))
    net = HFNet(dims, act, B)
    net.prof_enable(True)
    net.prof_reset()
    f = float(host(net.hf_loss(dev(p["theta"]), dev(p["X"]), dev(p["y"])))[0])
    stats = net.prof_stats()
    net.prof_enable(False)
    net.hf_check()
    assert "hf_narrow_forward4" in stats, sorted(stats)
    assert not any(k.startswith("hf_gemm") for k in stats), sorted(stats)
    f_o = O.loss(dims, act, p["theta"], p["X"], p["y"])
    print("%s loss: rel %.2e" % (sid(case), abs(f - f_o) / abs(f_o)))
    assert abs(f - f_o) <= 1e-5 * abs(f_o)
    net.close()


@pytest.mark.parametrize("solver", ["cg", "bicgstab"])
@pytest.mark.parametrize("curvature", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", [((64, 100, 10), "sigmoid", 200),
                                  ((96, 40, 30, 17), "tanh", 77)],
                         ids=["64x100x10-sigmoid-b200", "96x40x30x17-tanh-b77"])
def test_narrow_iterate(case, curvature, solver):
    """One outer iteration (gradient, solve, line search, damping product)
    on a narrow net against the oracle's, with the bar of the other outer
    iteration tests; every pass runs in the narrow kernels (no forward GEMM
    is launched)."""
    from paper_1606_00511_amd.hf import HFNet
    from tests.test_gpu_iterate import compare_step
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=6700 + B)
    th = p["theta"].astype(np.float64)
    kw = dict(solver=solver, curvature=curvature, damping=1e-2, max_iters=6,
              adapt_damping=True)
    o = O.iterate(dims, act, th, p["X"], p["y"], p["X"], p["y"], solver=solver,
                  curvature_kind=curvature, lam=1e-2, max_iters=6,
                  damping_adapt=True)
    net = HFNet(dims, act, B)
    net.prof_enable(True)
    net.prof_reset()
    W = dev(p["theta"].copy())
    delta = dev(np.zeros_like(p["theta"]))
    gi, _, _ = compare_step(net, dims, act, p, th, delta, kw, 0, o, W)
    stats = net.prof_stats()
    net.prof_enable(False)
    print("%s %s %s: dir %d alpha %g evals %d f %.6f -> %.6f (oracle %.6f) rho "
          "%.4f/%.4f" % (sid(case), curvature, solver, gi["direction"], gi["alpha"],
                         gi["evals"], gi["f0"], gi["f1"], o["f1"], gi["rho"],
                         o["rho"]))
    assert stats["hf_narrow_forward4"]["launches"] >= gi["evals"] + 2, stats
    assert not any(k.startswith("hf_gemm_fwd") or k.startswith("hf_softmax")
                   for k in stats), sorted(stats)
    # (Bi-CG-STAB's step can move by its rounding sensitivity, which
    # compare_step allows for; rho is compared for CG)
    if solver == "cg" and gi["accepted"] and o["accepted"] and \
            gi["alpha"] == o["alpha"] and gi["direction"] == o["direction"]:
        assert gi["rho"] == pytest.approx(o["rho"], rel=1e-2)
        if min(abs(o["rho"] - 0.25), abs(o["rho"] - 0.75)) > 1e-2:
            assert gi["damping_next"] == pytest.approx(o["lam_next"], rel=1e-6)
    net.close()


def test_narrow_bad_label_is_reported():
    """The narrow cache build checks the labels of a Hessian product or
    solve as the softmax row kernel does: a label outside [0, C) is
    reported (HF_ELABEL) and the flag is cleared once read."""
    from paper_1606_00511_amd.hf import HFNet, HFError, HF_ELABEL
    dims, act, B = (64, 100, 10), "tanh", 200
    p = WL.make_small(dims, act, B, seed=6400)
    y = p["y"].copy()
    y[7] = 10
    net = HFNet(dims, act, B)
    W, X, v = dev(p["theta"]), dev(p["X"]), dev(p["v"])
    net.prof_enable(True)
    net.prof_reset()
    host(net.hf_hvp(W, X, dev(y), v, "hessian"))
    assert "hf_narrow_forward4" in net.prof_stats()
    net.prof_enable(False)
    with pytest.raises(HFError) as ei:
        net.hf_check()
    assert ei.value.code == HF_ELABEL
    net.hf_check()
    _, g = net.hf_loss_grad(W, X, dev(p["y"]))
    with pytest.raises(HFError) as ei:
        net.hf_cg(W, X, dev(y), g, 1e-2, 3, "hessian")
    assert ei.value.code == HF_ELABEL
    net.hf_check()
    # a Gauss-Newton solve reads no labels
    net.hf_cg(W, X, dev(y), g, 1e-2, 3, "gauss_newton")
    net.hf_check()
    # the loss-only forward checks them
    host(net.hf_loss(W, X, dev(y)))
    with pytest.raises(HFError) as ei:
        net.hf_check()
    assert ei.value.code == HF_ELABEL
    net.hf_check()
    net.close()
