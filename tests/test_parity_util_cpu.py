"""CPU checks of the ReLU bracket used by the GPU parity tests
(tests/parity_util.py): the oracle's per-unit step positions reduce to the
scalar ones, and the per-unit margins cover the rounding of an fp32 forward
pass computed on the CPU."""

import numpy as np

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests import parity_util as PU


def test_per_unit_kink_reduces_to_the_scalar_kink():
    dims, act = (9, 7, 6, 5), "relu"
    p = WL.make_small(dims, act, 23, seed=61, x_dist="normal", bias_std=0.5)
    th = p["theta"].astype(np.float64)
    Z, _ = O.forward(dims, act, th, p["X"])
    for kink in (0.0, 0.3, -0.2):
        arrs = [np.full_like(z, kink) for z in Z[:-1]]
        for mode in ("hessian", "gauss_newton"):
            a = O.curvature(dims, act, th, p["X"], p["y"], p["v"], mode, kink=kink)
            b = O.curvature(dims, act, th, p["X"], p["y"], p["v"], mode, kink=arrs)
            assert np.array_equal(a, b)
        assert np.array_equal(O.loss_grad(dims, act, th, p["X"], p["y"], kink=kink)[1],
                              O.loss_grad(dims, act, th, p["X"], p["y"], kink=arrs)[1])
        assert np.array_equal(O.fisher_diag(dims, act, th, p["X"], p["y"], kink=kink),
                              O.fisher_diag(dims, act, th, p["X"], p["y"], kink=arrs))


def test_per_unit_kink_moves_only_its_unit():
    """Flipping one unit's step changes the product, and flipping it back by
    a kink on the other side of its z restores the kink-0 result."""
    dims, act = (9, 7, 6, 5), "relu"
    p = WL.make_small(dims, act, 23, seed=62, x_dist="normal", bias_std=0.5)
    th = p["theta"].astype(np.float64)
    Z, _ = O.forward(dims, act, th, p["X"])
    base = O.curvature(dims, act, th, p["X"], p["y"], p["v"], "hessian")
    arrs = [np.zeros_like(z) for z in Z[:-1]]
    i, j = 3, 2
    z = Z[0][i, j]
    arrs[0][i, j] = z + 1.0 if z > 0 else z - 1.0     # flips this unit only
    moved = O.curvature(dims, act, th, p["X"], p["y"], p["v"], "hessian", kink=arrs)
    assert not np.allclose(moved, base)
    arrs[0][i, j] = z - 1e-3 if z > 0 else z + 1e-3   # same side as kink 0
    back = O.curvature(dims, act, th, p["X"], p["y"], p["v"], "hessian", kink=arrs)
    assert np.array_equal(back, base)


def test_margins_cover_an_fp32_forward_pass():
    """An fp32 forward pass (NumPy's float32 GEMM, another accumulation order
    than the GPU's) stays inside the margins with room to spare: its largest
    error is below a third of the 8-sigma margin of its unit."""
    dims, act = (784, 500, 500, 500, 10), "relu"
    p = WL.make_small(dims, act, 2000, seed=63)
    th = p["theta"]
    margins = PU.relu_margins(dims, act, th, p["X"])
    Z, _ = O.forward(dims, act, th.astype(np.float64), p["X"])
    layers = O.unpack(th, dims)     # the fp32 parameters
    a = p["X"].astype(np.float32)
    worst = 0.0
    for l, (W, b) in enumerate(layers[:-1]):
        z32 = a @ W.astype(np.float32).T + b.astype(np.float32)
        err = np.abs(z32.astype(np.float64) - Z[l])
        worst = max(worst, float((err / margins[l]).max()))
        a = np.maximum(z32, np.float32(0))
    assert worst < 1.0 / 3.0, worst
    assert PU.relu_margins(dims, "tanh", th, p["X"]) is None


def test_ambiguous_units_are_few():
    """At the ReLU digit workload's curvature batch the bracket holds a
    few dozen units per layer (the fixed margin of 2e-5 held 69 to 156)."""
    w = WL.WORKLOADS["mnist_784_500x3_10_relu_b60000_c6000"]
    inp = WL.make(w, rows=w.curv_batch)
    m = PU.relu_margins(w.dims, w.act, inp["theta"], inp["X"])
    n = PU.ambiguous_units(w.dims, w.act, inp["theta"], inp["X"], m)
    assert 0 < n < 3 * 60, n
