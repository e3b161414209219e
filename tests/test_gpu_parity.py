"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded float32 inputs.

Bar: relative L2 error <= 1e-4 for the loss, the gradient, H v and G v
(fp32 path); for CG, identical iteration and product counts and identical
negative-curvature decisions.  Shapes span several 128 x 128 tiles with
ragged tails, unaligned widths (scalar-load path), a single row, and both
output widths of the workloads (10 and 1,973 classes).
"""

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests.parity_util import check, relu_margins

pytestmark = pytest.mark.gpu

TOL = 1e-4


def torch_mod():
    import torch
    return torch


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def dev(a, dtype=None):
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to("cuda")


def host(t):
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def net(dims, act, max_batch):
    from paper_1606_00511_amd.hf import HFNet
    return HFNet(dims, act, max_batch)


SMALL = [
    # dims, act, batch: several tiles + ragged tails, aligned widths
    ((100, 200, 150, 37), "sigmoid", 300),
    ((100, 200, 150, 37), "tanh", 300),
    ((100, 200, 150, 37), "relu", 300),
    # unaligned widths -> scalar global loads everywhere
    ((37, 45, 13), "tanh", 130),
    ((37, 45, 13), "sigmoid", 1),
    # one weight layer (no hidden layer)
    ((64, 10), "sigmoid", 257),
    # digit-image shaped net at its full batch
    ((784, 100, 10), "sigmoid", 1000),
    # wide output layer, like the speech workload
    ((40, 96, 1973), "sigmoid", 200),
    # enough rows for the 256 x 256 tiles, with ragged tile edges ...
    ((64, 1100, 10), "tanh", 15000),
    # ... and with unaligned widths (scalar global loads)
    ((63, 1101, 10), "sigmoid", 15000),
    # few rows through wide layers: the batch-row GEMMs have too few tiles
    # and run as split-K partials plus a reduce that applies the epilogue
    ((256, 2048, 2048, 10), "tanh", 256),
    ((250, 2049, 1999, 13), "relu", 200),
]


def ids(c):
    return "%s-%s-b%d" % ("x".join(map(str, c[0])), c[1], c[2])


@pytest.mark.parametrize("case", SMALL, ids=[ids(c) for c in SMALL])
def test_loss_grad(case):
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=101 + B)
    f_o, g_o = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    h = net(dims, act, B)
    loss, grad = h.hf_loss_grad(dev(p["theta"]), dev(p["X"]), dev(p["y"]))
    h.hf_check()
    assert abs(float(host(loss)[0]) - f_o) <= TOL * abs(f_o)
    check(host(grad), g_o, act, lambda k: O.loss_grad(
        dims, act, p["theta"], p["X"], p["y"], kink=k)[1],
        margins=relu_margins(dims, act, p["theta"], p["X"]))


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", SMALL, ids=[ids(c) for c in SMALL])
def test_curvature_product(case, mode):
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=202 + B)
    ref = O.curvature(dims, act, p["theta"], p["X"], p["y"], p["v"], mode)
    h = net(dims, act, B)
    out = h.hf_hvp(dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"]), mode)
    check(host(out), ref, act, lambda k: O.curvature(
        dims, act, p["theta"], p["X"], p["y"], p["v"], mode, kink=k),
        margins=relu_margins(dims, act, p["theta"], p["X"]))


def test_gauss_newton_ignores_labels_and_is_deterministic():
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=7)
    h = net(dims, act, B)
    W, X, v = dev(p["theta"]), dev(p["X"]), dev(p["v"])
    a = host(h.hf_hvp(W, X, dev(p["y"]), v, "gauss_newton"))
    b = host(h.hf_hvp(W, X, dev(p["y"][::-1].copy()), v, "gauss_newton"))
    c = host(h.hf_hvp(W, X, None, v, "gauss_newton"))
    assert np.array_equal(a, b) and np.array_equal(a, c)
    h1 = host(h.hf_hvp(W, X, dev(p["y"]), v, "hessian"))
    h2 = host(h.hf_hvp(W, X, dev(p["y"]), v, "hessian"))
    assert np.array_equal(h1, h2)


def test_bad_label_is_reported():
    from paper_1606_00511_amd.hf import HFError, HF_ELABEL
    dims, act, B = (16, 8, 5), "sigmoid", 12
    p = WL.make_small(dims, act, B, seed=3)
    y = p["y"].copy()
    y[4] = 5
    h = net(dims, act, B)
    h.hf_loss_grad(dev(p["theta"]), dev(p["X"]), dev(y))
    with pytest.raises(HFError) as ei:
        h.hf_check()
    assert ei.value.code == HF_ELABEL
    h.hf_check()   # flag cleared


def gpu_cg(dims, act, p, g, lam, iters, mode, Bc=None, rel_tol=0.0):
    Xc = p["X"] if Bc is None else p["X"][:Bc]
    yc = p["y"] if Bc is None else p["y"][:Bc]
    h = net(dims, act, max(p["X"].shape[0], Xc.shape[0]))
    step, nd, info = h.hf_cg(dev(p["theta"]), dev(Xc), dev(yc),
                             dev(g.astype(np.float32)), lam, iters, mode,
                             rel_tol=rel_tol)
    return host(step), host(nd), info


def oracle_cg(dims, act, p, g, lam, iters, mode, Bc=None, rel_tol=0.0):
    Xc = p["X"] if Bc is None else p["X"][:Bc]
    yc = p["y"] if Bc is None else p["y"][:Bc]
    return O.cg_network(dims, act, p["theta"], Xc, yc,
                        g.astype(np.float32).astype(np.float64), lam, iters,
                        mode, rel_tol=rel_tol, record=True)


def assert_cg_parity(gi, oi):
    assert gi["iters"] == oi["iters"]
    assert gi["products"] == oi["products"]
    assert gi["neg_curv"] == oi["neg_curv"]
    assert gi["neg_iter"] == oi["neg_iter"]
    if oi["neg_curv"]:
        assert np.sign(gi["pBp"]) == np.sign(oi["pBp"])
        assert gi["gTd"] <= 0.0


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", [((784, 100, 10), "sigmoid", 1000, 10),
                                  ((100, 200, 150, 37), "tanh", 300, 12),
                                  ((100, 200, 150, 37), "relu", 300, 12),
                                  ((256, 2048, 2048, 10), "tanh", 256, 6)],
                         ids=["digit-784-100-10", "tanh-ragged", "relu-ragged",
                              "split-k-rows"])
def test_cg_counts_and_signs(case, mode):
    dims, act, B, iters = case
    p = WL.make_small(dims, act, B, seed=303, bias_std=0.0)
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    lam = 1e-2
    step, nd, gi = gpu_cg(dims, act, p, g, lam, iters, mode)
    oi = oracle_cg(dims, act, p, g, lam, iters, mode)
    assert_cg_parity(gi, oi)
    assert gi["rr0"] == pytest.approx(oi["rr0"], rel=1e-5)
    if oi["neg_curv"]:
        # the returned direction is the oracle's oriented direction
        assert rel(nd, oi["neg_dir"]) <= 1e-3
        assert gi["pBp"] == pytest.approx(oi["pBp"], rel=1e-3)
        if oi["neg_iter"] == 0:
            assert np.array_equal(step, -g.astype(np.float32))
    else:
        assert not np.any(nd)
    if oi["iters"] <= 3:
        assert rel(step, oi["step"]) <= 1e-3


def test_cg_damped_single_layer_reaches_exact_solution():
    """L = 1: B = G + lambda I is SPD and formable; n CG steps solve it."""
    dims, act = (3, 3), "sigmoid"
    p = WL.make_small(dims, act, 10, seed=4, x_dist="normal")
    th = p["theta"].astype(np.float64)
    n = th.size
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    g32 = g.astype(np.float32)
    G = np.stack([O.gvp(dims, act, th, p["X"], e) for e in np.eye(n)], axis=1)
    lam = 0.05
    x = np.linalg.solve(G + lam * np.eye(n), -g32.astype(np.float64))
    for mode in ("gauss_newton", "hessian"):
        step, nd, gi = gpu_cg(dims, act, p, g32, lam, n + 4, mode)
        assert gi["neg_curv"] == 0 and gi["iters"] == n + 4
        assert rel(step, x) <= 1e-4


def test_cg_edge_cases():
    dims, act = (37, 45, 13), "tanh"
    p = WL.make_small(dims, act, 50, seed=9)
    n = WL.num_params(dims)
    # zero gradient: nothing to do
    step, nd, gi = gpu_cg(dims, act, p, np.zeros(n), 0.01, 5, "hessian")
    assert gi["iters"] == 0 and gi["products"] == 0 and not np.any(step)
    # zero budget
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    step, nd, gi = gpu_cg(dims, act, p, g, 0.01, 0, "gauss_newton")
    assert gi["iters"] == 0 and gi["products"] == 0 and not np.any(step)
    assert gi["rr0"] == pytest.approx(float(g.astype(np.float32) @ g.astype(np.float32)), rel=1e-6)
    # relative tolerance stops early on the PSD path
    oi = oracle_cg(dims, act, p, g, 1.0, 200, "gauss_newton", rel_tol=1e-2)
    step, nd, gi = gpu_cg(dims, act, p, g, 1.0, 200, "gauss_newton", rel_tol=1e-2)
    assert gi["iters"] == oi["iters"] < 200
    # repeated solves are bit-identical
    s1, n1, i1 = gpu_cg(dims, act, p, g, 0.01, 8, "hessian")
    s2, n2, i2 = gpu_cg(dims, act, p, g, 0.01, 8, "hessian")
    assert np.array_equal(s1, s2) and np.array_equal(n1, n2) and i1 == i2


def test_shard_average_on_gpu():
    """A product on a batch equals the row-weighted mean of the products on
    its shards (the data-parallel reduce of Alg. 2 with equal shares)."""
    dims, act, B = (100, 200, 150, 37), "sigmoid", 512
    p = WL.make_small(dims, act, B, seed=55)
    h = net(dims, act, B)
    W, v = dev(p["theta"]), dev(p["v"])
    for mode in ("hessian", "gauss_newton"):
        full = host(h.hf_hvp(W, dev(p["X"]), dev(p["y"]), v, mode)).astype(np.float64)
        acc = np.zeros_like(full)
        for s, e in ((0, 128), (128, 300), (300, 512)):
            part = h.hf_hvp(W, dev(p["X"][s:e]), dev(p["y"][s:e]), v, mode)
            acc += (e - s) / B * host(part)
        assert rel(acc, full) <= 1e-5
