"""GPU parity of Bi-CG-STAB (Alg. 3) with oriented negative-curvature
candidates (Sec. 2.2), through the C ABI, against the fp64 oracle.

Bar: identical iteration and product counts, identical first
negative-curvature iteration and sign of its curvature; exact solution of a
damped single-layer (SPD) system.  The returned candidate is checked on
its own: the oracle recomputes d~^T H d~ and g^T d~ for the GPU's vector.
The iterate and the candidate must agree with the oracle's within 1e-3
relative L2 plus a term for the conditioning of the recurrences: on an
indefinite Hessian, Bi-CG-STAB can pass close to a breakdown ((r, r0*) or
(A p, r0*) near 0 while r is not), where the rounding of the stored vectors
to float32 is amplified by orders of magnitude.  The test measures that
amplification with the oracle itself, rerun with every stored vector
rounded to float32 and with its products perturbed by a seeded relative
noise of 1e-7, and allows 10 times the resulting deviation.
"""

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL

pytestmark = pytest.mark.gpu


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def run(dims, act, p, g, lam, iters, mode, rows=None, rel_tol=0.0):
    import torch
    from paper_1606_00511_amd.hf import HFNet
    X = p["X"] if rows is None else p["X"][:rows]
    y = p["y"] if rows is None else p["y"][:rows]
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    h = HFNet(dims, act, X.shape[0])
    step, nd, info = h.hf_bicgstab(d(p["theta"]), d(X), d(y),
                                   d(g.astype(np.float32)), lam, iters, mode,
                                   rel_tol=rel_tol)
    torch.cuda.synchronize()
    g64 = g.astype(np.float32).astype(np.float64)
    oi = O.bicgstab_network(dims, act, p["theta"], X, y, g64, lam, iters, mode,
                            rel_tol=rel_tol)
    rng = np.random.default_rng(12345)
    f32 = lambda v: v.astype(np.float32).astype(np.float64)

    def noisy(v):
        w = O.curvature(dims, act, p["theta"], X, y, v, mode)
        return w * (1.0 + 1e-7 * rng.standard_normal(w.size))
    on = O.bicgstab_minimize(noisy, g64, lam, iters, rel_tol, store=f32)
    oi["sensitivity"] = rel(on["step"], oi["step"]) if iters else 0.0
    nd = nd.cpu().numpy()
    if info["neg_curv"]:
        d64 = nd.astype(np.float64)
        oi["gpu_dHd"] = float(d64 @ O.curvature(dims, act, p["theta"], X, y,
                                                d64, "hessian"))
        oi["gpu_gTd"] = float(g64 @ d64)
    return step.cpu().numpy(), nd, info, oi


def check(step, nd, gi, oi, tol=1e-3):
    tol = tol + 10.0 * oi["sensitivity"]
    print("step rel %.3e, bound %.3e (oracle sensitivity %.2e)" % (
        rel(step, oi["step"]), tol, oi["sensitivity"]))
    assert gi["iters"] == oi["iters"]
    assert gi["products"] == oi["products"]
    assert gi["neg_curv"] == oi["neg_curv"]
    assert gi["neg_iter"] == oi["neg_iter"]
    assert rel(step, oi["step"]) <= tol
    if oi["neg_curv"]:
        assert gi["pHp"] < 0 and gi["gTd"] < 0
        # the candidate itself: its curvature and slope, recomputed in fp64
        assert oi["gpu_dHd"] < 0 and oi["gpu_gTd"] < 0
        assert gi["pHp"] == pytest.approx(oi["gpu_dHd"], rel=1e-3)
        assert gi["gTd"] == pytest.approx(oi["gpu_gTd"], rel=1e-3)
        assert rel(nd, oi["neg_dir"]) <= tol
    else:
        assert not np.any(nd)


CASES = [((784, 100, 10), "sigmoid", 1000, 4),
         ((100, 200, 150, 37), "tanh", 300, 4),
         ((100, 200, 150, 37), "relu", 300, 4),
         ((37, 45, 13), "tanh", 130, 3)]


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-%s" % (
    "x".join(map(str, c[0])), c[1]))
def test_bicgstab_parity(case, mode):
    dims, act, B, iters = case
    p = WL.make_small(dims, act, B, seed=404, bias_std=0.0)
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    step, nd, gi, oi = run(dims, act, p, g, 1e-2, iters, mode)
    print(mode, dims, act, {k: gi[k] for k in ("iters", "products", "neg_curv",
                                               "neg_iter", "pHp")},
          "oracle", oi["iters"], oi["products"], oi["neg_iter"], oi["dHd"])
    check(step, nd, gi, oi)


def test_bicgstab_damped_single_layer_is_exact():
    dims, act = (3, 3), "sigmoid"
    p = WL.make_small(dims, act, 10, seed=4, x_dist="normal")
    th = p["theta"].astype(np.float64)
    n = th.size
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    g32 = g.astype(np.float32)
    G = np.stack([O.gvp(dims, act, th, p["X"], e) for e in np.eye(n)], axis=1)
    lam = 0.05
    x = np.linalg.solve(G + lam * np.eye(n), -g32.astype(np.float64))
    # (iteration counts are not compared here: the relative-residual stop
    # sits near the fp32 rounding floor of the residual)
    step, nd, gi, oi = run(dims, act, p, g32, lam, 3 * n, "gauss_newton",
                           rel_tol=1e-6)
    assert rel(step, x) <= 1e-4
    assert gi["neg_curv"] == 0


def test_bicgstab_edge_cases():
    dims, act = (37, 45, 13), "tanh"
    p = WL.make_small(dims, act, 50, seed=9)
    n = WL.num_params(dims)
    step, nd, gi, oi = run(dims, act, p, np.zeros(n), 0.01, 5, "hessian")
    assert gi["iters"] == 0 and gi["products"] == 0 and not np.any(step)
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    step, nd, gi, oi = run(dims, act, p, g, 0.01, 0, "hessian")
    assert gi["iters"] == 0 and gi["products"] == 0 and not np.any(step)


@pytest.mark.parametrize("name,iters", [
    ("mnist_784_500x3_10_tanh_b10000", 4),
    ("speech_440_2048x4_1973_sigmoid_b4096_c1024", 3),
    ("speech_440_2048x4_1973_sigmoid_b4096_c1024", 1)])
def test_bicgstab_full_size(name, iters):
    w = WL.WORKLOADS[name]
    inp = WL.make(w)
    p = dict(X=inp["X"], y=inp["y"], theta=inp["theta"])
    _, g = O.loss_grad(w.dims, w.act, inp["theta"], inp["X"][:w.curv_batch],
                       inp["y"][:w.curv_batch])
    step, nd, gi, oi = run(w.dims, w.act, p, g, w.damping, iters, "hessian",
                           rows=w.curv_batch)
    print(name, gi, "oracle", oi["iters"], oi["neg_iter"], oi["dHd"])
    check(step, nd, gi, oi)
