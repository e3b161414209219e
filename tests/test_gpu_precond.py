"""GPU parity of Martens' diagonal preconditioner (Sec. 2.1 lists it among
the modifications of HF): the squared per-example gradient F
(hf_fisher_diag), preconditioned CG (hf_pcg) and the preconditioned outer
iteration with either solver, against the fp64 oracle on the same seeded
inputs; preconditioned Bi-CG-STAB (hf_pbicgstab) has its own tests beside
the unpreconditioned ones.

Bars: F within rel-L2 1e-4 (a sum of non-negative terms, no cancellation),
2e-2 with bf16 GEMM operands; PCG with identical iterations, products,
detections and sign of the detected curvature, and on a damped
single-layer net the exact solve within 1e-4; the outer iteration with the
bar of the other iteration tests.
At the speech net's full size, where per-example backpropagation in fp64 is
out of reach, the output layer's blocks of F are checked against their
forward-only closed form, and every block against F >= g^2.
"""

import gc

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


def net(dims, act, B, prec="fp32"):
    from paper_1606_00511_amd.hf import HFNet
    return HFNet(dims, act, B, prec=prec)


CASES = [((100, 200, 150, 37), "tanh", 300),
         ((100, 200, 150, 37), "relu", 300),
         ((37, 45, 13), "sigmoid", 130),
         ((40, 96, 1973), "sigmoid", 200),
         ((64, 1100, 10), "tanh", 300)]


@pytest.mark.parametrize("case", CASES, ids=["x".join(map(str, c[0])) + "-" + c[1]
                                             for c in CASES])
def test_fisher_diag(case):
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=41 + B)
    h = net(dims, act, B)
    F = host(h.hf_fisher_diag(dev(p["theta"]), dev(p["X"]), dev(p["y"])))
    h.hf_check()
    ref = O.fisher_diag(dims, act, p["theta"], p["X"], p["y"])
    err, bound = check(F, ref, act, lambda k: O.fisher_diag(
        dims, act, p["theta"], p["X"], p["y"], kink=k),
        margins=relu_margins(dims, act, p["theta"], p["X"]))
    print("F rel %.2e (bound %.2e)" % (err, bound))
    assert np.all(F >= 0.0)


def pcg_pair(dims, act, p, g, minv, lam, iters, mode, rel_tol=0.0):
    h = net(dims, act, p["X"].shape[0])
    step, nd, gi = h.hf_pcg(dev(p["theta"]), dev(p["X"]), dev(p["y"]),
                            dev(g.astype(np.float32)), dev(minv.astype(np.float32)),
                            lam, iters, mode, rel_tol=rel_tol)
    oi = O.cg_network(dims, act, p["theta"], p["X"], p["y"],
                      g.astype(np.float32).astype(np.float64), lam, iters, mode,
                      rel_tol, minv=minv.astype(np.float32).astype(np.float64))
    return host(step), host(nd), gi, oi


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("act", ["sigmoid", "tanh"])
def test_pcg_counts_and_signs(act, mode):
    dims, B = (100, 200, 150, 37), 300
    p = WL.make_small(dims, act, B, seed=43)
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    lam = 1e-2
    minv = O.precond_inverse(O.fisher_diag(dims, act, p["theta"], p["X"], p["y"]),
                             lam)
    step, nd, gi, oi = pcg_pair(dims, act, p, g, minv, lam, 8, mode)
    print(act, mode, {k: gi[k] for k in ("iters", "products", "neg_curv",
                                         "neg_iter", "pBp")}, oi["pBp"])
    assert (gi["iters"], gi["products"], gi["neg_curv"], gi["neg_iter"]) == \
        (oi["iters"], oi["products"], oi["neg_curv"], oi["neg_iter"])
    if oi["neg_curv"]:
        assert np.sign(gi["pBp"]) == np.sign(oi["pBp"])
        assert gi["pBp"] == pytest.approx(oi["pBp"], rel=1e-3)
    assert rel(step, oi["step"]) <= 1e-3


def test_pcg_damped_single_layer_reaches_the_solution():
    """L = 1 with damping: B = G + lambda I is SPD and explicit; PCG with
    the Fisher preconditioner reaches numpy.linalg.solve (stopped at a
    relative residual of 1e-6, so the error is below cond(B) 1e-6)."""
    dims, act, B = (5, 4), "sigmoid", 40
    p = WL.make_small(dims, act, B, seed=44)
    n = WL.num_params(dims)
    lam = 0.05
    Bm = np.stack([O.curvature(dims, act, p["theta"], p["X"], p["y"], e,
                               "gauss_newton") for e in np.eye(n)], axis=1)
    Bm += lam * np.eye(n)
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    g32 = g.astype(np.float32).astype(np.float64)
    minv = O.precond_inverse(O.fisher_diag(dims, act, p["theta"], p["X"], p["y"]),
                             lam)
    step, _, gi, oi = pcg_pair(dims, act, p, g32, minv, lam, 2 * n, "gauss_newton",
                               rel_tol=1e-6)
    ex = np.linalg.solve(Bm, -g32)
    print("cond", np.linalg.cond(Bm), "iters", gi["iters"], oi["iters"],
          "err", rel(step, ex), rel(oi["step"], ex))
    assert gi["neg_curv"] == 0 and gi["iters"] < 2 * n
    assert rel(step, ex) <= 1e-4
    assert rel(oi["step"], ex) <= 1e-4


@pytest.mark.parametrize("solver", ["cg", "bicgstab"])
@pytest.mark.parametrize("curv", ["hessian", "gauss_newton"])
def test_iterate_preconditioned(curv, solver):
    """One preconditioned outer iteration against the oracle: curvature,
    solver counts and detections, chosen direction, acceptance, evaluation
    count, step length, f and the new weights."""
    from tests.test_gpu_iterate import MARGIN, TOL_F, TOL_W, ties
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=45)
    th = p["theta"].astype(np.float64)
    iters = 8 if solver == "cg" else 3
    o = O.iterate(dims, act, th, p["X"], p["y"], p["X"], p["y"], solver=solver,
                  curvature_kind=curv, lam=1e-2, max_iters=iters,
                  precondition=True)
    h = net(dims, act, B)
    W = dev(p["theta"].copy())
    gi, _ = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]),
                         dev(np.zeros(h.n, np.float32)), solver=solver,
                         curvature=curv, damping=1e-2, max_iters=iters,
                         precondition=True)
    s, so = gi["solve"], o["solve"]
    print(curv, solver, s["iters"], so["iters"], gi["direction"], o["direction"],
          gi["alpha"], o["alpha"], gi["f1"], o["f1"])
    assert (s["iters"], s["products"], s["neg_curv"]) == \
        (so["iters"], so["products"], so["neg_curv"])
    assert gi["f0"] == pytest.approx(o["f0"], rel=TOL_F)
    Wn = host(W).astype(np.float64)
    if ties(o):
        assert O.loss(dims, act, Wn, p["X"], p["y"]) <= o["f0"] + 1e-4 * \
            gi["alpha"] * gi["gTd"] + MARGIN * abs(o["f0"])
        return
    assert gi["direction"] == o["direction"] and gi["accepted"] == o["accepted"]
    assert gi["evals"] == o["evals"] and gi["alpha"] == o["alpha"]
    assert gi["f1"] == pytest.approx(o["f1"], rel=TOL_F)
    assert rel(Wn, o["theta"]) <= TOL_W


def test_preconditioning_rejections():
    """Preconditioning, with either solver and either precision, takes
    damping > 0 (M = (F + lambda)^xi needs a positive diagonal) and a finite
    xi >= 0.  Rejections are HF_EINVAL and leave W untouched."""
    from paper_1606_00511_amd.hf import HFError, HF_EINVAL
    dims, act, B = (20, 16, 5), "sigmoid", 32
    p = WL.make_small(dims, act, B, seed=46)
    args = (dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]))
    for prec in ("fp32", "bf16"):
        h = net(dims, act, B, prec)
        for solver in ("cg", "bicgstab"):
            for kw in (dict(damping=0.0), dict(precond_exp=-0.5),
                       dict(precond_exp=float("nan"))):
                W = dev(p["theta"].copy())
                with pytest.raises(HFError) as ei:
                    h.hf_iterate(W, *args, dev(np.zeros(h.n, np.float32)),
                                 solver=solver, precondition=True, **kw)
                assert ei.value.code == HF_EINVAL
                assert np.array_equal(host(W), p["theta"])
        h.close()


BF16_CASES = [((100, 200, 150, 37), "tanh", 300),
              ((37, 45, 13), "sigmoid", 130),
              ((40, 96, 1973), "sigmoid", 200)]


@pytest.mark.parametrize("case", BF16_CASES, ids=[
    "x".join(map(str, c[0])) + "-" + c[1] for c in BF16_CASES])
def test_fisher_diag_bf16(case):
    """bf16 GEMM operands: each squared operand is rounded to bf16 again
    before the fp32-accumulated contraction, so F carries a few 2^-8
    relative errors per term; against the oracle at 2e-2, and F >= 0."""
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=51 + B)
    h = net(dims, act, B, "bf16")
    F = host(h.hf_fisher_diag(dev(p["theta"]), dev(p["X"]), dev(p["y"])))
    h.hf_check()
    ref = O.fisher_diag(dims, act, p["theta"], p["X"], p["y"])
    err = rel(F, ref)
    print("bf16 F rel %.2e" % err)
    assert err <= 2e-2
    assert np.all(F >= 0.0)
    h.close()


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
def test_pcg_bf16(mode):
    """bf16 GEMM operands: PCG's counts and detection as the oracle's; the
    detected curvature within 5% and the step within 5e-2 (the bf16 CG
    bar of the full-size tests)."""
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=52)
    _, g = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    lam = 1e-2
    minv = O.precond_inverse(O.fisher_diag(dims, act, p["theta"], p["X"], p["y"]),
                             lam)
    h = net(dims, act, B, "bf16")
    step, nd, gi = h.hf_pcg(dev(p["theta"]), dev(p["X"]), dev(p["y"]),
                            dev(g.astype(np.float32)), dev(minv.astype(np.float32)),
                            lam, 6, mode)
    step = host(step)
    oi = O.cg_network(dims, act, p["theta"], p["X"], p["y"],
                      g.astype(np.float32).astype(np.float64), lam, 6, mode,
                      minv=minv.astype(np.float32).astype(np.float64))
    print(mode, {k: gi[k] for k in ("iters", "products", "neg_curv", "neg_iter",
                                    "pBp")}, oi["iters"], oi["neg_iter"],
          oi["pBp"], "step rel %.2e" % rel(step, oi["step"]))
    assert (gi["iters"], gi["products"], gi["neg_curv"], gi["neg_iter"]) == \
        (oi["iters"], oi["products"], oi["neg_curv"], oi["neg_iter"])
    if oi["neg_curv"]:
        assert np.sign(gi["pBp"]) == np.sign(oi["pBp"])
        assert abs(gi["pBp"] - oi["pBp"]) <= 0.05 * abs(oi["pBp"])
    assert rel(step, oi["step"]) <= 5e-2
    h.close()


@pytest.mark.parametrize("solver", ["cg", "bicgstab"])
def test_iterate_preconditioned_bf16_descends(solver):
    """bf16 GEMM operands with preconditioning: the accepted step descends
    on the exact (fp64) objective, and the reported f0 and f1 agree with it
    at 2e-2."""
    dims, act, B = (100, 200, 150, 37), "sigmoid", 300
    p = WL.make_small(dims, act, B, seed=53)
    h = net(dims, act, B, "bf16")
    W = dev(p["theta"].copy())
    f0 = O.loss(dims, act, p["theta"], p["X"], p["y"])
    gi, _ = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]),
                         dev(np.zeros_like(p["theta"])), solver=solver,
                         curvature="gauss_newton", damping=1e-2,
                         max_iters=6 if solver == "cg" else 3, precondition=True)
    f1 = O.loss(dims, act, host(W).astype(np.float64), p["X"], p["y"])
    print(solver, gi["accepted"], gi["direction"], gi["alpha"], f0, f1)
    assert gi["accepted"] == 1
    assert abs(gi["f0"] - f0) <= 2e-2 * f0
    assert f1 < f0
    assert abs(gi["f1"] - f1) <= 2e-2 * f0
    h.close()


def test_fisher_diag_full_size_speech_net():
    """The speech-frame net at full batch: the output layer's blocks of F
    against the forward-only closed form (fp64), and F >= g^2 in every
    block with the GPU's own gradient (up to fp32 rounding)."""
    import torch
    w = WL.WORKLOADS["speech_440_2048x4_1973_sigmoid_b16384"]
    inp = WL.make(w)
    gc.collect()
    torch.cuda.empty_cache()
    h = net(w.dims, w.act, w.batch)
    W, X, y = dev(inp["theta"]), dev(inp["X"]), dev(inp["y"])
    F = host(h.hf_fisher_diag(W, X, y)).astype(np.float64)
    _, g = h.hf_loss_grad(W, X, y)
    g = host(g).astype(np.float64)
    FW, Fb = O.fisher_diag_output_layer(w.dims, w.act, inp["theta"], inp["X"],
                                        inp["y"])
    C, d = w.dims[-1], w.dims[-2]
    Fo = F[-(C * d + C):]
    eW, eb = rel(Fo[:C * d], FW.ravel()), rel(Fo[C * d:], Fb)
    print("output-layer F rel: weights %.2e bias %.2e" % (eW, eb))
    assert eW <= 1e-4 and eb <= 1e-4
    assert np.all(F >= g * g * (1 - 1e-4) - 1e-30)
    h.close()
