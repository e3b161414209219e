"""GPU parity of the loss-only forward (hf_loss) and of one outer HF
iteration (hf_iterate: gradient, warm-started solve, direction choice,
Armijo backtracking, Hybrid-CG policy; Alg. 2, Sec. 2.2, Sec. 3) against
the fp64 oracle on the same seeded float32 inputs.

Bar (fp32 path): f within 1e-4 relative; identical curvature used, solver
counts and detections, chosen direction, acceptance, number of loss
evaluations and step length; the new weights within 1e-3 relative L2 (the
solver's step drifts between fp32 and fp64 only by its rounding).  The line
search compares objective values with an Armijo bound, a decision taken on
a float: when the oracle finds any trial within fp32 rounding of its bound,
the two sides may legitimately decide differently, and only the Armijo
condition of the GPU's own step is then checked (with the oracle).  The same
holds when the solve itself is ill-conditioned: Bi-CG-STAB near a breakdown
amplifies the rounding of its float32 vectors (measured, as in the
Bi-CG-STAB parity tests, by rerunning the oracle's solve with float32
storage and 1e-7 product noise); when that moves the step by more than
1e-4, the GPU step is checked for the Armijo condition instead.
"""

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests.parity_util import rel

pytestmark = pytest.mark.gpu

TOL_F = 1e-4
TOL_W = 1e-3
MARGIN = 1e-5          # relative distance to an Armijo bound treated as a tie


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


MODE_NAMES = {0: "hessian", 1: "gauss_newton"}


@pytest.mark.parametrize("prec,tol", [("fp32", 1e-4), ("bf16", 2e-2)])
@pytest.mark.parametrize("case", [((100, 200, 150, 37), "sigmoid", 300),
                                  ((37, 45, 13), "relu", 130),
                                  ((40, 96, 1973), "tanh", 200)])
def test_loss_only(case, prec, tol):
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=31 + B)
    f = O.loss(dims, act, p["theta"], p["X"], p["y"])
    h = net(dims, act, B, prec)
    got = float(host(h.hf_loss(dev(p["theta"]), dev(p["X"]), dev(p["y"])))[0])
    h.hf_check()
    assert abs(got - f) <= tol * abs(f)


def ties(o):
    return any(abs(ft - bound) <= MARGIN * abs(o["f0"])
               for _, _, ft, bound in o["trials"])


def sensitivity(dims, act, th, p, kw, mode, x0):
    """How far float32 storage and 1e-7 product noise move the oracle's
    Bi-CG-STAB step (0 for CG)."""
    if kw.get("solver", "cg") != "bicgstab":
        return 0.0
    _, g = O.loss_grad(dims, act, th, p["X"], p["y"])
    rng = np.random.default_rng(12345)
    f32 = lambda v: v.astype(np.float32).astype(np.float64)

    def noisy(v):
        w = O.curvature(dims, act, th, p["X"], p["y"], v, mode)
        return w * (1.0 + 1e-7 * rng.standard_normal(w.size))
    lam, iters = kw.get("damping", 1e-2), kw.get("max_iters", 10)
    a = O.bicgstab_minimize(noisy, g, lam, iters, store=f32, x0=x0)
    b = O.bicgstab_minimize(lambda v: O.curvature(dims, act, th, p["X"], p["y"],
                                                  v, mode), g, lam, iters, x0=x0)
    return rel(a["step"], b["step"])


def compare_step(h, dims, act, p, th, delta, kw, hybrid, o, W, x0=None):
    """Run hf_iterate on (th, delta) and compare with the oracle's step o."""
    gi, hs = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]),
                          dev(p["y"]), delta, hybrid_state=hybrid, **kw)
    Wn = host(W).astype(np.float64)
    assert MODE_NAMES[gi["mode_used"]] == o["mode_used"]
    s, so = gi["solve"], o["solve"]
    assert (s["iters"], s["products"], s["neg_curv"]) == \
        (so["iters"], so["products"], so["neg_curv"])
    assert gi["f0"] == pytest.approx(o["f0"], rel=TOL_F)
    if ties(o) or sensitivity(dims, act, th, p, kw, o["mode_used"], x0) > 1e-4:
        # a decision within rounding of its bound: check the GPU's own step
        if gi["accepted"]:
            f_new = O.loss(dims, act, Wn, p["X"], p["y"])
            assert f_new <= o["f0"] + kw.get("armijo_c", 1e-4) * gi["alpha"] * \
                gi["gTd"] + MARGIN * abs(o["f0"])
        return gi, hs, Wn
    assert gi["direction"] == o["direction"]
    assert gi["accepted"] == o["accepted"]
    assert gi["evals"] == o["evals"]
    assert gi["alpha"] == o["alpha"]
    assert gi["f1"] == pytest.approx(o["f1"], rel=TOL_F)
    assert rel(Wn, o["theta"]) <= TOL_W
    assert hs == int(o["hybrid_g"])
    return gi, hs, Wn


@pytest.mark.parametrize("solver", ["cg", "bicgstab"])
@pytest.mark.parametrize("curvature", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("act", ["sigmoid", "tanh"])
def test_iterate_one_step(act, curvature, solver):
    dims, B = (100, 200, 150, 37), 300
    p = WL.make_small(dims, act, B, seed=57)
    th = p["theta"].astype(np.float64)
    kw = dict(solver=solver, curvature=curvature, damping=1e-2, max_iters=6)
    o = O.iterate(dims, act, th, p["X"], p["y"], p["X"], p["y"], solver=solver,
                  curvature_kind=curvature, lam=1e-2, max_iters=6)
    h = net(dims, act, B)
    W = dev(p["theta"].copy())
    delta = dev(np.zeros_like(p["theta"]))
    gi, _, _ = compare_step(h, dims, act, p, th, delta, kw, 0, o, W)
    print("%s %s %s: dir %d alpha %g evals %d f %.6f -> %.6f (oracle %.6f)"
          % (act, curvature, solver, gi["direction"], gi["alpha"], gi["evals"],
             gi["f0"], gi["f1"], o["f1"]))


@pytest.mark.parametrize("solver", ["cg", "bicgstab"])
def test_iterate_hybrid_warm_started_trajectory(solver):
    """Four iterations of Hybrid-CG with warm starts eta = 0.5: the curvature
    used, the decisions and the objective follow the oracle step by step
    (each oracle step starts from the GPU's weights, so rounding does not
    accumulate across steps)."""
    dims, act, B = (20, 16, 12, 5), "tanh", 64
    p = WL.make_small(dims, act, B, seed=3)
    h = net(dims, act, B)
    W = dev(p["theta"].copy())
    delta = dev(np.zeros_like(p["theta"]))
    kw = dict(solver=solver, curvature="hybrid", damping=1e-2, max_iters=6,
              eta=0.5)
    hyb = 0
    modes = []
    for k in range(4):
        th = host(W).astype(np.float64)
        dprev = host(delta).astype(np.float64)
        o = O.iterate(dims, act, th, p["X"], p["y"], p["X"], p["y"],
                      solver=solver, curvature_kind="hybrid", lam=1e-2,
                      max_iters=6, eta=0.5, delta_prev=dprev, hybrid_g=bool(hyb))
        gi, hyb, _ = compare_step(h, dims, act, p, th, delta, kw, hyb, o, W,
                                  x0=0.5 * dprev if k > 0 else None)
        modes.append(gi["mode_used"])
        assert gi["f1"] <= gi["f0"]
    print("modes", modes)


def test_iterate_bf16_descends():
    """bf16 GEMM operands: the step is a descent step for the exact (fp64)
    objective and satisfies its Armijo condition up to the 2e-2 bound."""
    dims, act, B = (100, 200, 150, 37), "sigmoid", 300
    p = WL.make_small(dims, act, B, seed=57)
    h = net(dims, act, B, "bf16")
    W = dev(p["theta"].copy())
    delta = dev(np.zeros_like(p["theta"]))
    f0 = O.loss(dims, act, p["theta"], p["X"], p["y"])
    gi, _ = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]),
                         delta, curvature="gauss_newton", max_iters=6)
    assert gi["accepted"] == 1
    f1 = O.loss(dims, act, host(W).astype(np.float64), p["X"], p["y"])
    assert abs(gi["f0"] - f0) <= 2e-2 * f0
    assert f1 < f0
    assert abs(gi["f1"] - f1) <= 2e-2 * f0


def test_iterate_rejects_uphill_nothing_to_accept():
    """max_iters = 0: the solver returns the zero step, which is not a
    descent direction; nothing is accepted and W is unchanged."""
    dims, act, B = (20, 16, 12, 5), "sigmoid", 64
    p = WL.make_small(dims, act, B, seed=8)
    h = net(dims, act, B)
    W = dev(p["theta"].copy())
    delta = dev(np.ones_like(p["theta"]))
    gi, _ = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]),
                         delta, max_iters=0)
    assert gi["accepted"] == 0 and gi["direction"] == -1 and gi["evals"] == 0
    assert np.array_equal(host(W), p["theta"])
    assert not host(delta).any()
    assert gi["f1"] == gi["f0"]


def test_iterate_full_size_speech_net():
    """The speech-frame net at full batch: one Hessian CG iteration (its
    solve meets negative curvature at the second product) and the line
    search, against the oracle."""
    w = WL.WORKLOADS["speech_440_2048x4_1973_sigmoid_b16384"]
    inp = WL.make(w)
    h = net(w.dims, w.act, w.batch)
    W = dev(inp["theta"].copy())
    delta = dev(np.zeros_like(inp["theta"]))
    kw = dict(solver="cg", curvature="hessian", damping=w.damping, max_iters=4)
    o = O.iterate(w.dims, w.act, inp["theta"].astype(np.float64), inp["X"],
                  inp["y"], inp["X"], inp["y"], solver="cg",
                  curvature_kind="hessian", lam=w.damping, max_iters=4)
    gi, _, _ = compare_step(h, w.dims, w.act, inp, inp["theta"], delta, kw, 0,
                            o, W)
    print("speech: dir %d alpha %g evals %d f %.6f -> %.6f"
          % (gi["direction"], gi["alpha"], gi["evals"], gi["f0"], gi["f1"]))


# ---------------------------------------------- CG-backtracking and damping
def test_kept_iterates_are_the_truncated_solves():
    """The iterates kept for CG-backtracking are bit-identical to the steps
    of the same GPU solve truncated at their iteration counts; slots of
    iterations the solve never reached (it stops at negative curvature on
    the Hessian) are left untouched."""
    import torch
    dims, act, B = (37, 45, 13), "tanh", 130
    p = WL.make_small(dims, act, B, seed=61)
    h = net(dims, act, B)
    W0, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    for curv, iters in (("gauss_newton", 9), ("hessian", 9)):
        J = O.backtrack_schedule(iters, 4)
        keep = torch.full((len(J), h.n), 123.0, device="cuda")
        gi, _ = h.hf_iterate(W0.clone(), X, y, X, y, dev(np.zeros(h.n, np.float32)),
                             solver="cg", curvature=curv, max_iters=iters,
                             keep=keep)
        f, g = h.hf_loss_grad(W0, X, y)
        reached = gi["solve"]["iters"]
        for i, j in enumerate(J):
            k = host(keep[i])
            if j <= reached:
                step, _, _ = h.hf_cg(W0, X, y, g, 1e-2, j, curv)
                assert np.array_equal(k, host(step)), (curv, j)
            else:
                assert bool((k == 123.0).all()), (curv, j)
        print(curv, "reached", reached, "kept", J)


@pytest.mark.parametrize("solver", ["cg", "bicgstab"])
@pytest.mark.parametrize("seed", [24, 25])
def test_iterate_backtracking_and_damping(solver, seed):
    """CG-backtracking and the damping rule against the oracle iteration:
    the chosen iterate, the evaluation count, the accepted update, rho and
    the next lambda.  Backtracking compares objective values of successive
    iterates, which can lie within fp32 rounding of each other; where the
    oracle's compared values do, only the objective of the GPU's choice is
    checked (equal to the oracle's choice within that rounding)."""
    import torch
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=seed)
    th = p["theta"].astype(np.float64)
    lam, iters = 1e-2, 8
    o = O.iterate(dims, act, th, p["X"], p["y"], p["X"], p["y"], solver=solver,
                  curvature_kind="gauss_newton", lam=lam, max_iters=iters,
                  damping_adapt=True, backtrack_cap=20)
    h = net(dims, act, B)
    W = dev(p["theta"].copy())
    keep = torch.zeros((len(O.backtrack_schedule(iters, 20)), h.n), device="cuda")
    gi, _ = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]),
                         dev(np.zeros(h.n, np.float32)), solver=solver,
                         curvature="gauss_newton", damping=lam, max_iters=iters,
                         adapt_damping=True, keep=keep)
    sol = o["solve"]
    assert (gi["solve"]["iters"], gi["solve"]["products"]) == \
        (sol["iters"], sol["products"])
    f = lambda x: O.loss(dims, act, th + x, p["X"], p["y"])
    js = [sol["iters"]] + sorted((j for j in sol["kept"] if j < sol["iters"]),
                                 reverse=True)
    xs = {sol["iters"]: sol["step"], **{j: sol["kept"][j] for j in js[1:]}}
    fs = {j: f(xs[j]) for j in js}
    # pairs the walk compares, up to one past the oracle's choice
    k = js.index(o["backtrack_iter"])
    pairs = [(js[i], js[i + 1]) for i in range(min(k + 1, len(js) - 1))]
    close = any(abs(fs[a] - fs[b]) <= MARGIN * abs(o["f0"]) for a, b in pairs)
    print("%s seed %d: oracle bt %d gpu bt %d evals %d/%d rho %.4f/%.4f "
          "lam %.4g/%.4g close %s" % (solver, seed, o["backtrack_iter"],
                                      gi["backtrack_iter"], o["evals"], gi["evals"],
                                      o["rho"], gi["rho"], o["lam_next"],
                                      gi["damping_next"], close))
    if close:
        assert gi["backtrack_iter"] in fs
        assert abs(fs[gi["backtrack_iter"]] - fs[o["backtrack_iter"]]) <= \
            2 * MARGIN * abs(o["f0"])
        return
    assert gi["backtrack_iter"] == o["backtrack_iter"]
    kw = dict(solver=solver, damping=lam, max_iters=iters)
    if sensitivity(dims, act, th, p, kw, "gauss_newton", None) > 1e-4:
        # Bi-CG-STAB near a breakdown: check the GPU's own update
        Wn = host(W).astype(np.float64)
        assert gi["accepted"] == 1
        assert O.loss(dims, act, Wn, p["X"], p["y"]) <= o["f0"] + 1e-4 * \
            gi["alpha"] * gi["gTd"] + MARGIN * abs(o["f0"])
        assert gi["damping_next"] == pytest.approx(
            O.adapt_damping(np.float32(lam), gi["rho"]), rel=1e-6)
        return
    assert gi["evals"] == o["evals"]
    assert gi["direction"] == o["direction"] and gi["accepted"] == o["accepted"]
    assert gi["alpha"] == o["alpha"]
    assert gi["f1"] == pytest.approx(o["f1"], rel=TOL_F)
    assert rel(host(W).astype(np.float64), o["theta"]) <= TOL_W
    assert gi["rho"] == pytest.approx(o["rho"], rel=1e-2)
    if min(abs(o["rho"] - 0.25), abs(o["rho"] - 0.75)) > 1e-2:
        assert gi["damping_next"] == pytest.approx(o["lam_next"], rel=1e-6)


def test_damping_without_an_accepted_step_and_when_off():
    """Nothing accepted (zero solver budget): rho = -inf and lambda rises by
    3/2.  Adaptation off: rho is NaN and lambda is returned unchanged."""
    dims, act, B = (20, 16, 12, 5), "sigmoid", 64
    p = WL.make_small(dims, act, B, seed=8)
    h = net(dims, act, B)
    args = (dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]))
    gi, _ = h.hf_iterate(dev(p["theta"].copy()), *args,
                         dev(np.zeros(h.n, np.float32)), max_iters=0,
                         damping=0.02, adapt_damping=True)
    assert gi["accepted"] == 0 and gi["rho"] == float("-inf")
    assert gi["damping_next"] == pytest.approx(1.5 * np.float32(0.02), rel=1e-7)
    gi, _ = h.hf_iterate(dev(p["theta"].copy()), *args,
                         dev(np.zeros(h.n, np.float32)), max_iters=4,
                         damping=0.02)
    assert np.isnan(gi["rho"]) and gi["backtrack_iter"] == -1
    assert gi["damping_next"] == pytest.approx(np.float32(0.02), rel=1e-7)


def test_iterate_all_features_trajectory():
    """Three outer iterations with every option on (Hybrid-CG, warm start
    eta = 0.5, preconditioned CG, CG-backtracking, damping adjustment), the
    caller carrying lambda from damping_next: each step against the oracle
    started from the GPU's weights, delta and lambda."""
    import torch
    dims, act, B = (20, 16, 12, 5), "tanh", 64
    p = WL.make_small(dims, act, B, seed=5)
    h = net(dims, act, B)
    W = dev(p["theta"].copy())
    delta = dev(np.zeros_like(p["theta"]))
    iters = 6
    keep = torch.zeros((len(O.backtrack_schedule(iters, 8)), h.n), device="cuda")
    lam, hyb = np.float32(0.05), 0
    for k in range(3):
        th = host(W).astype(np.float64)
        dprev = host(delta).astype(np.float64)
        o = O.iterate(dims, act, th, p["X"], p["y"], p["X"], p["y"], solver="cg",
                      curvature_kind="hybrid", lam=float(lam), max_iters=iters,
                      eta=0.5, delta_prev=dprev, hybrid_g=bool(hyb),
                      damping_adapt=True, backtrack_cap=8, precondition=True)
        gi, hyb_new = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]),
                                   dev(p["y"]), delta, solver="cg",
                                   curvature="hybrid", damping=float(lam),
                                   max_iters=iters, eta=0.5, hybrid_state=hyb,
                                   adapt_damping=True, keep=keep, precondition=True)
        s, so = gi["solve"], o["solve"]
        print("step %d: mode %d/%s iters %d/%d bt %d/%d dir %d/%d alpha %g/%g rho "
              "%.4f/%.4f lam %.4g" % (k, gi["mode_used"], o["mode_used"], s["iters"],
                                      so["iters"], gi["backtrack_iter"],
                                      o["backtrack_iter"], gi["direction"],
                                      o["direction"], gi["alpha"], o["alpha"],
                                      gi["rho"], o["rho"], gi["damping_next"]))
        assert MODE_NAMES[gi["mode_used"]] == o["mode_used"]
        assert (s["iters"], s["products"], s["neg_curv"]) == \
            (so["iters"], so["products"], so["neg_curv"])
        assert gi["f0"] == pytest.approx(o["f0"], rel=TOL_F)
        if not ties(o):
            assert gi["backtrack_iter"] == o["backtrack_iter"]
            assert gi["direction"] == o["direction"] and gi["alpha"] == o["alpha"]
            assert gi["f1"] == pytest.approx(o["f1"], rel=TOL_F)
            assert rel(host(W).astype(np.float64), o["theta"]) <= TOL_W
            if min(abs(o["rho"] - 0.25), abs(o["rho"] - 0.75)) > 1e-2:
                assert gi["damping_next"] == pytest.approx(o["lam_next"], rel=1e-6)
        assert gi["f1"] <= gi["f0"]
        assert hyb_new == int(o["hybrid_g"]) or ties(o)
        lam, hyb = np.float32(gi["damping_next"]), hyb_new


def test_iterate_bf16_with_backtracking_and_damping():
    """bf16 GEMM operands with CG-backtracking and the damping adjustment:
    the accepted update descends the exact (fp64) objective, the chosen
    iterate is one the solve kept (or its final one), and lambda follows the
    rule applied to the reported rho."""
    import torch
    dims, act, B = (100, 200, 150, 37), "sigmoid", 300
    p = WL.make_small(dims, act, B, seed=58)
    h = net(dims, act, B, "bf16")
    W = dev(p["theta"].copy())
    keep = torch.zeros((len(O.backtrack_schedule(10, 16)), h.n), device="cuda")
    gi, _ = h.hf_iterate(W, dev(p["X"]), dev(p["y"]), dev(p["X"]), dev(p["y"]),
                         dev(np.zeros(h.n, np.float32)), curvature="gauss_newton",
                         max_iters=10, adapt_damping=True, keep=keep)
    f0 = O.loss(dims, act, p["theta"], p["X"], p["y"])
    f1 = O.loss(dims, act, host(W).astype(np.float64), p["X"], p["y"])
    assert gi["accepted"] == 1 and f1 < f0
    assert gi["backtrack_iter"] in O.backtrack_schedule(10, 16) + [gi["solve"]["iters"]]
    assert gi["damping_next"] == pytest.approx(
        O.adapt_damping(np.float32(1e-2), gi["rho"]), rel=1e-6)
