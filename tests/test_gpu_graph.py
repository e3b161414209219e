"""CG with each iteration replayed from one captured graph, against the same
solve launched kernel by kernel.

When nothing needs host work between the kernels of an iteration (no kernel
timing, no kept iterates, no product trace), hf_cg and hf_pcg capture one
iteration (the cached curvature product and the vector kernels, with the
iteration index kept on the device) and launch that graph once per
iteration.  The kernels and their order are the same, so the step, the
negative-curvature direction and every field of the solve's report must be
bit-identical to the kernel-by-kernel solve (forced here by turning kernel
timing on).  Cases: detection at the first iteration and later, the
relative-residual stop, a budget of one iteration, preconditioned CG, split
batch-row GEMMs, a warm start through hf_iterate, a captured graph reused
and rebuilt when an argument changes, and a non-default stream.
"""

import numpy as np
import pytest

from paper_1606_00511_amd import workloads as WL

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().copy()


def solve(net, eager, *args, pcg=None, **kw):
    net.prof_enable(eager)
    if pcg is None:
        step, nd, info = net.hf_cg(*args, **kw)
    else:
        W, X, y, g, lam, iters, mode = args
        step, nd, info = net.hf_pcg(W, X, y, g, pcg, lam, iters, mode, **kw)
    out = host(step), host(nd), dict(info)
    net.prof_enable(False)
    return out


def same(a, b):
    (s0, d0, i0), (s1, d1, i1) = a, b
    i0, i1 = dict(i0), dict(i1)
    assert i0.pop("replayed") == 1 and i1.pop("replayed") == 0
    assert i0 == i1
    assert np.array_equal(s0, s1) and np.array_equal(d0, d1)


CASES = [
    ((100, 200, 150, 37), "tanh", 300, "hessian", 12, 0.0),
    ((100, 200, 150, 37), "sigmoid", 300, "gauss_newton", 12, 0.0),
    ((100, 200, 150, 37), "relu", 300, "hessian", 12, 0.0),
    ((37, 45, 13), "tanh", 33, "gauss_newton", 1, 0.0),
    ((37, 45, 13), "sigmoid", 130, "gauss_newton", 200, 1e-3),
    ((784, 100, 10), "sigmoid", 1000, "hessian", 10, 0.0),
    ((256, 2048, 2048, 10), "tanh", 256, "gauss_newton", 6, 0.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-%s-%s-%d" % (
    "x".join(map(str, c[0])), c[1], c[3], c[4]))
def test_replayed_cg_matches_launch_by_launch(case):
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B, mode, iters, tol = case
    p = WL.make_small(dims, act, B, seed=6100 + B)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, X, y)
    args = (W, X, y, g, 1e-2, iters, mode)
    r = solve(net, False, *args, rel_tol=tol)
    e = solve(net, True, *args, rel_tol=tol)
    print(dims, act, mode, {k: r[2][k] for k in ("iters", "products", "neg_curv",
                                                 "neg_iter", "replayed")})
    same(r, e)
    # the captured iteration is reused by a second solve with the same
    # arguments, and rebuilt for another gradient
    r2 = solve(net, False, *args, rel_tol=tol)
    same(r2, e)
    g2 = (g * 0.5).contiguous()
    args2 = (W, X, y, g2, 1e-2, iters, mode)
    same(solve(net, False, *args2, rel_tol=tol), solve(net, True, *args2, rel_tol=tol))
    net.close()


def test_replayed_pcg_and_detection_at_first_iteration():
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=6200)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, X, y)
    F = net.hf_fisher_diag(W, X, y)
    import torch
    minv = ((F + 1e-2) ** -0.75).contiguous()
    args = (W, X, y, g, 1e-2, 15, "gauss_newton")
    same(solve(net, False, *args, pcg=minv), solve(net, True, *args, pcg=minv))
    # detection at the first iteration: with g = -d~ for a direction d~ of
    # negative curvature (from a Hessian solve's detection) and no damping,
    # p_0 = d~ and p_0^T H p_0 < 0
    _, nd, info = net.hf_cg(W, X, y, g, 1e-2, 20, "hessian")
    if info["neg_curv"]:
        gneg = (-nd).contiguous()
        args = (W, X, y, gneg, 0.0, 5, "hessian")
        r = solve(net, False, *args)
        e = solve(net, True, *args)
        same(r, e)
    del torch
    net.close()


def test_replayed_on_a_non_default_stream_and_after_iterate():
    import torch
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = (100, 200, 150, 37), "sigmoid", 300
    p = WL.make_small(dims, act, B, seed=6300)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, X, y)
    args = (W, X, y, g, 1e-2, 10, "gauss_newton")
    ref = solve(net, True, *args)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = solve(net, False, *args)
    s.synchronize()
    same(out, ref)
    # an outer iteration with a warm start (its solve is replayed too), then
    # a plain solve again
    delta = torch.zeros(net.n, device="cuda")
    Wc = W.clone()
    info, _ = net.hf_iterate(Wc, X, y, X, y, delta, curvature="gauss_newton",
                             max_iters=4, eta=0.5)
    assert info["solve"]["replayed"] == 1
    same(solve(net, False, *args), ref)
    net.close()
