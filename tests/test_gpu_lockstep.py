"""Lock-step diagnostic: every curvature product a solve evaluates inside its
loop, compared element by element with the oracle's product at the same
operand.

CG-Minimize applies B_k(d) = A d + lambda d to each conjugate direction
(Alg. 1 steps 3-4), with A = H or G on the one minibatch of Alg. 2.  Inside a
solve the library evaluates A p on the activations it cached for that
minibatch (the in-CG product, whose GEMMs the benchmark times), not by the
stateless path of hf_hvp.  hf_set_trace copies each product's operand p_j
and result q_j = A p_j out of the solve; the oracle then recomputes
A p_j in fp64 from the same fp32 p_j.  The bar is the fp32 one, rel-L2
<= 1e-4 per product (2e-2 for bf16 GEMM operands), with the ReLU bracket of
tests/parity_util.py.  The first direction of a solve from 0 is -g exactly,
and the slots of products the solve never evaluated stay untouched.

Cases: every workload in the benchmark's launch configuration (the digit
net's 50 Gauss-Newton iterations in full; the speech net's first three and
the one-worker share's first five), the split-K shapes (batch-row GEMMs with
too few tiles, split weight gradients), unaligned widths, Bi-CG-STAB (both
products per iteration), a warm start's product, and the bf16 path.
"""

import gc

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests.parity_util import check, relu_margins

pytestmark = pytest.mark.gpu

TOL = 1e-4
TOL_BF16 = 2e-2


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def compare_trace(tr, products, dims, act, theta, Xc, yc, mode, tol, tag,
                  g=None, tau=None):
    """Check every traced product against the oracle; slots past the
    products evaluated must still hold the NaN fill."""
    cap = tr.shape[0] // 2
    worst = 0.0
    margins = relu_margins(dims, act, theta, Xc) if tau is None else None
    for k in range(cap):
        v, q = tr[2 * k], tr[2 * k + 1]
        if k >= products:
            assert np.isnan(v).all() and np.isnan(q).all(), \
                "%s: slot %d written past the %d products" % (tag, k, products)
            continue
        assert np.isfinite(v).all() and np.isfinite(q).all(), (tag, k)
        if k == 0 and g is not None:
            assert np.array_equal(v, -g), "%s: p_0 != -g" % tag
        v64 = v.astype(np.float64)
        ref = O.curvature(dims, act, theta, Xc, yc, v64, mode)
        kw = {"tau": tau} if tau is not None else {"margins": margins}
        err, bound = check(q, ref, act, lambda kink: O.curvature(
            dims, act, theta, Xc, yc, v64, mode, kink=kink), tol=tol, **kw)
        worst = max(worst, err)
        print("%s product %d: rel %.2e (bound %.2e)" % (tag, k, err, bound),
              flush=True)
    return worst


# ------------------------------------------------------------ small shapes
SMALL = [
    # several 128 x 128 tiles with ragged tails
    ((100, 200, 150, 37), "sigmoid", 300),
    ((100, 200, 150, 37), "tanh", 300),
    ((100, 200, 150, 37), "relu", 300),
    # unaligned widths: register-staged loads
    ((37, 45, 13), "tanh", 33),
    # few rows through wide layers: batch-row GEMMs as split-K partials
    ((256, 2048, 2048, 10), "tanh", 256),
    ((250, 2049, 1999, 13), "sigmoid", 200),
    # many rows: split weight gradients
    ((64, 1100, 10), "tanh", 15000),
]


def sid(c):
    return "%s-%s-b%d" % ("x".join(map(str, c[0])), c[1], c[2])


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", SMALL, ids=[sid(c) for c in SMALL])
def test_lockstep_small(case, mode):
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=4100 + B)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, X, y)
    g_np = host(g)
    cap = 8
    buf = net.set_trace(cap)
    _, _, info = net.hf_cg(W, X, y, g, 1e-2, cap + 2, mode)
    net.set_trace(0)
    tr = host(buf)
    prods = min(cap, info["products"])
    assert prods >= 1
    compare_trace(tr, info["products"], dims, act, p["theta"].astype(np.float64),
                  p["X"], p["y"], mode, TOL, "%s %s" % (sid(case), mode), g=g_np)
    net.close()


def test_lockstep_trace_is_passive():
    """Tracing changes nothing: the solve's step, direction and info are
    bit-identical with and without it."""
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=4099)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, X, y)
    s0, d0, i0 = net.hf_cg(W, X, y, g, 1e-2, 10, "gauss_newton")
    s0, d0 = host(s0), host(d0)
    net.set_trace(4)
    s1, d1, i1 = net.hf_cg(W, X, y, g, 1e-2, 10, "gauss_newton")
    net.set_trace(0)
    assert i0["replayed"] == 1 and i1["replayed"] == 0   # tracing runs launch by launch
    i0.pop("replayed")
    i1.pop("replayed")
    assert i0 == i1
    assert np.array_equal(s0, host(s1)) and np.array_equal(d0, host(d1))
    net.close()


# --------------------------------------------------------------- workloads
# products compared per workload: (hessian, gauss_newton)
CAPS = {
    "mnist_784_100_10_sigmoid_b1000": (10, 10),
    "mnist_784_500x3_10_tanh_b10000": (50, 50),
    "mnist_784_500x3_10_relu_b60000_c6000": (12, 6),
    "speech_440_2048x4_1973_sigmoid_b16384": (3, 3),
    "speech_440_2048x4_1973_sigmoid_b4096_c1024": (5, 5),
}
_cache = {}


def setup(name):
    import torch
    from paper_1606_00511_amd.hf import HFNet
    if name in _cache:
        return _cache[name]
    for k in list(_cache):
        _cache.pop(k)["net"].close()
    gc.collect()
    torch.cuda.empty_cache()
    w = WL.WORKLOADS[name]
    inp = WL.make(w)
    st = dict(w=w, inp=inp, W=dev(inp["theta"]), X=dev(inp["X"]), y=dev(inp["y"]),
              Xc=dev(inp["X"][:w.curv_batch]), yc=dev(inp["y"][:w.curv_batch]),
              net=HFNet(w.dims, w.act, max(w.batch, w.curv_batch)))
    _, st["grad"] = st["net"].hf_loss_grad(st["W"], st["X"], st["y"])
    st["g_np"] = host(st["grad"])
    _cache[name] = st
    return st


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("name", list(WL.WORKLOADS))
def test_lockstep_workload(name, mode):
    s = setup(name)
    w, inp = s["w"], s["inp"]
    cap = CAPS[name][0 if mode == "hessian" else 1]
    buf = s["net"].set_trace(cap)
    _, _, info = s["net"].hf_cg(s["W"], s["Xc"], s["yc"], s["grad"], w.damping,
                                w.cg_iters, mode)
    s["net"].set_trace(0)
    tr = host(buf)
    del buf
    Xc, yc = inp["X"][:w.curv_batch], inp["y"][:w.curv_batch]
    worst = compare_trace(tr, info["products"], w.dims, w.act, inp["theta"],
                          Xc, yc, mode, TOL, "%s %s" % (name, mode), g=s["g_np"])
    print("%s %s: %d products traced of %d, worst rel %.2e" % (
        name, mode, min(cap, info["products"]), info["products"], worst))


# -------------------------------------------------------------- Bi-CG-STAB
@pytest.mark.parametrize("name,iters", [
    ("small", 5), ("speech_440_2048x4_1973_sigmoid_b4096_c1024", 3)])
def test_lockstep_bicgstab(name, iters):
    """Both products of every Bi-CG-STAB iteration (on p and on s)."""
    from paper_1606_00511_amd.hf import HFNet
    mode = "gauss_newton"
    if name == "small":
        dims, act, B = (100, 200, 150, 37), "sigmoid", 300
        p = WL.make_small(dims, act, B, seed=4200)
        theta, Xn, yn, lam = p["theta"], p["X"], p["y"], 1e-2
        net = HFNet(dims, act, B)
        W, Xc, yc = dev(theta), dev(Xn), dev(yn)
        _, g = net.hf_loss_grad(W, Xc, yc)
    else:
        s = setup(name)
        w, inp = s["w"], s["inp"]
        dims, act, theta, lam = w.dims, w.act, inp["theta"], w.damping
        Xn, yn = inp["X"][:w.curv_batch], inp["y"][:w.curv_batch]
        net, W, Xc, yc, g = s["net"], s["W"], s["Xc"], s["yc"], s["grad"]
    buf = net.set_trace(2 * iters)
    _, _, info = net.hf_bicgstab(W, Xc, yc, g, lam, iters, mode)
    net.set_trace(0)
    tr = host(buf)
    assert info["products"] == 2 * iters
    compare_trace(tr, info["products"], dims, act, np.asarray(theta, np.float64),
                  Xn, yn, mode, TOL, "bicgstab %s" % name)
    # the first operand of Bi-CG-STAB from 0 is p_0 = r_0 = -g
    assert np.array_equal(tr[0], -host(g))


def test_lockstep_pbicgstab():
    """Right-preconditioned Bi-CG-STAB: its products are on M^-1 p and
    M^-1 s, each against the oracle's A at the same operand; the first
    operand is M^-1 r_0 = minv (.) (-g), rounded once to fp32."""
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B, iters = (100, 200, 150, 37), "tanh", 300, 4
    p = WL.make_small(dims, act, B, seed=4250)
    lam = 1e-2
    minv = O.precond_inverse(O.fisher_diag(dims, act, p["theta"], p["X"],
                                           p["y"]), lam).astype(np.float32)
    net = HFNet(dims, act, B)
    W, Xc, yc = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = net.hf_loss_grad(W, Xc, yc)
    for mode in ("hessian", "gauss_newton"):
        buf = net.set_trace(2 * iters)
        _, _, info = net.hf_pbicgstab(W, Xc, yc, g, dev(minv), lam, iters, mode)
        net.set_trace(0)
        tr = host(buf)
        compare_trace(tr, info["products"], dims, act,
                      p["theta"].astype(np.float64), p["X"], p["y"], mode, TOL,
                      "pbicgstab %s" % mode)
        first = (minv.astype(np.float64) * -host(g).astype(np.float64))
        assert np.array_equal(tr[0], first.astype(np.float32))
    net.close()


# -------------------------------------------------------------- warm start
def test_lockstep_warm_start():
    """hf_iterate from eta delta: product 0 is on x_0 = eta delta (rounded
    once to fp32), the solver's products follow."""
    import torch
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=4300)
    net = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    rng = np.random.default_rng(4301)
    d_np = (1e-2 * rng.standard_normal(net.n)).astype(np.float32)
    delta = dev(d_np)
    buf = net.set_trace(4)
    info, _ = net.hf_iterate(W.clone(), X, y, X, y, delta, curvature="gauss_newton",
                             max_iters=3, eta=0.5)
    net.set_trace(0)
    tr = host(buf)
    assert info["solve"]["products"] == 4
    assert np.array_equal(tr[0], (0.5 * d_np).astype(np.float32))
    compare_trace(tr, 4, dims, act, p["theta"].astype(np.float64), p["X"], p["y"],
                  "gauss_newton", TOL, "warm start")
    del torch


# -------------------------------------------------------------------- bf16
@pytest.mark.parametrize("name,mode,cap", [
    ("small", "hessian", 6), ("small", "gauss_newton", 6),
    ("speech_440_2048x4_1973_sigmoid_b16384", "gauss_newton", 3)])
def test_lockstep_bf16(name, mode, cap):
    """The bf16-operand in-CG product against the oracle at 2e-2."""
    import torch
    from paper_1606_00511_amd.hf import HFNet
    if name == "small":
        dims, act, B = (100, 200, 150, 37), "tanh", 300
        p = WL.make_small(dims, act, B, seed=4400)
        theta, Xn, yn, lam, Bc = p["theta"], p["X"], p["y"], 1e-2, B
    else:
        for k in list(_cache):
            _cache.pop(k)["net"].close()
        gc.collect()
        torch.cuda.empty_cache()
        w = WL.WORKLOADS[name]
        inp = WL.make(w)
        dims, act, theta, lam = w.dims, w.act, inp["theta"], w.damping
        Xn, yn, B, Bc = inp["X"], inp["y"], w.batch, w.curv_batch
    net = HFNet(dims, act, B, prec="bf16")
    W, X, y = dev(theta), dev(Xn), dev(yn)
    _, g = net.hf_loss_grad(W, X, y)
    buf = net.set_trace(cap)
    _, _, info = net.hf_cg(W, X[:Bc], y[:Bc], g, lam, cap, mode)
    net.set_trace(0)
    tr = host(buf)
    del buf
    compare_trace(tr, info["products"], dims, act, np.asarray(theta, np.float64),
                  Xn[:Bc], yn[:Bc], mode, TOL_BF16, "bf16 %s %s" % (name, mode),
                  g=host(g), tau=2.0 ** -5)
    net.close()
