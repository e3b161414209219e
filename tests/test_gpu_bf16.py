"""GPU parity of the bf16-input path (HF_BF16_INPUTS: bf16 GEMM operands,
fp32 accumulation and epilogues), through the C ABI, against the fp64
oracle on the same seeded float32 inputs.

Bar: relative L2 error <= 2e-2 for the loss, the gradient, H v and G v; for
CG on the speech-frame net, identical iteration and product counts and
identical negative-curvature decisions and signs.  Shapes span several
128 x 128 tiles with ragged tails, unaligned widths (padded bf16 rows and
guarded loads), a single row, one weight layer, split-K weight gradients
and both output widths of the workloads.

ReLU: 1[z > 0] is decided on a pre-activation that carries the rounding of
its bf16 operands, about 2^-8 of |z|'s scale (unit variance here).  As in
the fp32 tests the oracle brackets the decision by moving the kink to -tau
and +tau, with tau = 2^-5, eight times that rounding.
"""

import gc

import numpy as np
import pytest

from oracle import hf_oracle as O
from paper_1606_00511_amd import workloads as WL
from tests.parity_util import check, rel

pytestmark = pytest.mark.gpu

TOL = 2e-2
TAU = 2.0 ** -5


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def net(dims, act, max_batch):
    from paper_1606_00511_amd.hf import HFNet
    return HFNet(dims, act, max_batch, prec="bf16")


SMALL = [
    ((100, 200, 150, 37), "sigmoid", 300),
    ((100, 200, 150, 37), "tanh", 300),
    ((100, 200, 150, 37), "relu", 300),
    ((37, 45, 13), "tanh", 130),
    ((37, 45, 13), "sigmoid", 1),
    ((64, 10), "sigmoid", 257),
    ((784, 100, 10), "sigmoid", 1000),
    ((40, 96, 1973), "sigmoid", 200),
    ((64, 1100, 10), "tanh", 15000),
    ((63, 1101, 10), "sigmoid", 15000),
]


def ids(c):
    return "%s-%s-b%d" % ("x".join(map(str, c[0])), c[1], c[2])


@pytest.mark.parametrize("case", SMALL, ids=[ids(c) for c in SMALL])
def test_bf16_loss_grad(case):
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=101 + B)
    f_o, g_o = O.loss_grad(dims, act, p["theta"], p["X"], p["y"])
    h = net(dims, act, B)
    loss, grad = h.hf_loss_grad(dev(p["theta"]), dev(p["X"]), dev(p["y"]))
    h.hf_check()
    lerr = abs(float(host(loss)[0]) - f_o) / abs(f_o)
    err, bound = check(host(grad), g_o, act, lambda k: O.loss_grad(
        dims, act, p["theta"], p["X"], p["y"], kink=k)[1], tol=TOL, tau=TAU)
    print("loss rel %.2e grad rel %.2e (bound %.2e)" % (lerr, err, bound))
    assert lerr <= TOL


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("case", SMALL, ids=[ids(c) for c in SMALL])
def test_bf16_curvature_product(case, mode):
    dims, act, B = case
    p = WL.make_small(dims, act, B, seed=202 + B)
    ref = O.curvature(dims, act, p["theta"], p["X"], p["y"], p["v"], mode)
    h = net(dims, act, B)
    out = h.hf_hvp(dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"]), mode)
    err, bound = check(host(out), ref, act, lambda k: O.curvature(
        dims, act, p["theta"], p["X"], p["y"], p["v"], mode, kink=k),
        tol=TOL, tau=TAU)
    print("%s rel %.2e (bound %.2e)" % (mode, err, bound))


def test_bf16_cached_product_matches_stateless():
    """The solve's cached product path against the stateless one: with no
    damping the first CG iterate is x_1 = -(g.g / g.A g) g, where A g is
    evaluated on the cache, while hf_hvp recomputes the forward pass."""
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=17)
    h = net(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    g = p["v"].astype(np.float32)
    for mode in ("gauss_newton", "hessian"):
        hg = host(h.hf_hvp(W, X, y, dev(g), mode)).astype(np.float64)
        g64 = g.astype(np.float64)
        gHg = float(g64 @ hg)
        step, _, info = h.hf_cg(W, X, y, dev(g), 0.0, 1, mode)
        if gHg > 0:
            assert info["iters"] == 1 and info["neg_curv"] == 0
            x1 = -(g64 @ g64) / gHg * g64
            assert rel(host(step), x1) <= 1e-3
        else:
            assert info["neg_curv"] == 1 and info["neg_iter"] == 0


def test_bf16_deterministic_and_label_free():
    dims, act, B = (100, 200, 150, 37), "sigmoid", 300
    p = WL.make_small(dims, act, B, seed=7)
    h = net(dims, act, B)
    W, X, v = dev(p["theta"]), dev(p["X"]), dev(p["v"])
    a = host(h.hf_hvp(W, X, dev(p["y"]), v, "gauss_newton"))
    b = host(h.hf_hvp(W, X, None, v, "gauss_newton"))
    assert np.array_equal(a, b)
    h1 = host(h.hf_hvp(W, X, dev(p["y"]), v, "hessian"))
    h2 = host(h.hf_hvp(W, X, dev(p["y"]), v, "hessian"))
    assert np.array_equal(h1, h2)
    s1, _, i1 = h.hf_cg(W, X, dev(p["y"]), v, 1e-2, 8, "gauss_newton")
    s1 = host(s1).copy()
    s2, _, i2 = h.hf_cg(W, X, dev(p["y"]), v, 1e-2, 8, "gauss_newton")
    assert np.array_equal(s1, host(s2)) and i1 == i2


# ------------------------------------------------------------ full size
SPEECH = ["speech_440_2048x4_1973_sigmoid_b16384",
          "speech_440_2048x4_1973_sigmoid_b4096_c1024"]
# CG iterations compared against the oracle: (hessian, gauss_newton)
CAPS = {SPEECH[0]: (4, 3), SPEECH[1]: (6, 5)}
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
              v=dev(inp["v"]), Xc=dev(inp["X"][:w.curv_batch]),
              yc=dev(inp["y"][:w.curv_batch]),
              net=HFNet(w.dims, w.act, max(w.batch, w.curv_batch), prec="bf16"))
    _cache[name] = st
    return st


@pytest.mark.parametrize("name", SPEECH)
def test_bf16_full_loss_grad(name):
    st = setup(name)
    w, inp = st["w"], st["inp"]
    loss, grad = st["net"].hf_loss_grad(st["W"], st["X"], st["y"])
    f_o, g_o = O.loss_grad(w.dims, w.act, inp["theta"], inp["X"], inp["y"])
    lerr = abs(float(host(loss)[0]) - f_o) / abs(f_o)
    err = rel(host(grad), g_o)
    print("%s loss rel %.2e grad rel %.2e" % (name, lerr, err))
    assert lerr <= TOL and err <= TOL


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("name", SPEECH)
def test_bf16_full_product(name, mode):
    """The stateless product at full size.  Where 256 x 256 tiles of the
    first layer cover the 256 CUs (16,384 rows here) it takes the cached
    route (the forward pass of a solve, then its product); at fewer rows the
    fused forward / R-forward kernels."""
    st = setup(name)
    w, inp = st["w"], st["inp"]
    net = st["net"]
    net.prof_enable(True)
    net.prof_reset()
    out = net.hf_hvp(st["W"], st["Xc"], st["yc"], st["v"], mode)
    host(out)
    stats = net.prof_stats()
    net.prof_enable(False)
    cached = (w.curv_batch // 256) * (w.dims[1] // 256) >= 256
    assert ("hf_hgemm_rfwd" in stats) == cached, sorted(stats)
    assert ("hf_hgemm_fwd_rfwd" in stats) != cached, sorted(stats)
    ref = O.curvature(w.dims, w.act, inp["theta"], inp["X"][:w.curv_batch],
                      inp["y"][:w.curv_batch], inp["v"], mode)
    err = rel(host(out), ref)
    print("%s %s rel %.2e (%s route)" % (name, mode, err, "cached" if cached else "fused"))
    assert err <= TOL


@pytest.mark.parametrize("mode", ["hessian", "gauss_newton"])
@pytest.mark.parametrize("name", SPEECH)
def test_bf16_full_cg(name, mode):
    st = setup(name)
    w, inp = st["w"], st["inp"]
    cap = CAPS[name][0 if mode == "hessian" else 1]
    _, g_o = O.loss_grad(w.dims, w.act, inp["theta"], inp["X"], inp["y"])
    g32 = g_o.astype(np.float32)
    _, _, gi = st["net"].hf_cg(st["W"], st["Xc"], st["yc"], dev(g32), w.damping,
                               cap, mode)
    oi = O.cg_network(w.dims, w.act, inp["theta"], inp["X"][:w.curv_batch],
                      inp["y"][:w.curv_batch], g32.astype(np.float64),
                      w.damping, cap, mode)
    print("%s %s cap %d: gpu %s | oracle iters %d neg %d/%d pBp %.4g"
          % (name, mode, cap, {k: gi[k] for k in ("iters", "products",
                                                   "neg_curv", "neg_iter", "pBp")},
             oi["iters"], oi["neg_curv"], oi["neg_iter"], oi["pBp"]))
    assert gi["iters"] == oi["iters"] and gi["products"] == oi["products"]
    assert gi["neg_curv"] == oi["neg_curv"] and gi["neg_iter"] == oi["neg_iter"]
    if oi["neg_curv"]:
        assert np.sign(gi["pBp"]) == np.sign(oi["pBp"])
        assert abs(gi["pBp"] - oi["pBp"]) <= 0.05 * abs(oi["pBp"])
