"""Streams: every call runs on the stream the binding hands the context (the
caller's current torch stream).  Results on a non-default stream, and two
contexts working at the same time on two streams, are bit-identical to the
same calls made one after another on the default stream (every kernel sums
in a fixed order).  All streams have the default priority.
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
    return t.detach().cpu().numpy()


def run_all(h, W, X, y, v):
    """loss + gradient, H v, G v and a short Hessian CG solve."""
    f, g = h.hf_loss_grad(W, X, y)
    hv = h.hf_hvp(W, X, y, v, "hessian")
    gv = h.hf_hvp(W, X, y, v, "gauss_newton")
    step, nd, info = h.hf_cg(W, X, y, g, 1e-2, 6, "hessian")
    return [f, g, hv, gv, step, nd], info


def test_non_default_stream_matches_default():
    import torch
    from paper_1606_00511_amd.hf import HFNet
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=91)
    h = HFNet(dims, act, B)
    W, X, y, v = dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"])
    ref, iref = run_all(h, W, X, y, v)
    ref = [host(t).copy() for t in ref]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out, iout = run_all(h, W, X, y, v)
        # a torch op on the same stream sees the finished results
        total = out[2].sum()
    s.synchronize()
    for a, b in zip(ref, out):
        assert np.array_equal(a, host(b))
    assert iref == iout
    assert float(total) == pytest.approx(float(ref[2].astype(np.float64).sum()),
                                         rel=1e-5)


def test_two_contexts_on_two_streams():
    import torch
    from paper_1606_00511_amd.hf import HFNet
    cases = [((100, 200, 150, 37), "sigmoid", 300, 92),
             ((64, 1100, 10), "tanh", 2000, 93)]
    nets, data, refs = [], [], []
    for dims, act, B, seed in cases:
        p = WL.make_small(dims, act, B, seed=seed)
        h = HFNet(dims, act, B)
        d = (dev(p["theta"]), dev(p["X"]), dev(p["y"]), dev(p["v"]))
        r, info = run_all(h, *d)
        nets.append(h)
        data.append(d)
        refs.append(([host(t).copy() for t in r], info))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    outs = [None, None]
    for rep in range(3):
        for i in (0, 1):
            with torch.cuda.stream(streams[i]):
                outs[i] = run_all(nets[i], *data[i])
        for s in streams:
            s.synchronize()
        for i in (0, 1):
            res, info = outs[i]
            for a, b in zip(refs[i][0], res):
                assert np.array_equal(a, host(b)), (i, rep)
            assert info == refs[i][1]
