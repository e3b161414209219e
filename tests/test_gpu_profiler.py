"""The kernel profiler (hf_prof_*): launch counts and work per kernel name,
the retraction of the launches a stopped CG solve turned into no-ops, and
hf_prof_only, which times the launches of one name and still counts (and
retracts) every other.  The bench relies on these counts for its roofline
figures."""

import numpy as np
import pytest

from paper_1606_00511_amd import workloads as WL

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def run(h, W, X, y, g, only):
    import torch
    h.prof_enable(True)
    h.prof_reset()
    if only:
        h.prof_only(only)
    _, _, info = h.hf_cg(W, X, y, g, 1e-2, 12, "hessian")
    torch.cuda.synchronize()
    st = h.prof_stats()
    h.prof_enable(False)
    return st, info


def test_profiler_counts_and_filter():
    from paper_1606_00511_amd.hf import HFNet, HFError, HF_EINVAL
    dims, act, B = (100, 200, 150, 37), "tanh", 300
    p = WL.make_small(dims, act, B, seed=61)
    h = HFNet(dims, act, B)
    W, X, y = dev(p["theta"]), dev(p["X"]), dev(p["y"])
    _, g = h.hf_loss_grad(W, X, y)
    with pytest.raises(HFError) as ei:          # timing off
        h.prof_only("hf_gemm_rfwd")
    assert ei.value.code == HF_EINVAL
    full, info = run(h, W, X, y, g, None)
    part, info2 = run(h, W, X, y, g, "hf_gemm_rfwd")
    assert info == info2
    print(info["iters"], info["products"], info["neg_curv"],
          {k: v["launches"] for k, v in full.items()})
    # the solve stops early on negative curvature: launches queued after
    # the stop were retracted, the same way with and without the filter
    assert info["neg_curv"] == 1 and info["products"] < 12
    assert set(full) == set(part)
    for k in full:
        assert full[k]["launches"] == part[k]["launches"], k
        assert full[k]["flops"] == part[k]["flops"], k
        assert full[k]["bytes"] == part[k]["bytes"], k
        assert full[k]["ms"] > 0.0, k
        if k == "hf_gemm_rfwd":
            assert part[k]["ms"] > 0.0
        else:
            assert part[k]["ms"] == 0.0, k
    # one R-forward GEMM per layer and curvature product evaluated
    L = len(dims) - 1
    assert full["hf_gemm_rfwd"]["launches"] == L * info["products"]
    h.close()
