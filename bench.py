"""Benchmark of the Hessian-free curvature path on one MI355X.

One step is one pass of the whole hot path over the speech-frame-shaped
workload (440-2048x4-1973 sigmoid network, batch 16,384, Zipf(1.1) labels
over 1,973 classes, fp32):
  1. loss + gradient on the batch                      (Alg. 1 step 1)
  2. one exact Hessian-vector product H v              (Sec. 2.1)
  3. one Gauss-Newton product G v                      (Sec. 2.1)
  4. CG-Minimize on G + lambda I, 50 iterations        (Alg. 1 steps 3-4)
  5. CG-Minimize on H + lambda I, up to 50 iterations, stopping at the first
     negative-curvature direction                      (Sec. 2.1, 2.2)
with lambda = 1e-2 and all inputs resident in HBM before timing starts.

value = curvature-vector products per second over the timed steps (the
stateless H v and G v plus every product inside both CG solves), with fp32
GEMMs.  The same step is then timed with bf16 GEMM operands and fp32
accumulation (reported under "bf16_inputs").  After each leg's timed steps,
10 Bi-CG-STAB iterations (Alg. 3) and one full outer iteration (Alg. 2:
gradient, Hessian CG, direction choice, Armijo line search) are timed on
their own, and once more on the Gauss-Newton matrix with CG-backtracking
over 16 kept iterates and the damping adjustment, unpreconditioned and (fp32
only) with Martens' diagonal preconditioner.

Prints one JSON line (rank 0; there is only one GPU).
"""

import argparse
import json
import math
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("curvature-vector products/sec (Hv & Gv) at batch B; "
          "CG iteration ms; % MFMA peak")
PEAK_FP32_TFLOPS = 157.3      # MI355X dense fp32 matrix peak
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
DEFAULT_WORKLOAD = "speech_440_2048x4_1973_sigmoid_b16384"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-share", action="store_true",
                    help="skip the one-worker-share CG timing")
    ap.add_argument("--no-bf16", action="store_true",
                    help="skip the bf16-operand leg")
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="rows of the curvature batch the oracle sample uses "
                         "(0 = all of them)")
    ap.add_argument("--timed-events", choices=("dominant", "none"), default="dominant",
                    help="dominant: the timed steps carry kernel events on the "
                         "dominant GEMM (the roofline is measured over them); "
                         "none: no events in the timed steps, so that CG replays "
                         "its captured iteration (the roofline then comes from "
                         "the fully profiled step)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, copy a buffer of this many MiB with a "
                         "plain device copy (reference point for HBM counters)")
    return ap.parse_args()


def counter_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None when the summary was taken on
    another workload, does not cover the kernel, or its GEMM source
    (gemm.hip, or gemm_bf16.hip for the bf16 kernels) has changed since the
    counters were taken."""
    import hashlib
    bf16 = kernel.startswith("hf_hgemm")
    path = os.path.join(ROOT, "profiles", "speech_b16384_hbm_counters.md")
    src = os.path.join(ROOT, "paper_1606_00511_amd", "csrc",
                       "gemm_bf16.hip" if bf16 else "gemm.hip")
    tag = "gemm_bf16_source_sha256" if bf16 else "gemm_source_sha256"
    try:
        lines = open(path).read().split("\n")
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    vals = {}
    for l in lines:
        t = l.split()
        if len(t) == 3 and t[0] == "traffic_bytes_per_launch":
            vals[t[1]] = float(t[2])
        if len(t) == 2 and t[0] == tag:
            vals["sha"] = t[1]
        if len(t) == 2 and t[0] == "workload":
            vals["workload"] = t[1]
    if vals.get("sha") != sha or vals.get("workload") != workload:
        return None
    return vals.get(kernel)


def cpu_model():
    """The host CPU's model name (lscpu), or None."""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    return None


def cpu_baseline(w, inp, rows, min_s=12.0, max_pairs=1000):
    """The fp64 oracle timed on this host's cores on a bounded sample: pairs
    of one H v and one G v on the first `rows` rows, repeated until at least
    min_s seconds have passed (at most max_pairs pairs), scaled to the full
    batch."""
    from oracle import hf_oracle as O
    blas = []
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        cores = max([int(i.get("num_threads", 1)) for i in info] or [1])
        blas = [{k: i.get(k) for k in ("internal_api", "version", "num_threads",
                                       "threading_layer", "architecture")}
                for i in info]
    except Exception:
        cores = len(os.sched_getaffinity(0))
    rows = w.curv_batch if rows <= 0 else min(rows, w.curv_batch)
    X, y = inp["X"][:rows], inp["y"][:rows]
    th, v = inp["theta"], inp["v"]
    pairs = 0
    t0 = time.perf_counter()
    while True:
        O.hvp(w.dims, w.act, th, X, y, v)
        O.gvp(w.dims, w.act, th, X, v)
        pairs += 1
        elapsed = time.perf_counter() - t0
        if elapsed >= min_s or pairs >= max_pairs:
            break
    scale = w.curv_batch / float(rows)
    per_product = elapsed / (2 * pairs) * scale
    what = ("the full %d-row batch" % rows if rows == w.curv_batch else
            "the first %d of %d rows, time scaled by %.0fx to the full batch"
            % (rows, w.curv_batch, scale))
    return {"value": 1.0 / per_product, "unit": "curvature-vector products/s",
            "cores": cores, "kind": "oracle", "cpu_model": cpu_model(),
            "host_cpus": len(os.sched_getaffinity(0)), "blas": blas,
            "sample": "fp64 NumPy oracle, %d x (one Hv and one Gv) on %s (%.2f s measured)"
                      % (pairs, what, elapsed)}


def run_leg(args, w, inp, prec):
    """Warm up; run one step with every kernel timed (the per-kernel
    breakdown, and which GEMM takes the most time); then time args.steps
    steps with the library's events on that GEMM alone, so that timing the
    many small kernels does not slow the timed steps.  Returns the
    measurements of this precision."""
    import torch
    from paper_1606_00511_amd.hf import HFNet

    dev = torch.device("cuda:0")
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    W, X, y, v = d(inp["theta"]), d(inp["X"]), d(inp["y"]), d(inp["v"])
    Xc, yc = X[:w.curv_batch].contiguous(), y[:w.curv_batch].contiguous()
    net = HFNet(w.dims, w.act, max(w.batch, w.curv_batch), prec=prec)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    grad = torch.empty(net.n, dtype=torch.float32, device=dev)
    hv = torch.empty_like(grad)
    gv = torch.empty_like(grad)
    step_g, nd_g = torch.empty_like(grad), torch.empty_like(grad)
    step_h, nd_h = torch.empty_like(grad), torch.empty_like(grad)
    lam = w.damping

    names = ["loss_grad", "hv", "gv", "cg_gn", "cg_hess"]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]

    def step():
        ev[0].record()
        net.hf_loss_grad(W, X, y, loss, grad)
        ev[1].record()
        net.hf_hvp(W, Xc, yc, v, "hessian", hv)
        ev[2].record()
        net.hf_hvp(W, Xc, yc, v, "gauss_newton", gv)
        ev[3].record()
        _, _, ig = net.hf_cg(W, Xc, yc, grad, lam, w.cg_iters, "gauss_newton",
                             step=step_g, neg_dir=nd_g)
        ev[4].record()
        _, _, ih = net.hf_cg(W, Xc, yc, grad, lam, w.cg_iters, "hessian",
                             step=step_h, neg_dir=nd_h)
        ev[5].record()
        return ig, ih

    def progress(msg):
        print("[bench %s] %s" % (prec, msg), file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    progress("warm-up done")
    net.prof_enable(True)
    net.prof_reset()
    step()
    torch.cuda.synchronize()
    breakdown = net.prof_stats()
    progress("profiled step done")
    gemms = {k: st for k, st in breakdown.items() if k.startswith(("hf_gemm", "hf_hgemm"))}
    dom = max(gemms, key=lambda k: gemms[k]["ms"])
    net.prof_reset()
    if args.timed_events == "none":
        net.prof_enable(False)
    else:
        net.prof_only(dom)
    comp = {k: 0.0 for k in names}
    products = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_ms = []
    for _ in range(args.steps):
        ts = time.perf_counter()
        ig, ih = step()
        products += 2 + ig["products"] + ih["products"]
        torch.cuda.synchronize()
        step_ms.append(1e3 * (time.perf_counter() - ts))
        progress("timed step %d: %.1f ms" % (len(step_ms), step_ms[-1]))
        for i, k in enumerate(names):
            comp[k] += ev[i].elapsed_time(ev[i + 1])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if args.timed_events == "none":
        stats = breakdown
    else:
        stats = net.prof_stats()
        net.prof_enable(False)

    # Bi-CG-STAB (Alg. 3) on the same curvature batch, timed on its own after
    # the steps: 10 iterations on the Hessian, two products per iteration
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    _, _, ib = net.hf_bicgstab(W, Xc, yc, grad, lam, 10, "hessian",
                               step=step_h, neg_dir=nd_h)
    e1.record()
    torch.cuda.synchronize()
    bicg_ms = e0.elapsed_time(e1)
    # one outer iteration (Alg. 2): gradient, Hessian CG from 0, direction
    # choice and Armijo line search, on a copy of the weights
    Wk = W.clone()
    dk = torch.zeros_like(grad)
    e0.record()
    it, _ = net.hf_iterate(Wk, X, y, Xc, yc, dk, solver="cg",
                           curvature="hessian", damping=lam,
                           max_iters=w.cg_iters)
    e1.record()
    torch.cuda.synchronize()
    outer = {"ms": e0.elapsed_time(e1), "direction": it["direction"],
             "alpha": it["alpha"], "evals": it["evals"], "f0": it["f0"],
             "f1": it["f1"], "solve_products": it["solve"]["products"]}
    # the same iteration on the Gauss-Newton matrix with CG-backtracking over
    # kept iterates (Sec. 2.2) and the damping adjustment (Alg. 1)
    Wk.copy_(W)
    dk.zero_()
    keep = torch.empty((16, net.n), dtype=torch.float32, device=dev)
    e0.record()
    it, _ = net.hf_iterate(Wk, X, y, Xc, yc, dk, solver="cg",
                           curvature="gauss_newton", damping=lam,
                           max_iters=w.cg_iters, adapt_damping=True, keep=keep)
    e1.record()
    torch.cuda.synchronize()
    outer_bt = {"ms": e0.elapsed_time(e1), "direction": it["direction"],
                "alpha": it["alpha"], "evals": it["evals"], "f0": it["f0"],
                "f1": it["f1"], "solve_products": it["solve"]["products"],
                "backtrack_iter": it["backtrack_iter"],
                "rho": it["rho"] if math.isfinite(it["rho"]) else None,
                "damping_next": it["damping_next"]}
    # and preconditioned (Martens' diagonal preconditioner)
    Wk.copy_(W)
    dk.zero_()
    e0.record()
    it, _ = net.hf_iterate(Wk, X, y, Xc, yc, dk, solver="cg",
                           curvature="gauss_newton", damping=lam,
                           max_iters=w.cg_iters, adapt_damping=True,
                           keep=keep, precondition=True)
    e1.record()
    torch.cuda.synchronize()
    outer_pc = {"ms": e0.elapsed_time(e1), "direction": it["direction"],
                "alpha": it["alpha"], "evals": it["evals"], "f0": it["f0"],
                "f1": it["f1"], "solve_products": it["solve"]["products"],
                "backtrack_iter": it["backtrack_iter"],
                "rho": it["rho"] if math.isfinite(it["rho"]) else None,
                "damping_next": it["damping_next"]}
    progress("extras done")
    del Wk, dk, keep
    res = dict(stats=stats, breakdown=breakdown, dom=dom, comp=comp,
               products=products, elapsed=t1 - t0,
               step_ms=step_ms,
               ig=ig, ih=ih, ib=ib, bicg_ms=bicg_ms,
               outer=outer, outer_bt=outer_bt, outer_pc=outer_pc,
               loss=float(loss.item()))
    net.close()
    del net, W, X, y, v, Xc, yc, loss, grad, hv, gv, step_g, nd_g, step_h, nd_h
    torch.cuda.empty_cache()
    return res


def one_worker_share(WL):
    """The speech net at one worker's share of a 32-worker step: the gradient
    on 4,096 rows, then CG on G + lambda I over a 1,024-row curvature batch
    for 200 iterations, with the per-iteration time split into the
    curvature product and the CG vector kernels.  The solve is timed without
    the per-kernel profiler (its two events per launch cost about 18% of
    this small batch's iteration time); a second, profiled solve gives the
    vector kernels' share."""
    import torch
    from paper_1606_00511_amd.hf import HFNet
    w = WL.WORKLOADS["speech_440_2048x4_1973_sigmoid_b4096_c1024"]
    inp = WL.make(w)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")
    W, X, y = d(inp["theta"]), d(inp["X"]), d(inp["y"])
    Xc, yc = X[:w.curv_batch].contiguous(), y[:w.curv_batch].contiguous()
    net = HFNet(w.dims, w.act, w.batch)
    loss, grad = net.hf_loss_grad(W, X, y)
    net.hf_cg(W, Xc, yc, grad, w.damping, 5, "gauss_newton")       # warm-up
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    e[0].record()
    net.hf_loss_grad(W, X, y, loss, grad)
    e[1].record()
    _, _, info = net.hf_cg(W, Xc, yc, grad, w.damping, w.cg_iters, "gauss_newton")
    e[2].record()
    torch.cuda.synchronize()
    net.prof_enable(True)
    net.prof_reset()
    _, _, info_p = net.hf_cg(W, Xc, yc, grad, w.damping, w.cg_iters, "gauss_newton")
    torch.cuda.synchronize()
    st = net.prof_stats()
    net.prof_enable(False)
    net.close()
    vec = [k for k in st if k.startswith("hf_cg_")]
    vec_ms = sum(st[k]["ms"] for k in vec)
    vec_b = sum(st[k]["bytes"] for k in vec)
    cg_ms = e[1].elapsed_time(e[2])
    it = max(info["iters"], 1)
    vec_it = vec_ms / max(info_p["iters"], 1)
    return {"workload": w.name, "grad_ms": e[0].elapsed_time(e[1]),
            "cg_iters": info["iters"], "cg_products": info["products"],
            "neg_curv": info["neg_curv"], "cg_ms": cg_ms,
            "cg_ms_per_iter": cg_ms / it,
            "vector_ms_per_iter": vec_it,
            "product_ms_per_iter": cg_ms / it - vec_it,
            "vector_GB/s": vec_b / (vec_ms * 1e-3) / 1e9 if vec_ms else None,
            "vector_frac_hbm": vec_b / (vec_ms * 1e-3) / 1e9 / PEAK_HBM_GBS
            if vec_ms else None}


def summary(res, K, peak):
    """Roofline figures of one leg: the dominant GEMM kernel by time (its
    launches timed over the timed steps), and all GEMMs together and the CG
    vector kernels (from the one fully profiled step)."""
    dom = res["dom"]
    ds = res["stats"][dom]
    achieved = ds["flops"] / (ds["ms"] * 1e-3) / 1e12
    stats = res["breakdown"]      # one step
    gemms = {k: s for k, s in stats.items() if k.startswith(("hf_gemm", "hf_hgemm"))}
    gemm_ms = sum(s["ms"] for s in gemms.values())
    gemm_fl = sum(s["flops"] for s in gemms.values())
    # the separate passes that complete split-K GEMMs (epilogue of the
    # batch-row partials, reduce of the weight-gradient partials)
    split_ms = sum(s["ms"] for k, s in stats.items()
                   if k in ("hf_splitk_epi", "hf_splitk_reduce"))
    vec = {k: s for k, s in stats.items() if k in (
        "hf_cg_dot", "hf_cg_update", "hf_cg_dir")}
    vec_ms = sum(s["ms"] for s in vec.values())
    vec_b = sum(s["bytes"] for s in vec.values())
    comp, ig, ih, ib = res["comp"], res["ig"], res["ih"], res["ib"]
    return dict(
        dom=dom, ds=ds, achieved=achieved,
        gemm_all={"tflops": gemm_fl / (gemm_ms * 1e-3) / 1e12,
                  "frac": gemm_fl / (gemm_ms * 1e-3) / 1e12 / peak,
                  "ms_per_step": gemm_ms,
                  "frac_with_split_passes":
                      gemm_fl / ((gemm_ms + split_ms) * 1e-3) / 1e12 / peak,
                  "split_pass_ms_per_step": split_ms},
        cg_vector={"GB/s": vec_b / (vec_ms * 1e-3) / 1e9 if vec_ms else None,
                   "frac_hbm": (vec_b / (vec_ms * 1e-3) / 1e9 / PEAK_HBM_GBS)
                   if vec_ms else None, "ms_per_step": vec_ms},
        components_ms={k: comp[k] / K for k in comp},
        step_ms={"median": float(np.median(res["step_ms"])),
                 "p10": float(np.percentile(res["step_ms"], 10)),
                 "p90": float(np.percentile(res["step_ms"], 90)),
                 "all": [round(t, 3) for t in res["step_ms"]]},
        cg_gn={"iters": ig["iters"], "products": ig["products"],
               "ms_per_iter": comp["cg_gn"] / K / max(ig["products"], 1)},
        cg_hess={"iters": ih["iters"], "products": ih["products"],
                 "neg_curv": ih["neg_curv"], "neg_iter": ih["neg_iter"]},
        bicgstab_hessian={"iters": ib["iters"], "products": ib["products"],
                          "neg_iter": ib["neg_iter"], "ms": res["bicg_ms"],
                          "ms_per_product": res["bicg_ms"] / max(ib["products"], 1)},
        outer_iteration=res["outer"],
        outer_iteration_gn_backtrack=res["outer_bt"],
        outer_iteration_gn_precond=res["outer_pc"],
        hv_per_s_stateless=1e3 * K / comp["hv"],
        gv_per_s_stateless=1e3 * K / comp["gv"],
        kernels={k: {"launches": s["launches"], "ms_per_step": s["ms"],
                     "avg_us": 1e3 * s["ms"] / max(s["launches"], 1),
                     "tflops": s["flops"] / max(s["ms"], 1e-9) / 1e9,
                     "gbs": s["bytes"] / max(s["ms"], 1e-9) / 1e6}
                 for k, s in sorted(stats.items(), key=lambda kv: -kv[1]["ms"])})


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU "
              "path (asked for --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1606_00511_amd import workloads as WL

    w = WL.WORKLOADS[args.workload]
    inp = WL.make(w)
    if args.copy_probe_mib > 0:
        nel = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(nel, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    K = args.steps
    r32 = run_leg(args, w, inp, "fp32")
    s32 = summary(r32, K, PEAK_FP32_TFLOPS)
    ds = s32["ds"]
    out = {
        "metric": METRIC,
        "value": r32["products"] / r32["elapsed"],
        "unit": "curvature-vector products/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * r32["elapsed"] / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "dims": list(w.dims), "act": w.act,
            "batch": w.batch, "curv_batch": w.curv_batch,
            "cg_iters": w.cg_iters, "damping": w.damping,
            "parallelism": "single GPU (one worker's share)",
        },
        "roofline": {
            "bound": "mfma", "kernel": s32["dom"],
            "achieved": s32["achieved"], "peak": PEAK_FP32_TFLOPS,
            "unit": "TFLOP/s", "frac": s32["achieved"] / PEAK_FP32_TFLOPS,
            "traffic": counter_traffic(s32["dom"], w.name),
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "launches": ds["launches"], "avg_launch_ms": ds["ms"] / ds["launches"],
            "flops_per_launch": ds["flops"] / ds["launches"],
            "measured_over": ("the timed steps" if args.timed_events == "dominant"
                              else "the fully profiled step"),
        },
        "cg_replayed": r32["ig"].get("replayed"),
        "loss": r32["loss"],
    }
    for k in ("step_ms", "gemm_all", "cg_vector", "components_ms", "cg_gn",
              "cg_hess", "bicgstab_hessian", "outer_iteration",
              "outer_iteration_gn_backtrack", "outer_iteration_gn_precond",
              "hv_per_s_stateless", "gv_per_s_stateless", "kernels"):
        out[k] = s32[k]
    if not args.no_share:
        out["one_worker_share"] = one_worker_share(WL)
    if not args.no_bf16:
        # the same step with bf16 GEMM operands (fp32 accumulation)
        r16 = run_leg(args, w, inp, "bf16")
        s16 = summary(r16, K, PEAK_BF16_TFLOPS)
        d16 = s16["ds"]
        out["bf16_inputs"] = {
            "value": r16["products"] / r16["elapsed"],
            "ms_per_step": 1e3 * r16["elapsed"] / K,
            "dtype": "bf16 operands, f32 accumulate",
            "roofline": {
                "bound": "mfma", "kernel": s16["dom"], "achieved": s16["achieved"],
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": s16["achieved"] / PEAK_BF16_TFLOPS,
                "traffic": counter_traffic(s16["dom"], w.name),
                "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "launches": d16["launches"],
                "avg_launch_ms": d16["ms"] / d16["launches"],
                "flops_per_launch": d16["flops"] / d16["launches"]},
            "loss": r16["loss"],
        }
        for k in ("step_ms", "gemm_all", "cg_vector", "components_ms", "cg_gn",
                  "cg_hess", "bicgstab_hessian", "outer_iteration",
                  "outer_iteration_gn_backtrack", "outer_iteration_gn_precond",
                  "kernels"):
            out["bf16_inputs"][k] = s16[k]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, inp, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
