"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle
checks.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic (no forward pass, no loss, no curvature product, no CG).
Both the HIP path and the fp64 oracle consume the float32/int32 arrays it
returns, so a parity error measures only the arithmetic of the side under
test.

The workloads stand in for the paper's digit-image and speech-frame data
(Sec. 3: MNIST-shaped 784-dim inputs with 10 classes; TIMIT-shaped frames
with 1,973 classes).  No item of either dataset is reproduced: inputs are
iid draws with the stated shapes and distributions.

Generation order for one workload (one ``numpy.random.Generator(PCG64)``
stream per role):
  data stream    : X (float64 draw, cast to float32, row-major), then y
  weight stream  : for each layer W_l ~ N(0, 1/fan_in) then b_l
  vector stream  : v ~ N(0, 1) over all n parameters
Seeds are ``16060511 + 10 k + {0: data, 1: weights, 2: vector}`` for the
named configuration k = 1..5.
"""

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 16060511


@dataclass(frozen=True)
class Workload:
    name: str
    dims: tuple          # (d_0, d_1, ..., d_L)
    act: str             # hidden activation: sigmoid | tanh | relu
    batch: int           # rows used for loss + gradient
    curv_batch: int      # rows used for curvature products (first rows)
    x_dist: str          # "uniform01" | "normal"
    y_dist: str          # "uniform" | "zipf1.1"
    cg_iters: int
    damping: float = 1e-2
    modes: tuple = ("hessian", "gauss_newton")
    index: int = 0
    note: str = field(default="", compare=False)


WORKLOADS = {
    "mnist_784_100_10_sigmoid_b1000": Workload(
        "mnist_784_100_10_sigmoid_b1000", (784, 100, 10), "sigmoid",
        1000, 1000, "uniform01", "uniform", 10, modes=("hessian",), index=1,
        note="digit-image shaped, 1 hidden layer"),
    "mnist_784_500x3_10_tanh_b10000": Workload(
        "mnist_784_500x3_10_tanh_b10000", (784, 500, 500, 500, 10), "tanh",
        10000, 10000, "uniform01", "uniform", 50, index=2,
        note="digit-image shaped, 4 weight layers"),
    "mnist_784_500x3_10_relu_b60000_c6000": Workload(
        "mnist_784_500x3_10_relu_b60000_c6000", (784, 500, 500, 500, 10),
        "relu", 60000, 6000, "uniform01", "uniform", 100, index=3,
        note="full synthetic digit-shaped set, curvature on a 6,000 subsample"),
    "speech_440_2048x4_1973_sigmoid_b16384": Workload(
        "speech_440_2048x4_1973_sigmoid_b16384",
        (440, 2048, 2048, 2048, 2048, 1973), "sigmoid", 16384, 16384,
        "normal", "zipf1.1", 50, index=4,
        note="speech-frame shaped: 40 coefficients x 11 frames, 1,973 classes"),
    "speech_440_2048x4_1973_sigmoid_b4096_c1024": Workload(
        "speech_440_2048x4_1973_sigmoid_b4096_c1024",
        (440, 2048, 2048, 2048, 2048, 1973), "sigmoid", 4096, 1024,
        "normal", "zipf1.1", 200, index=5,
        note="one worker's share of a 32-worker data-parallel step"),
}


def num_params(dims):
    return sum(int(dims[l]) * (int(dims[l - 1]) + 1) for l in range(1, len(dims)))


def draw_inputs(rng, rows, d0, n_classes, x_dist, y_dist):
    """X (rows x d0 float32) and labels y (int32) from one generator."""
    if x_dist == "uniform01":
        X = rng.random((rows, d0))
    elif x_dist == "normal":
        X = rng.standard_normal((rows, d0))
    else:
        raise ValueError(x_dist)
    X = np.ascontiguousarray(X.astype(np.float32))
    if y_dist == "uniform":
        y = rng.integers(0, n_classes, rows)
    elif y_dist.startswith("zipf"):
        s = float(y_dist[4:])
        w = np.arange(1, n_classes + 1, dtype=np.float64) ** (-s)
        y = rng.choice(n_classes, rows, p=w / w.sum())
    else:
        raise ValueError(y_dist)
    return X, y.astype(np.int32)


def draw_params(rng, dims, bias_std=0.0):
    """Flat float32 theta: per layer W_l ~ N(0, 1/fan_in) row-major, then
    b_l (zero unless ``bias_std`` > 0)."""
    parts = []
    for l in range(1, len(dims)):
        o, i = int(dims[l]), int(dims[l - 1])
        parts.append(rng.standard_normal(o * i) / np.sqrt(i))
        if bias_std > 0.0:
            parts.append(rng.standard_normal(o) * bias_std)
        else:
            parts.append(np.zeros(o))
    return np.ascontiguousarray(np.concatenate(parts).astype(np.float32))


def draw_vector(rng, n, scale=1.0):
    return np.ascontiguousarray((rng.standard_normal(n) * scale).astype(np.float32))


def make(workload, rows=None):
    """Inputs for a named workload: dict with X, y, theta, v (numpy)."""
    w = WORKLOADS[workload] if isinstance(workload, str) else workload
    k = w.index
    rows = w.batch if rows is None else rows
    data = np.random.Generator(np.random.PCG64(SEED_BASE + 10 * k + 0))
    wts = np.random.Generator(np.random.PCG64(SEED_BASE + 10 * k + 1))
    vec = np.random.Generator(np.random.PCG64(SEED_BASE + 10 * k + 2))
    X, y = draw_inputs(data, w.batch, w.dims[0], w.dims[-1], w.x_dist, w.y_dist)
    theta = draw_params(wts, w.dims)
    v = draw_vector(vec, num_params(w.dims))
    return dict(X=X[:rows], y=y[:rows], theta=theta, v=v, workload=w)


def make_small(dims, act, batch, seed, x_dist="uniform01", y_dist="uniform",
               bias_std=0.5, weight_scale=1.0):
    """A small seeded problem for parity tests: nonzero biases by default so
    that every bias path is exercised."""
    data = np.random.Generator(np.random.PCG64(seed))
    wts = np.random.Generator(np.random.PCG64(seed + 1))
    vec = np.random.Generator(np.random.PCG64(seed + 2))
    X, y = draw_inputs(data, batch, dims[0], dims[-1], x_dist, y_dist)
    theta = draw_params(wts, dims, bias_std)
    if weight_scale != 1.0:
        theta = (theta * np.float32(weight_scale)).astype(np.float32)
    n = num_params(dims)
    return dict(X=X, y=y, theta=theta, v=draw_vector(vec, n),
                u=draw_vector(vec, n), dims=tuple(dims), act=act)
