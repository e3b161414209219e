"""Parity bounds shared by the GPU tests.

For sigmoid and tanh the bound is the fp32 target: rel-L2 <= 1e-4 against
the fp64 oracle.  ReLU adds one term.  Its derivative 1[z > 0] is a decision
taken on a floating-point value: a pre-activation whose fp64 value lies
within the fp32 error of 0 can fall on either side in fp32, and both
outcomes are correct results of fp32 arithmetic.

Which units are ambiguous is decided per unit, from the oracle's own fp64
operands (relu_margins).  The fp32 value of z_i = sum_k a_k w_ik + b_i
carries one rounding of relative size <= u = 2^-24 per product and per
partial sum, with random signs; over K terms they add up to an error of
standard deviation about sigma_i = u sqrt(K) sqrt(sum_k (a_k w_ik)^2)
(partial sums of terms of random sign grow like the root-sum-square), plus
what the fp32 errors of the layer's inputs carry through the weights,
sqrt(sum_k (sigma_k w_ik)^2).  A unit is bracketed when |z_i| < 8 sigma_i; a
Gaussian error beyond 8 sigma has probability about 1e-15, so over the
workloads' 10^7 units none is missed.  (A CPU fp32 GEMM of the 784-500x3-10
ReLU net at 6,000 rows measured errors up to 2.2 sigma.)  The oracle is
then run with the step of every bracketed unit forced to 0 and to 1 (the
kink moved to +8 sigma_i and -8 sigma_i, 0 elsewhere); the distance between
the two results bounds what those decisions can change, and is added to the
bound.

The bf16-operand tests keep a single margin tau = 2^-5 for every unit (the
rounding of bf16 operands, about 2^-8 of z's scale, dominates there).
"""

import numpy as np

from oracle import hf_oracle as O

TOL = 1e-4
RELU_TAU = 2e-5
U32 = 2.0 ** -24
SIGMAS = 8.0


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def relu_margins(dims, act, theta, X, sigmas=SIGMAS, u=U32):
    """Per-unit margins (one array per hidden layer, shaped like its Z) of
    the ReLU decisions of an fp32 forward pass over the rows X, or None for
    other activations."""
    if act != "relu":
        return None
    layers = O.unpack(np.asarray(theta, dtype=np.float64), dims)
    Z, A = O.forward(dims, act, theta, X)
    margins = []
    var_in = np.zeros_like(A[0])          # X is exact in fp32
    for l in range(1, len(layers)):       # hidden layers
        W, b = layers[l - 1]
        K = W.shape[1]
        W2 = (W * W).T
        var = (u * u) * (K * ((A[l - 1] ** 2) @ W2) + b * b) + var_in @ W2
        sigma = np.sqrt(var)
        margins.append(sigmas * sigma)
        var_in = var
    return margins


def check(gpu, ref, act, bracket=None, tol=TOL, tau=RELU_TAU, margins=None):
    """Assert ||gpu - ref|| <= tol ||ref|| (+ the ReLU bracket width).

    bracket(kink) must return the oracle's result with ReLU's step at kink
    (a scalar, or one array per hidden layer).  With `margins` (from
    relu_margins) the bracket is per unit, else [-tau, +tau] for every unit.
    Returns (error, bound) relative to ||ref||."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    nref = max(np.linalg.norm(ref), 1e-300)
    err = np.linalg.norm(gpu - ref) / nref
    bound = tol
    if act == "relu" and bracket is not None:
        if margins is not None:
            lo = np.asarray(bracket([-m for m in margins]), dtype=np.float64)
            hi = np.asarray(bracket(list(margins)), dtype=np.float64)
        else:
            lo = np.asarray(bracket(-tau), dtype=np.float64)
            hi = np.asarray(bracket(+tau), dtype=np.float64)
        bound += np.linalg.norm(lo - hi) / nref
    assert err <= bound, "rel error %.3e above bound %.3e" % (err, bound)
    return err, bound


def ambiguous_units(dims, act, theta, X, margins):
    """Number of units whose |z| lies inside its margin (for reports)."""
    if margins is None:
        return 0
    Z, _ = O.forward(dims, act, theta, X)
    return int(sum((np.abs(z) < m).sum() for z, m in zip(Z[:-1], margins)))
