"""Parity bounds shared by the GPU tests.

For sigmoid and tanh the bound is the fp32 target: rel-L2 <= 1e-4 against
the fp64 oracle.  ReLU adds one term.  Its derivative 1[z > 0] is a decision
taken on a floating-point value: a pre-activation whose fp64 value lies
within the fp32 accumulation error of 0 can fall on either side in fp32, and
both outcomes are correct results of fp32 arithmetic.  The oracle brackets
those units by moving the kink to -tau and +tau; the distance between the
two bracketing results bounds what such decisions can change, and is added
to the bound.  tau = 2e-5 is more than ten times the fp32 error of a
pre-activation at the workloads' widths (about sqrt(K) * 2^-24 * |partial
sums| ~ 1e-6 after three layers).
"""

import numpy as np

TOL = 1e-4
RELU_TAU = 2e-5


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def check(gpu, ref, act, bracket=None, tol=TOL, tau=RELU_TAU):
    """Assert ||gpu - ref|| <= tol ||ref|| (+ the ReLU bracket width).

    bracket(kink) must return the oracle's result with ReLU's step at kink;
    the bracket is [-tau, +tau].  Returns (error, bound) relative to ||ref||."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    nref = max(np.linalg.norm(ref), 1e-300)
    err = np.linalg.norm(gpu - ref) / nref
    bound = tol
    if act == "relu" and bracket is not None:
        lo = np.asarray(bracket(-tau), dtype=np.float64)
        hi = np.asarray(bracket(+tau), dtype=np.float64)
        bound += np.linalg.norm(lo - hi) / nref
    assert err <= bound, "rel error %.3e above bound %.3e" % (err, bound)
    return err, bound
