"""fp64 CPU oracle for the Hessian-free curvature path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers, tables or pre/post-processing); the
only thing both sides consume is the seeded input generator, which holds none
of the method's arithmetic.

What is computed, and where it comes from
-----------------------------------------
Paper: He, Mudigere, Smelyanskiy, Takac, "Distributed Hessian-Free
Optimization for Deep Neural Network" (arXiv 1606.00511).

* The objective f(theta) and its gradient g_k = grad f(theta_k) (Alg. 1,
  first step; Alg. 2, gradient and reduce steps): a fully connected network
  with sigmoid / tanh / ReLU hidden units and a softmax cross-entropy output,
  averaged over the minibatch.  The paper gives the network only by its
  shapes and class counts (Sec. 3); the softmax cross-entropy objective and
  mean-over-batch are the readings recorded in the design notes.
* The exact Hessian-vector product H(theta) v.  The paper (Sec. 2.1, the
  paragraph after Alg. 1) says it is obtained by a forward-backward pass with
  the R-operator at about twice the cost of a gradient, without writing the
  equations.  Here it is the directional derivative of the gradient,
  R{grad f} = d/de grad f(theta + e v) at e = 0, carried through every step
  of backpropagation (forward-mode differentiation of the gradient program).
* The Gauss-Newton product G v (same paragraph): G = J^T H_L J, where J is
  the Jacobian of the logits with respect to theta and H_L the Hessian of the
  batch-mean cross-entropy with respect to the logits.  It is positive
  semi-definite.
* CG-Minimize on the damped operator B_k(d) = H d + lambda d (Alg. 1, steps
  3-4) minimising the quadratic model m_k (Sec. 2.1, eq. (1)), stopping when a
  conjugate direction p has p^T B_k p < 0 and returning the current iterate,
  or -g_k when that happens at the first iteration (Sec. 2.1, text after
  eq. (1)); the negative-curvature direction is oriented as
  d~ = -sgn(g^T d) d with sgn(0) = +1 (Sec. 2.2); the iteration count is a
  fixed budget (Sec. 2.2).  The CG recurrences are the textbook linear CG
  (Nocedal & Wright, cited in Sec. 1 for line-search Newton-CG).

* One outer iteration of the distributed method on one worker's share
  (Alg. 2): gradient, solve from 0 or from the warm start eta delta_{k-1},
  the choice between the solver's step and the negative-curvature direction,
  Armijo backtracking, and the Hybrid-CG curvature policy (Sec. 3).
  Optionally CG-backtracking over the solver's iterates (Sec. 2.2, after
  Martens 2010) and the damping adjustment of Alg. 1's second step.

Readings where the paper is silent (each also listed in the design notes):
mean over the batch; biases present; ReLU'(0) = 0; detection on B_k with
kappa <= 0 (the paper writes "< 0"); x_0 = 0 unless a warm start is given;
a relative-residual stop that is off by default; the outer iteration's
"best descent direction" is the candidate whose Armijo step reaches the
lower loss, the negative-curvature candidate is rescaled to the length of
the solver's step, and the Armijo constants are c = 1e-4, shrink 0.5;
CG-backtracking keeps iterates at a ratio-1.3 schedule and walks back from
the final one while f decreases; the damping rule is Levenberg-Marquardt on
the reduction ratio against the damped model m_k of eq. (1); the
preconditioner is M = (F + lambda)^(3/4) with F the batch-average squared
per-example gradient (Martens' form).

Parity pins
-----------
Every function here is pinned by ``tests/test_oracle_pins.py`` against things
other than itself: ln C at zero weights, finite differences of the loss,
brute-force Hessians from second differences, symmetry, PSD-ness, the L = 1
multinomial-logistic closed form, label independence of G v, hand-computed
CG cases, exact n-step convergence of CG against ``numpy.linalg.solve``,
the CG-backtracking rule on a hand-made sequence, rho = 1 on an exactly
quadratic objective, rho against finite-difference curvature, F against the
one-layer closed form, and preconditioned CG against plain CG on the
transformed system.
"""

import numpy as np

ACTIVATIONS = ("sigmoid", "tanh", "relu")


# ---------------------------------------------------------------- parameters
def layer_sizes(dims):
    """(d_out, d_in) for every weight layer l = 1..L."""
    return [(int(dims[l]), int(dims[l - 1])) for l in range(1, len(dims))]


def num_params(dims):
    """n = sum_l d_l (d_{l-1} + 1): W_l then b_l for every layer."""
    return sum(o * i + o for o, i in layer_sizes(dims))


def unpack(theta, dims):
    """Split the flat parameter vector into [(W_l, b_l)].

    Layout: for l = 1..L, W_l row-major (d_l x d_{l-1}) followed by b_l (d_l).
    """
    theta = np.asarray(theta, dtype=np.float64)
    out, off = [], 0
    for o, i in layer_sizes(dims):
        W = theta[off:off + o * i].reshape(o, i)
        off += o * i
        b = theta[off:off + o]
        off += o
        out.append((W, b))
    assert off == theta.size, "theta length does not match dims"
    return out


def pack(layers):
    """Inverse of ``unpack``."""
    parts = []
    for W, b in layers:
        parts.append(np.asarray(W, dtype=np.float64).ravel())
        parts.append(np.asarray(b, dtype=np.float64).ravel())
    return np.concatenate(parts)


# --------------------------------------------------------------- activations
def phi(act, z):
    """Hidden activation a = phi(z)."""
    if act == "sigmoid":
        return 1.0 / (1.0 + np.exp(-z))
    if act == "tanh":
        return np.tanh(z)
    if act == "relu":
        return np.maximum(z, 0.0)
    raise ValueError(act)


def dphi(act, z, kink=0.0):
    """phi'(z), written directly from the definition of each activation.

    ``kink`` moves ReLU's step: phi'(z) = 1[z > kink], a scalar or an array
    shaped like z (one position per unit).  The method uses kink = 0
    (ReLU'(0) = 0); tests move it to either side of 0 by each unit's fp32
    rounding margin to bound the effect of pre-activations that lie within
    that margin of 0."""
    if act == "sigmoid":
        s = 1.0 / (1.0 + np.exp(-z))
        return s * (1.0 - s)
    if act == "tanh":
        t = np.tanh(z)
        return 1.0 - t * t
    if act == "relu":
        return (z > kink).astype(np.float64)    # reading: ReLU'(0) = 0
    raise ValueError(act)


def d2phi(act, z):
    """phi''(z)."""
    if act == "sigmoid":
        s = 1.0 / (1.0 + np.exp(-z))
        return s * (1.0 - s) * (1.0 - 2.0 * s)
    if act == "tanh":
        t = np.tanh(z)
        return -2.0 * t * (1.0 - t * t)
    if act == "relu":
        return np.zeros_like(z)
    raise ValueError(act)


def _kink(kink, i):
    """ReLU step position for the pre-activations Z[i] of hidden layer i + 1:
    ``kink`` is one scalar for every unit, or a sequence holding one array
    per hidden layer, shaped like that layer's Z."""
    return kink if np.isscalar(kink) else kink[i]


# ---------------------------------------------------------------- the network
def forward(dims, act, theta, X):
    """Pre-activations Z_l and activations A_l (A_0 = X, A_L unused).

    Z_l = A_{l-1} W_l^T + b_l;  A_l = phi(Z_l) for hidden layers; Z_L are the
    logits of the softmax output.
    """
    X = np.asarray(X, dtype=np.float64)
    layers = unpack(theta, dims)
    A = [X]
    Z = []
    for l, (W, b) in enumerate(layers, start=1):
        z = A[-1] @ W.T + b
        Z.append(z)
        if l < len(layers):
            A.append(phi(act, z))
    return Z, A


def softmax(z):
    """Row softmax with the usual max shift."""
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=1, keepdims=True)


def loss(dims, act, theta, X, y):
    """f(theta) = (1/B) sum_i [logsumexp(z_i) - z_{i, y_i}]."""
    Z, _ = forward(dims, act, theta, X)
    z = Z[-1]
    y = np.asarray(y, dtype=np.int64)
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    return float(np.mean(lse - z[np.arange(z.shape[0]), y]))


def loss_grad(dims, act, theta, X, y, kink=0.0):
    """(f, g) with g = grad f by backpropagation (Alg. 1 step 1; Alg. 2)."""
    layers = unpack(theta, dims)
    Z, A = forward(dims, act, theta, X)
    B = Z[-1].shape[0]
    y = np.asarray(y, dtype=np.int64)
    P = softmax(Z[-1])
    Y = np.zeros_like(P)
    Y[np.arange(B), y] = 1.0
    f = loss(dims, act, theta, X, y)
    delta = (P - Y) / B                               # df/dZ_L
    grads = [None] * len(layers)
    for l in range(len(layers), 0, -1):               # l = L .. 1
        W, _ = layers[l - 1]
        grads[l - 1] = (delta.T @ A[l - 1], delta.sum(axis=0))
        if l > 1:
            delta = (delta @ W) * dphi(act, Z[l - 2], _kink(kink, l - 2))  # df/dZ_{l-1}
    return f, pack(grads)


def _r_forward(dims, act, theta, v, X, kink=0.0):
    """Directional derivatives RZ_l = d Z_l / de along theta + e v."""
    layers = unpack(theta, dims)
    vlayers = unpack(v, dims)
    Z, A = forward(dims, act, theta, X)
    RZ, RA = [], [np.zeros_like(A[0])]
    for l in range(1, len(layers) + 1):
        W, _ = layers[l - 1]
        V, c = vlayers[l - 1]
        rz = A[l - 1] @ V.T + c + RA[l - 1] @ W.T
        RZ.append(rz)
        if l < len(layers):
            RA.append(dphi(act, Z[l - 1], _kink(kink, l - 1)) * rz)
    return layers, vlayers, Z, A, RZ, RA


def hvp(dims, act, theta, X, y, v, kink=0.0):
    """Exact H v by the R-operator: the directional derivative of the
    backpropagation program of ``loss_grad`` (Sec. 2.1, paragraph after
    Alg. 1)."""
    layers, vlayers, Z, A, RZ, RA = _r_forward(dims, act, theta, v, X, kink)
    B = Z[-1].shape[0]
    y = np.asarray(y, dtype=np.int64)
    P = softmax(Z[-1])
    Y = np.zeros_like(P)
    Y[np.arange(B), y] = 1.0
    delta = (P - Y) / B
    # R{P} = P * (RZ - rowsum(P * RZ)); R{delta_L} = R{P} / B
    rdelta = P * (RZ[-1] - (P * RZ[-1]).sum(axis=1, keepdims=True)) / B
    out = [None] * len(layers)
    for l in range(len(layers), 0, -1):
        W, _ = layers[l - 1]
        V, _ = vlayers[l - 1]
        out[l - 1] = (rdelta.T @ A[l - 1] + delta.T @ RA[l - 1],
                      rdelta.sum(axis=0))
        if l > 1:
            e = delta @ W
            re = rdelta @ W + delta @ V
            zp = Z[l - 2]
            dp = dphi(act, zp, _kink(kink, l - 2))
            new_delta = e * dp
            rdelta = re * dp + e * d2phi(act, zp) * RZ[l - 2]
            delta = new_delta
    return pack(out)


def gvp(dims, act, theta, X, v, kink=0.0):
    """Gauss-Newton G v = J^T H_L J v (Sec. 2.1, paragraph after Alg. 1).

    J v is the R-forward pass; H_L is the Hessian of the batch-mean softmax
    cross-entropy with respect to the logits, (diag p_i - p_i p_i^T) / B per
    row; J^T is ordinary backpropagation of that vector.  No labels enter.
    """
    layers, vlayers, Z, A, RZ, RA = _r_forward(dims, act, theta, v, X, kink)
    B = Z[-1].shape[0]
    P = softmax(Z[-1])
    u = P * (RZ[-1] - (P * RZ[-1]).sum(axis=1, keepdims=True)) / B
    out = [None] * len(layers)
    for l in range(len(layers), 0, -1):
        W, _ = layers[l - 1]
        out[l - 1] = (u.T @ A[l - 1], u.sum(axis=0))
        if l > 1:
            u = (u @ W) * dphi(act, Z[l - 2], _kink(kink, l - 2))
    return pack(out)


def curvature(dims, act, theta, X, y, v, mode, kink=0.0):
    """H v for mode 'hessian', G v for mode 'gauss_newton'."""
    if mode == "hessian":
        return hvp(dims, act, theta, X, y, v, kink)
    if mode == "gauss_newton":
        return gvp(dims, act, theta, X, v, kink)
    raise ValueError(mode)


# ------------------------------------------------------------------------ CG
def sgn(x):
    """sgn(x) = 1 for x >= 0, -1 otherwise (Sec. 2.2)."""
    return 1.0 if x >= 0.0 else -1.0


def cg_minimize(apply_A, g, lam, max_iters, rel_tol=0.0, record=False,
                x0=None, snap_at=(), minv=None):
    """CG-Minimize(B_k, -g_k) with B_k(d) = A d + lam d (Alg. 1 steps 3-4).

    Minimises m_k(d) = f + g^T d + d^T B_k d / 2 (Sec. 2.1, eq. (1)) from
    d = 0, or from d = x0 (Alg. 2 allows the warm start eta delta_{k-1}; one
    extra product forms its residual).  A conjugate direction p with
    p^T B_k p <= 0 stops the solve: the current iterate is returned, or -g if
    it happened at the first iteration (Sec. 2.1, after eq. (1)), together
    with d~ = -sgn(g^T p) p (Sec. 2.2).  ``max_iters`` is the fixed iteration
    budget (Sec. 2.2); the optional relative stop compares |r|^2 with
    rel_tol^2 |g|^2.

    With ``minv`` (the diagonal of M^-1, positive) the recurrences are those
    of preconditioned CG (Martens 2010 precondition the HF solve; the paper
    lists pre-conditioning among his modifications, Sec. 2.1): z = M^-1 r,
    alpha = r.z / kappa, beta = r'.z' / r.z, p = -z + beta p.  The curvature
    test, the returned step (-g at the first iteration) and the orientation
    are unchanged, and the relative stop still compares |r|^2.

    Returns a dict with step, neg_dir (None if no detection), iters (completed
    updates of the iterate), products (curvature products evaluated,
    including the warm start's), neg_curv, neg_iter, pBp, pHp, gTd,
    rr0 (= |g|^2), rr_final, kept (a copy of the iterate after j updates
    for every j in ``snap_at`` that the solve reached) and, if ``record``,
    the list of per-iteration kappa values and directions.
    """
    g = np.asarray(g, dtype=np.float64)
    nprod0 = 0
    if x0 is None:
        x = np.zeros_like(g)
        r = g.copy()             # residual of B x + g
    else:
        x = np.asarray(x0, dtype=np.float64).copy()
        r = g + apply_A(x) + lam * x
        nprod0 = 1
    z = r if minv is None else minv * r
    p = -z
    rr = float(r @ r)
    rz = float(r @ z)
    res = dict(step=x, neg_dir=None, iters=0, products=nprod0, neg_curv=0,
               neg_iter=-1, pBp=0.0, pHp=0.0, gTd=0.0, rr0=float(g @ g),
               rr_final=rr, kappas=[], dirs=[], kept={})
    if rr == 0.0:
        return res
    for j in range(max_iters):
        q = apply_A(p) + lam * p
        kappa = float(p @ q)
        if record:
            res["kappas"].append(kappa)
            res["dirs"].append(p.copy())
        res["products"] = nprod0 + j + 1
        if kappa <= 0.0:
            d = -sgn(float(g @ p)) * p
            res.update(step=(-g.copy() if j == 0 else x), neg_dir=d,
                       iters=j, neg_curv=1, neg_iter=j, pBp=kappa,
                       pHp=kappa - lam * float(p @ p), gTd=float(g @ d),
                       rr_final=rr)
            return res
        alpha = rz / kappa
        x = x + alpha * p
        r = r + alpha * q
        rr_new = float(r @ r)
        res.update(step=x, iters=j + 1, rr_final=rr_new)
        if j + 1 in snap_at:
            res["kept"][j + 1] = x.copy()
        if rel_tol > 0.0 and rr_new <= rel_tol * rel_tol * res["rr0"]:
            return res
        z = r if minv is None else minv * r
        rz_new = float(r @ z)
        beta = rz_new / rz
        rz = rz_new
        p = -z + beta * p
    return res


def cg_network(dims, act, theta, Xc, yc, g, lam, max_iters, mode,
               rel_tol=0.0, record=False, x0=None, snap_at=(), minv=None):
    """CG-Minimize with the curvature operator of the network on the fixed
    curvature batch (Xc, yc) (Alg. 2: the product on one minibatch)."""
    def apply_A(p):
        return curvature(dims, act, theta, Xc, yc, p, mode)
    return cg_minimize(apply_A, g, lam, max_iters, rel_tol, record, x0, snap_at,
                       minv)


def fisher_diag(dims, act, theta, X, y, kink=0.0):
    """F = (1/B) sum_b grad l_b (.) grad l_b: the average over the batch of
    the squared per-example gradients (l_b the cross-entropy of example b),
    each example's gradient taken on its own (a one-row batch).  Martens'
    preconditioner (2010, Sec. 4.7) is built from this diagonal."""
    X = np.asarray(X)
    B = X.shape[0]
    F = np.zeros(num_params(dims))
    for b in range(B):
        kb = kink if np.isscalar(kink) else [k[b:b + 1] for k in kink]
        _, gb = loss_grad(dims, act, theta, X[b:b + 1], np.asarray(y)[b:b + 1],
                          kb)
        F += gb * gb
    return F / B


def fisher_diag_output_layer(dims, act, theta, X, y):
    """The output layer's blocks of fisher_diag in closed form: the gradient
    of example b's cross-entropy with respect to (W_L, b_L) is
    (p_b - e_{y_b}) times [a_b; 1], a_b the last hidden activation, so the
    weight block is (1/B) (D^2)^T (A^2) and the bias block (1/B) sum_b D_b^2,
    D = P - E.  Needs one forward pass only.  Returns (F_W, F_b)."""
    X = np.asarray(X, dtype=np.float64)
    B = X.shape[0]
    Z, A = forward(dims, act, theta, X)
    D = softmax(Z[-1])
    D[np.arange(B), np.asarray(y)] -= 1.0
    Ah = A[-1]
    return (D * D).T @ (Ah * Ah) / B, (D * D).sum(axis=0) / B


def precond_inverse(F, lam, xi=0.75):
    """The diagonal of M^-1 for M = (F + lam)^xi (Martens 2010, Sec. 4.7;
    xi = 3/4 there)."""
    return (np.asarray(F, dtype=np.float64) + lam) ** (-xi)


# ----------------------------------------------------------------- Bi-CG-STAB
def bicgstab_minimize(apply_A, g, lam, max_iters, rel_tol=0.0, record=False,
                      store=None, x0=None, snap_at=(), minv=None):
    """Bi-CG-STAB (Alg. 3) for B_k d = -g_k, B_k = A + lam I, from d = 0 or
    from d = x0 (Alg. 2: the Newton system is solved by Bi-CG-STAB from 0 or
    from the warm start eta delta_{k-1}; one extra product forms its
    residual r0 = -g - B x0).

    Each iteration follows the listing's steps in order: alpha from
    (r_j, r0*) / (A p_j, r0*), the half step s_j, the stabilisation
    coefficient gamma_j = (s_j, A s_j) / (A s_j, A s_j), the new iterate and
    residual, beta_j = (r_{j+1}, r0*) / (r_j, r0*) * alpha_j / gamma_j and the
    new direction.  Every iterate x_{j+1} is a candidate direction (Sec. 2.2):
    its curvature x^T A x (undamped operator, computed here with an explicit
    product) classifies it as a Newton-type (> 0) or negative-curvature (< 0)
    direction; the first negative-curvature candidate is returned oriented as
    d~ = -sgn(g^T x) x.

    Readings of the listing (each also in the design notes): the "IF" is a
    loop over the fixed budget ``max_iters`` (Sec. 2.2) with an optional
    relative-residual stop; r0* = r0; gamma_j is the usual omega_j; a zero
    (A p_j, r0*) or (r_{j+1}, r0*) ends the solve; A s_j = 0 gives gamma_j = 0
    (then s_j = 0 for a nonsingular operator and x_{j+1} = x_j + alpha_j p_j).

    ``kept`` holds a copy of the iterate after j iterations for every j in
    ``snap_at`` that the solve reached.

    ``store`` (identity when None) is applied to every vector the recurrences
    keep (s, x, r, p) as it is formed.  Tests pass a rounding to float32 to
    measure how far storage rounding alone moves the iterates: near a
    breakdown of the recurrences that sensitivity is large, and it sets the
    bound for comparing a float32 implementation with this fp64 one.

    With ``minv`` (the diagonal of M^-1, positive) the solve is Bi-CG-STAB
    preconditioned on the right (the pre-conditioning of Martens' HF, which
    the paper lists among his modifications in Sec. 2.1, applied to Alg. 3):
    the products are taken of p^ = M^-1 p and s^ = M^-1 s, and the iterate
    advances along them, x += alpha p^ + gamma s^; everything else is
    unchanged.  This is plain Bi-CG-STAB on B M^-1 y = -g with x = M^-1 y, so
    r stays the residual -g - B x of the original system: the candidate
    curvature, the breakdown tests and the relative stop are those of the
    unpreconditioned solve.  (Reading: the paper gives no preconditioned
    form of Alg. 3; right preconditioning is the one that keeps r.)
    """
    keep = store if store is not None else (lambda v: v)
    g = np.asarray(g, dtype=np.float64)

    def B(v):
        return apply_A(v) + lam * v

    def pre(v):
        return v if minv is None else keep(minv * v)

    nprod0 = 0
    if x0 is None:
        x = np.zeros_like(g)
        r = -g.copy()
    else:
        x = keep(np.asarray(x0, dtype=np.float64).copy())
        r = keep(-g - B(x))
        nprod0 = 1
    rs = r.copy()            # r0*
    p = r.copy()
    rho = float(r @ rs)
    rr0 = float(g @ g)       # the relative stop is against |b| = |g|
    res = dict(step=x, neg_dir=None, iters=0, products=nprod0, neg_curv=0,
               neg_iter=-1, dBd=0.0, dHd=0.0, gTd=0.0, rr0=rr0,
               rr_final=float(r @ r), curvatures=[], kept={})
    if float(r @ r) == 0.0:
        return res
    for j in range(max_iters):
        ph = pre(p)
        Ap = B(ph)
        res["products"] += 1
        den = float(Ap @ rs)
        if den == 0.0 or not np.isfinite(den):
            break
        alpha = rho / den
        s = keep(r - alpha * Ap)
        sh = pre(s)
        t = B(sh)
        res["products"] += 1
        tt = float(t @ t)
        gamma = float(s @ t) / tt if tt != 0.0 else 0.0
        x = keep(x + alpha * ph + gamma * sh)
        r = keep(s - gamma * t)
        rr = float(r @ r)
        res.update(step=x, iters=j + 1, rr_final=rr)
        if j + 1 in snap_at:
            res["kept"][j + 1] = x.copy()
        dHd = float(x @ apply_A(x))
        if record:
            res["curvatures"].append(dHd)
        if dHd < 0.0 and not res["neg_curv"]:
            d = -sgn(float(g @ x)) * x
            res.update(neg_dir=d, neg_curv=1, neg_iter=j, dHd=dHd,
                       dBd=dHd + lam * float(x @ x), gTd=float(g @ d))
        if rel_tol > 0.0 and rr <= rel_tol * rel_tol * rr0:
            break
        rho_new = float(r @ rs)
        if rho_new == 0.0 or gamma == 0.0:
            break
        beta = (rho_new / rho) * (alpha / gamma)
        p = keep(r + beta * (p - gamma * Ap))
        rho = rho_new
    return res


def bicgstab_network(dims, act, theta, Xc, yc, g, lam, max_iters, mode,
                     rel_tol=0.0, record=False, store=None, x0=None, snap_at=(),
                     minv=None):
    """Bi-CG-STAB with the network's curvature operator on (Xc, yc)."""
    def apply_A(p):
        return curvature(dims, act, theta, Xc, yc, p, mode)
    return bicgstab_minimize(apply_A, g, lam, max_iters, rel_tol, record, store,
                             x0, snap_at, minv)


# --------------------------------------------------------- outer iteration
HESSIAN, GAUSS_NEWTON, HYBRID = "hessian", "gauss_newton", "hybrid"


def backtrack_schedule(max_iters, cap):
    """Iterations (counts of completed solver updates) whose iterates
    CG-backtracking keeps: j = 1, then j <- max(j + 1, ceil(1.3 j)), the
    geometric spacing with ratio 1.3 of Martens (2010, Sec. 4.6), which the
    paper cites for CG-backtracking (Sec. 2.2).  The ceiling is taken in
    integer arithmetic, ceil(13 j / 10).  Only j < max_iters are listed (the
    final iterate is always a candidate), and at most ``cap`` of them, the
    latest ones."""
    J, j = [], 1
    while j < max_iters:
        J.append(j)
        j = max(j + 1, (13 * j + 9) // 10)
    return J[-cap:] if cap > 0 else []


def cg_backtrack(f, chain):
    """CG-backtracking (Martens 2010, Sec. 4.6; the paper's Sec. 2.2 takes
    the solver's iterates as its candidates): ``chain`` lists (j, x_j) from
    the final iterate back to the earliest kept one.  The objective f is
    evaluated from the final iterate backwards for as long as it decreases;
    the last iterate before it rises again is chosen.  Returns (j, x_j,
    f(x_j), number of evaluations)."""
    j_best, x_best = chain[0]
    f_best = f(x_best)
    evals = 1
    for j, x in chain[1:]:
        fj = f(x)
        evals += 1
        if fj < f_best:
            j_best, x_best, f_best = j, x, fj
        else:
            break
    return j_best, x_best, f_best, evals


def reduction_ratio(f0, f1, g, p, Bp):
    """rho = (f(theta + p) - f(theta)) / (m_k(p) - m_k(0)), the actual over
    the predicted decrease, with the paper's quadratic model m_k of eq. (1)
    (the damped B_k).  Undefined, returned as -inf, when the model predicts
    no decrease (m_k(p) >= m_k(0))."""
    pred = float(g @ p) + 0.5 * float(p @ Bp)
    if not pred < 0.0:
        return float("-inf")
    return (f1 - f0) / pred


def adapt_damping(lam, rho):
    """Levenberg-Marquardt adjustment of lambda (Alg. 1, second step, leaves
    the rule open; this is the rule of Martens 2010, Sec. 4.1, which the
    paper cites): rho < 1/4 raises lambda by 3/2, rho > 3/4 lowers it by
    2/3, otherwise it is kept.  An iteration that accepted no step passes
    rho = -inf."""
    if rho < 0.25:
        return 1.5 * lam
    if rho > 0.75:
        return lam * (2.0 / 3.0)
    return lam


def iterate(dims, act, theta, X, y, Xc, yc, solver="cg", curvature_kind=HESSIAN,
            lam=1e-2, max_iters=10, rel_tol=0.0, eta=0.0, delta_prev=None,
            hybrid_g=False, c=1e-4, shrink=0.5, max_backtracks=20,
            damping_adapt=False, backtrack_cap=0, precondition=False, xi=0.75):
    """One iteration of the distributed HF method on one worker's share
    (Alg. 2, one k), in the paper's order:

    1. f_k and g_k on the batch (X, y).
    2. The curvature operator on the curvature batch (Xc, yc): the Hessian,
       the Gauss-Newton matrix, or Hybrid-CG (Sec. 3): the Hessian, except
       in the iteration right after a Hessian solve met negative curvature,
       which uses Gauss-Newton (``hybrid_g`` carries that across calls).
    3. The Newton system solved by CG-Minimize (Alg. 1) or Bi-CG-STAB
       (Alg. 3) with lambda damping, from 0 or from eta delta_{k-1} (Alg. 2).
    4. The candidate descent directions (Alg. 2, the step after the solve;
       Sec. 2.2): the solver's step s_k if g^T s_k < 0, and the oriented
       negative-curvature direction d~_k if one was met, rescaled to the
       length of s_k (of g_k when s_k = 0).  Reading: "the best descent
       direction" is the candidate whose Armijo step gives the lower f.
    5. For each candidate, Armijo backtracking (Alg. 2): alpha = 1, then
       alpha <- shrink alpha until f(theta + alpha delta) <= f + c alpha
       g^T delta, at most ``max_backtracks`` reductions.  c and shrink are
       not given in the paper (readings: 1e-4 and 0.5).
    6. theta_{k+1} = theta_k + alpha_k delta_k, or theta_k when no candidate
       was accepted.

    With ``precondition`` the solve is preconditioned CG, or right-
    preconditioned Bi-CG-STAB, with M = (F + lambda)^xi, F = fisher_diag on
    the batch (X, y) at theta_k.

    With ``backtrack_cap`` > 0 the solver keeps its iterates at
    backtrack_schedule(max_iters, backtrack_cap), and the step candidate of
    4. is the iterate cg_backtrack chooses among them and the final one; its
    objective value is the Armijo trial at alpha = 1.  With
    ``damping_adapt`` the iteration ends with rho of the accepted update
    p = alpha_k delta_k (reduction_ratio, with B_k p formed by a curvature
    product at theta_k) and the next lambda (adapt_damping).

    Returns a dict: theta (new), delta (the chosen direction, zeros when
    none), f0, f1, alpha, gTd, direction (0 step, 1 negative curvature,
    -1 none), accepted, evals (loss evaluations in backtracking and the line
    searches), trials (kind, alpha, f, Armijo bound) of every line-search
    evaluation, mode_used, hybrid_g (the state for the next call), solve
    (the solver's result), backtrack_iter (the chosen iterate's j, -1 without
    backtracking), rho (nan without damping adaptation) and lam_next.
    """
    theta = np.asarray(theta, dtype=np.float64)
    f0, g = loss_grad(dims, act, theta, X, y)
    if curvature_kind == HYBRID:
        mode = GAUSS_NEWTON if hybrid_g else HESSIAN
    else:
        mode = curvature_kind
    x0 = None
    if eta > 0.0 and delta_prev is not None:
        x0 = eta * np.asarray(delta_prev, dtype=np.float64)
    J = backtrack_schedule(max_iters, backtrack_cap) if backtrack_cap > 0 else []
    minv = None
    if precondition:
        minv = precond_inverse(fisher_diag(dims, act, theta, X, y), lam, xi)
    if solver == "cg":
        sol = cg_network(dims, act, theta, Xc, yc, g, lam, max_iters, mode,
                         rel_tol, x0=x0, snap_at=J, minv=minv)
    else:
        sol = bicgstab_network(dims, act, theta, Xc, yc, g, lam, max_iters,
                               mode, rel_tol, x0=x0, snap_at=J, minv=minv)
    s = sol["step"]
    evals = 0
    bt_iter, f_step = -1, None
    if backtrack_cap > 0:
        chain = [(sol["iters"], s)] + [(j, sol["kept"][j])
                                       for j in sorted(sol["kept"], reverse=True)
                                       if j < sol["iters"]]
        bt_iter, s_bt, f_step, evals = cg_backtrack(
            lambda x: loss(dims, act, theta + x, X, y), chain)
    else:
        s_bt = s
    cands = []
    if float(g @ s_bt) < 0.0:
        cands.append((0, s_bt))
    if sol["neg_curv"]:
        d = sol["neg_dir"]
        ns = float(np.linalg.norm(s))
        target = ns if ns > 0.0 else float(np.linalg.norm(g))
        nd = float(np.linalg.norm(d))
        if nd > 0.0:
            cands.append((1, d * (target / nd)))
    best = None
    trials = []
    for kind, d in cands:
        gTd = float(g @ d)
        alpha = 1.0
        for b in range(max_backtracks + 1):
            if kind == 0 and b == 0 and f_step is not None:
                ft = f_step          # known from backtracking
            else:
                ft = loss(dims, act, theta + alpha * d, X, y)
                evals += 1
            trials.append((kind, alpha, ft, f0 + c * alpha * gTd))
            if ft <= f0 + c * alpha * gTd:
                if best is None or ft < best[3]:
                    best = (kind, d, alpha, ft, gTd)
                break
            alpha *= shrink
    res = dict(f0=f0, evals=evals, trials=trials, mode_used=mode, solve=sol,
               hybrid_g=(curvature_kind == HYBRID and mode == HESSIAN
                         and bool(sol["neg_curv"])),
               backtrack_iter=bt_iter, rho=float("nan"), lam_next=lam)
    if best is None:
        res.update(theta=theta.copy(), delta=np.zeros_like(theta), f1=f0,
                   alpha=0.0, gTd=0.0, direction=-1, accepted=0)
        if damping_adapt:
            res.update(rho=float("-inf"), lam_next=adapt_damping(lam, float("-inf")))
    else:
        kind, d, alpha, ft, gTd = best
        res.update(theta=theta + alpha * d, delta=d, f1=ft, alpha=alpha,
                   gTd=gTd, direction=kind, accepted=1)
        if damping_adapt:
            p = alpha * d
            Bp = curvature(dims, act, theta, Xc, yc, p, mode) + lam * p
            rho = reduction_ratio(f0, ft, g, p, Bp)
            res.update(rho=rho, lam_next=adapt_damping(lam, rho))
    return res
