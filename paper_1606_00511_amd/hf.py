"""Thin ctypes binding of the C ABI in ``include/hf.h``.

Argument marshalling only: every step of the gradient, the curvature products
and CG runs in the HIP kernels of ``libhf.so``.  PyTorch provides the device
memory (the tensors and the workspace) and the stream.  There is no other
backend: without the built library every call raises.
"""

import ctypes
import os

from paper_1606_00511_amd.buildid import source_hash

HERE = os.path.dirname(os.path.abspath(__file__))
# HF_LIB_PATH names another build of the same sources (the host-sanitizer
# build of the CPU tests); by default the in-tree library.
LIB_PATH = os.environ.get("HF_LIB_PATH") or os.path.join(HERE, "libhf.so")

HF_SIGMOID, HF_TANH, HF_RELU = 0, 1, 2
HF_HESSIAN, HF_GAUSS_NEWTON, HF_HYBRID = 0, 1, 2
HF_SOLVER_CG, HF_SOLVER_BICGSTAB = 0, 1
HF_FP32, HF_BF16_INPUTS = 0, 1
HF_OK, HF_EINVAL, HF_ENOMEM, HF_EHIP, HF_ELABEL, HF_ENUMERIC, HF_EWORKSPACE = \
    0, -1, -2, -3, -4, -5, -6

ACTS = {"sigmoid": HF_SIGMOID, "tanh": HF_TANH, "relu": HF_RELU}
MODES = {"hessian": HF_HESSIAN, "gauss_newton": HF_GAUSS_NEWTON}
CURVATURES = {"hessian": HF_HESSIAN, "gauss_newton": HF_GAUSS_NEWTON,
              "hybrid": HF_HYBRID}
SOLVERS = {"cg": HF_SOLVER_CG, "bicgstab": HF_SOLVER_BICGSTAB}
PRECS = {"fp32": HF_FP32, "bf16": HF_BF16_INPUTS}

# Every function declared in include/hf.h.
EXPORTS = (
    "hf_create", "hf_destroy", "hf_set_stream", "hf_num_params",
    "hf_workspace_bytes", "hf_set_workspace", "hf_loss_grad", "hf_hvp",
    "hf_cg", "hf_pcg", "hf_fisher_diag", "hf_bicgstab", "hf_pbicgstab", "hf_loss",
    "hf_iterate",
    "hf_set_trace", "hf_build_id", "hf_hvp_noalloc", "hf_check", "hf_last_error",
    "hf_strerror", "hf_prof_enable", "hf_prof_only",
    "hf_prof_reset", "hf_prof_count", "hf_prof_get",
)


class hf_cg_info(ctypes.Structure):
    _fields_ = [
        ("iters", ctypes.c_int32), ("products", ctypes.c_int32),
        ("neg_curv", ctypes.c_int32), ("neg_iter", ctypes.c_int32),
        ("pBp", ctypes.c_double), ("pHp", ctypes.c_double),
        ("gTd", ctypes.c_double), ("rr0", ctypes.c_double),
        ("rr_final", ctypes.c_double), ("status", ctypes.c_int32),
        ("replayed", ctypes.c_int32),
    ]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class hf_iter_params(ctypes.Structure):
    _fields_ = [
        ("solver", ctypes.c_int32), ("curvature", ctypes.c_int32),
        ("damping", ctypes.c_float), ("max_iters", ctypes.c_int32),
        ("rel_tol", ctypes.c_float), ("eta", ctypes.c_float),
        ("armijo_c", ctypes.c_float), ("shrink", ctypes.c_float),
        ("max_backtracks", ctypes.c_int32), ("adapt_damping", ctypes.c_int32),
        ("keep_cap", ctypes.c_int32), ("keep_buf", ctypes.c_void_p),
        ("precondition", ctypes.c_int32), ("precond_exp", ctypes.c_float),
    ]


class hf_iter_info(ctypes.Structure):
    _fields_ = [
        ("solve", hf_cg_info), ("mode_used", ctypes.c_int32),
        ("direction", ctypes.c_int32), ("accepted", ctypes.c_int32),
        ("evals", ctypes.c_int32), ("f0", ctypes.c_double),
        ("f1", ctypes.c_double), ("alpha", ctypes.c_double),
        ("gTd", ctypes.c_double), ("backtrack_iter", ctypes.c_int32),
        ("rho", ctypes.c_double), ("damping_next", ctypes.c_double),
    ]

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "solve"}
        d["solve"] = self.solve.as_dict()
        return d


class HFError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s: %s" % (strerror(code), msg))
        self.code = code


_lib = None


def lib():
    """Load libhf.so (raises if it has not been built, or if it was built
    from sources other than those beside it)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            "libhf.so is not built (%s); run python -m paper_1606_00511_amd.build"
            % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    L.hf_build_id.restype = ctypes.c_char_p
    L.hf_build_id.argtypes = []
    built = L.hf_build_id().decode()
    want = source_hash()
    if built != want:
        raise RuntimeError(
            "libhf.so (%s) was built from other sources (build id %s, sources %s);"
            " rebuild with python -m paper_1606_00511_amd.build"
            % (LIB_PATH, built[:16], want[:16]))
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    F32, D = ctypes.c_float, ctypes.c_double
    sig = {
        "hf_create": (ctypes.c_int, [ctypes.POINTER(I32), I32, I32, I32, I64,
                                     P, ctypes.POINTER(P)]),
        "hf_destroy": (ctypes.c_int, [P]),
        "hf_set_stream": (ctypes.c_int, [P, P]),
        "hf_num_params": (I64, [P]),
        "hf_workspace_bytes": (SZ, [P, I64]),
        "hf_set_workspace": (ctypes.c_int, [P, P, SZ]),
        "hf_loss_grad": (ctypes.c_int, [P, P, P, P, I64, P, P]),
        "hf_hvp": (ctypes.c_int, [P, P, P, P, I64, P, I32, P]),
        "hf_hvp_noalloc": (ctypes.c_int, [P, P, P, P, I64, P, I32, P, P]),
        "hf_cg": (ctypes.c_int, [P, P, P, P, I64, P, F32, I32, F32, I32, P, P,
                                 ctypes.POINTER(hf_cg_info)]),
        "hf_bicgstab": (ctypes.c_int, [P, P, P, P, I64, P, F32, I32, F32, I32, P,
                                       P, ctypes.POINTER(hf_cg_info)]),
        "hf_pcg": (ctypes.c_int, [P, P, P, P, I64, P, F32, I32, F32, I32, P, P, P,
                                  ctypes.POINTER(hf_cg_info)]),
        "hf_pbicgstab": (ctypes.c_int, [P, P, P, P, I64, P, F32, I32, F32, I32, P,
                                        P, P, ctypes.POINTER(hf_cg_info)]),
        "hf_fisher_diag": (ctypes.c_int, [P, P, P, P, I64, P]),
        "hf_loss": (ctypes.c_int, [P, P, P, P, I64, P]),
        "hf_iterate": (ctypes.c_int, [P, P, P, P, I64, P, P, I64,
                                      ctypes.POINTER(hf_iter_params),
                                      ctypes.POINTER(I32), P,
                                      ctypes.POINTER(hf_iter_info)]),
        "hf_set_trace": (ctypes.c_int, [P, P, I32]),
        "hf_build_id": (ctypes.c_char_p, []),
        "hf_check": (ctypes.c_int, [P]),
        "hf_last_error": (ctypes.c_char_p, [P]),
        "hf_strerror": (ctypes.c_char_p, [I32]),
        "hf_prof_enable": (ctypes.c_int, [P, I32]),
        "hf_prof_only": (ctypes.c_int, [P, ctypes.c_char_p]),
        "hf_prof_reset": (ctypes.c_int, [P]),
        "hf_prof_count": (I32, [P]),
        "hf_prof_get": (ctypes.c_int, [P, I32, ctypes.POINTER(ctypes.c_char_p),
                                       ctypes.POINTER(I64), ctypes.POINTER(D),
                                       ctypes.POINTER(D), ctypes.POINTER(D)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def strerror(code):
    return lib().hf_strerror(code).decode()


def _ptr(t, dtype, numel, what):
    """Device pointer of a contiguous CUDA tensor, after checking it."""
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError("%s must be a CUDA tensor" % what)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (what, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    if numel is not None and t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (what, t.numel(), numel))
    return t.data_ptr()


class HFNet:
    """One context of the C library plus its torch-allocated workspace.

    dims: (d_0, ..., d_L); act: "sigmoid" | "tanh" | "relu"; max_batch: the
    largest batch any call will use; prec: "fp32" or "bf16" (bf16 GEMM
    operands, fp32 accumulation); ws_batch: size the workspace for calls of
    up to this many rows only (default max_batch).  Calls run on torch's
    current stream.
    """

    def __init__(self, dims, act, max_batch, device="cuda", prec="fp32",
                 ws_batch=None):
        import torch
        self.dims = tuple(int(d) for d in dims)
        self.act = act
        self.prec = prec
        self.max_batch = int(max_batch)
        L = lib()
        arr = (ctypes.c_int32 * len(self.dims))(*self.dims)
        h = ctypes.c_void_p()
        rc = L.hf_create(arr, len(self.dims), ACTS[act], PRECS[prec],
                         self.max_batch, None, ctypes.byref(h))
        if rc != HF_OK:
            raise HFError(rc, "hf_create rejected dims=%s act=%s max_batch=%d prec=%s"
                          % (self.dims, act, self.max_batch, prec))
        self._h = h
        self.n = int(L.hf_num_params(h))
        nbytes = int(L.hf_workspace_bytes(
            h, self.max_batch if ws_batch is None else int(ws_batch)))
        if nbytes == 0:
            raise ValueError("ws_batch %s outside [1, %d]" % (ws_batch, self.max_batch))
        self.device = torch.device(device)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self._check(L.hf_set_workspace(h, self.workspace.data_ptr(), nbytes))

    # ------------------------------------------------------------- plumbing
    def _check(self, rc):
        if rc != HF_OK:
            raise HFError(rc, lib().hf_last_error(self._h).decode())
        return rc

    def _stream(self):
        import torch
        self._check(lib().hf_set_stream(self._h, torch.cuda.current_stream(
            self.device).cuda_stream))

    def close(self):
        if getattr(self, "_h", None) is not None:
            lib().hf_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _rows(self, X):
        if X.dim() != 2 or X.shape[1] != self.dims[0]:
            raise ValueError("X must be B x %d" % self.dims[0])
        return int(X.shape[0])

    # -------------------------------------------------------------- the ABI
    def hf_loss_grad(self, W, X, y, loss=None, grad=None):
        import torch
        B = self._rows(X)
        if loss is None:
            loss = torch.empty(1, dtype=torch.float32, device=self.device)
        if grad is None:
            grad = torch.empty(self.n, dtype=torch.float32, device=self.device)
        self._stream()
        self._check(lib().hf_loss_grad(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(X, torch.float32, None, "X"), _ptr(y, torch.int32, B, "y"), B,
            _ptr(loss, torch.float32, 1, "loss"),
            _ptr(grad, torch.float32, self.n, "grad")))
        return loss, grad

    def hf_hvp(self, W, X, y, v, mode="hessian", out=None):
        import torch
        B = self._rows(X)
        if out is None:
            out = torch.empty(self.n, dtype=torch.float32, device=self.device)
        self._stream()
        self._check(lib().hf_hvp(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(X, torch.float32, None, "X"),
            _ptr(y, torch.int32, B, "y") if y is not None else None, B,
            _ptr(v, torch.float32, self.n, "v"), MODES[mode],
            _ptr(out, torch.float32, self.n, "out")))
        return out

    def hf_cg(self, W, Xc, yc, g, damping, max_iters, mode="hessian",
              rel_tol=0.0, step=None, neg_dir=None):
        return self._solve("hf_cg", W, Xc, yc, g, damping, max_iters, mode,
                           rel_tol, step, neg_dir)

    def hf_bicgstab(self, W, Xc, yc, g, damping, max_iters, mode="hessian",
                    rel_tol=0.0, step=None, neg_dir=None):
        return self._solve("hf_bicgstab", W, Xc, yc, g, damping, max_iters,
                           mode, rel_tol, step, neg_dir)

    def _solve(self, fn, W, Xc, yc, g, damping, max_iters, mode, rel_tol, step,
               neg_dir):
        import torch
        B = self._rows(Xc)
        if step is None:
            step = torch.empty(self.n, dtype=torch.float32, device=self.device)
        if neg_dir is None:
            neg_dir = torch.empty(self.n, dtype=torch.float32, device=self.device)
        info = hf_cg_info()
        self._stream()
        rc = getattr(lib(), fn)(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(Xc, torch.float32, None, "Xc"),
            _ptr(yc, torch.int32, B, "yc") if yc is not None else None, B,
            _ptr(g, torch.float32, self.n, "g"), float(damping), int(max_iters),
            float(rel_tol), MODES[mode], _ptr(step, torch.float32, self.n, "step"),
            _ptr(neg_dir, torch.float32, self.n, "neg_dir"), ctypes.byref(info))
        self._check(rc)
        return step, neg_dir, info.as_dict()

    def hf_pcg(self, W, Xc, yc, g, minv, damping, max_iters, mode="hessian",
               rel_tol=0.0, step=None, neg_dir=None):
        """CG preconditioned by diag(minv) = M^-1 (hf_pcg)."""
        return self._psolve("hf_pcg", W, Xc, yc, g, minv, damping, max_iters,
                            mode, rel_tol, step, neg_dir)

    def hf_pbicgstab(self, W, Xc, yc, g, minv, damping, max_iters,
                     mode="hessian", rel_tol=0.0, step=None, neg_dir=None):
        """Bi-CG-STAB preconditioned on the right by diag(minv) = M^-1
        (hf_pbicgstab)."""
        return self._psolve("hf_pbicgstab", W, Xc, yc, g, minv, damping,
                            max_iters, mode, rel_tol, step, neg_dir)

    def _psolve(self, fn, W, Xc, yc, g, minv, damping, max_iters, mode,
                rel_tol, step, neg_dir):
        import torch
        B = self._rows(Xc)
        if step is None:
            step = torch.empty(self.n, dtype=torch.float32, device=self.device)
        if neg_dir is None:
            neg_dir = torch.empty(self.n, dtype=torch.float32, device=self.device)
        info = hf_cg_info()
        self._stream()
        self._check(getattr(lib(), fn)(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(Xc, torch.float32, None, "Xc"),
            _ptr(yc, torch.int32, B, "yc") if yc is not None else None, B,
            _ptr(g, torch.float32, self.n, "g"), float(damping), int(max_iters),
            float(rel_tol), MODES[mode], _ptr(minv, torch.float32, self.n, "minv"),
            _ptr(step, torch.float32, self.n, "step"),
            _ptr(neg_dir, torch.float32, self.n, "neg_dir"), ctypes.byref(info)))
        return step, neg_dir, info.as_dict()

    def hf_fisher_diag(self, W, X, y, out=None):
        """(1/B) sum_b grad l_b^2 (hf_fisher_diag)."""
        import torch
        B = self._rows(X)
        if out is None:
            out = torch.empty(self.n, dtype=torch.float32, device=self.device)
        self._stream()
        self._check(lib().hf_fisher_diag(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(X, torch.float32, None, "X"), _ptr(y, torch.int32, B, "y"), B,
            _ptr(out, torch.float32, self.n, "out")))
        return out

    def hf_loss(self, W, X, y, loss=None):
        import torch
        B = self._rows(X)
        if loss is None:
            loss = torch.empty(1, dtype=torch.float32, device=self.device)
        self._stream()
        self._check(lib().hf_loss(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(X, torch.float32, None, "X"), _ptr(y, torch.int32, B, "y"), B,
            _ptr(loss, torch.float32, 1, "loss")))
        return loss

    def hf_iterate(self, W, X, y, Xc, yc, delta, solver="cg",
                   curvature="hessian", damping=1e-2, max_iters=10, rel_tol=0.0,
                   eta=0.0, armijo_c=1e-4, shrink=0.5, max_backtracks=20,
                   hybrid_state=0, adapt_damping=False, keep=None,
                   precondition=False, precond_exp=0.75):
        """One outer HF iteration; W and delta are updated in place.
        keep: None, or a CUDA float32 tensor of cap x n for the iterates that
        CG-backtracking keeps (cap = keep.shape[0]).  adapt_damping: report
        rho and the next lambda (info["damping_next"]).  precondition:
        the solver (PCG, or Bi-CG-STAB preconditioned on the right) with
        M = (F + lambda)^precond_exp.
        Returns (info dict, the new hybrid state)."""
        import torch
        B = self._rows(X)
        Bc = self._rows(Xc)
        cap, kbuf = 0, None
        if keep is not None:
            if keep.dim() != 2 or keep.shape[1] != self.n:
                raise ValueError("keep must be cap x %d" % self.n)
            cap = int(keep.shape[0])
            kbuf = _ptr(keep, torch.float32, None, "keep")
        prm = hf_iter_params(SOLVERS[solver], CURVATURES[curvature],
                             float(damping), int(max_iters), float(rel_tol),
                             float(eta), float(armijo_c), float(shrink),
                             int(max_backtracks), 1 if adapt_damping else 0,
                             cap, kbuf, 1 if precondition else 0,
                             float(precond_exp))
        hs = ctypes.c_int32(int(hybrid_state))
        info = hf_iter_info()
        self._stream()
        self._check(lib().hf_iterate(
            self._h, _ptr(W, torch.float32, self.n, "W"),
            _ptr(X, torch.float32, None, "X"), _ptr(y, torch.int32, B, "y"), B,
            _ptr(Xc, torch.float32, None, "Xc"),
            _ptr(yc, torch.int32, Bc, "yc") if yc is not None else None, Bc,
            ctypes.byref(prm), ctypes.byref(hs),
            _ptr(delta, torch.float32, self.n, "delta"), ctypes.byref(info)))
        return info.as_dict(), int(hs.value)

    def hf_check(self):
        self._check(lib().hf_check(self._h))

    def set_trace(self, cap):
        """Record the operand and result of the first `cap` curvature
        products of every later solve (hf_set_trace); cap = 0 turns it off.
        Returns the 2 cap x n trace tensor: row 2k the operand v of product
        k, row 2k + 1 the undamped product A v."""
        import torch
        if cap <= 0:
            self._check(lib().hf_set_trace(self._h, None, 0))
            self._trace = None
            return None
        buf = torch.full((2 * int(cap), self.n), float("nan"), dtype=torch.float32,
                         device=self.device)
        self._check(lib().hf_set_trace(self._h, buf.data_ptr(), int(cap)))
        self._trace = buf   # kept alive while tracing is on
        return buf

    # ------------------------------------------------------------ profiling
    def prof_enable(self, on=True):
        self._check(lib().hf_prof_enable(self._h, 1 if on else 0))

    def prof_only(self, name=None):
        """Time only the launches of kernel `name` (None: every kernel)."""
        self._check(lib().hf_prof_only(self._h, name.encode() if name else None))

    def prof_reset(self):
        self._check(lib().hf_prof_reset(self._h))

    def prof_stats(self):
        L = lib()
        out = {}
        for i in range(int(L.hf_prof_count(self._h))):
            name = ctypes.c_char_p()
            launches = ctypes.c_int64()
            ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
            self._check(L.hf_prof_get(self._h, i, ctypes.byref(name),
                                      ctypes.byref(launches), ctypes.byref(ms),
                                      ctypes.byref(fl), ctypes.byref(by)))
            out[name.value.decode()] = dict(launches=launches.value, ms=ms.value,
                                            flops=fl.value, bytes=by.value)
        return out
