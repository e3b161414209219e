/*
 * hf.h - C ABI of the MI355X (gfx950) Hessian-free curvature library.
 *
 * The library computes, for a fully connected network with sigmoid, tanh or
 * ReLU hidden units and a softmax cross-entropy output averaged over the
 * minibatch:
 *   - the objective f and gradient g_k = grad f(theta_k)       (Alg. 1, step 1)
 *   - curvature-vector products: the exact Hessian H v by the R-operator and
 *     the Gauss-Newton G v                       (Sec. 2.1, after Alg. 1)
 *   - CG-Minimize of the quadratic model m_k(d) = f + g^T d + d^T B_k d / 2
 *     with B_k(d) = A d + lambda d, A = H or G   (Alg. 1 steps 3-4, eq. (1)),
 *     stopping at the first conjugate direction with p^T B_k p <= 0 and
 *     returning the current iterate (or -g at the first iteration) and the
 *     oriented direction d~ = -sgn(g^T p) p      (Sec. 2.1 after eq. (1); Sec. 2.2)
 * on one GPU's share of a data-parallel minibatch (Alg. 2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Parameter layout (theta, v, g, H v, step, neg_dir): for l = 1..L the
 *   weight matrix W_l (d_l x d_{l-1}, row-major) followed by the bias b_l
 *   (d_l); n = sum_l d_l (d_{l-1} + 1) fp32 values.
 * X: B x d_0 row-major fp32.  y: B int32 labels in [0, d_L).
 * Every array argument is a device pointer, 16-byte aligned, owned by the
 *   caller; the library never allocates or frees device memory.  Scratch
 *   space comes from one caller-provided workspace (hf_set_workspace).
 * All device work is enqueued on the context's stream (hf_create's
 *   hip_stream, changed later with hf_set_stream; NULL = the null stream).
 *   hf_loss_grad and hf_hvp are asynchronous; hf_cg returns after its solve
 *   has finished (it synchronises the stream).
 * Return value: HF_OK or a negative HF_E* code; hf_last_error() gives the
 *   message.  Arguments are validated before any device call, so a bad
 *   argument never reaches the GPU.  No exception or abort crosses the ABI.
 * A context is not thread-safe; calls on one context must not overlap.
 */
#ifndef HF_H
#define HF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hf_ctx hf_ctx;

/* Hidden-layer activation; the output layer is always softmax. */
enum { HF_SIGMOID = 0, HF_TANH = 1, HF_RELU = 2 };
/* Curvature matrix for hf_hvp / hf_cg / hf_bicgstab; hf_iterate also takes
 * HF_HYBRID (the Hybrid-CG policy of Sec. 3). */
enum { HF_HESSIAN = 0, HF_GAUSS_NEWTON = 1, HF_HYBRID = 2 };
/* Newton-system solver of hf_iterate. */
enum { HF_SOLVER_CG = 0, HF_SOLVER_BICGSTAB = 1 };
/* Arithmetic of the GEMMs (every other step is fp32, reductions fp64):
 *   HF_FP32         fp32 operands, fp32 MFMA, fp32 accumulation;
 *   HF_BF16_INPUTS  every GEMM operand (X, W, v, the activations and deltas
 *                   of the forward, backward, R-forward and R-backward
 *                   passes) rounded to bf16 (nearest even), bf16 MFMA with
 *                   fp32 accumulation; biases, epilogues (phi, phi', phi''),
 *                   the softmax and R-softmax rows, the phi'' cache, the
 *                   weight-gradient sums and all CG arithmetic stay fp32. */
enum { HF_FP32 = 0, HF_BF16_INPUTS = 1 };

enum {
  HF_OK = 0,
  HF_EINVAL = -1,     /* bad argument (null, misaligned, out of range)      */
  HF_ENOMEM = -2,     /* host allocation failed                            */
  HF_EHIP = -3,       /* a HIP runtime call failed                         */
  HF_ELABEL = -4,     /* a label outside [0, d_L) was seen (device check)  */
  HF_ENUMERIC = -5,   /* NaN or Inf in a CG scalar                         */
  HF_EWORKSPACE = -6  /* no workspace set, or it is too small              */
};

/* Limits checked by hf_create. */
#define HF_MAX_LAYERS 16
#define HF_MAX_CLASSES 4096

/*
 * hf_create: build a context for the network d_0-d_1-...-d_L.
 *   dims      host array of n_dims = L + 1 >= 2 positive sizes; d_L is the
 *             number of classes (<= HF_MAX_CLASSES); L <= HF_MAX_LAYERS.
 *   act       HF_SIGMOID | HF_TANH | HF_RELU for hidden layers.
 *   prec      HF_FP32 or HF_BF16_INPUTS.
 *   max_batch largest B any later call may use (>= 1); every B x d_l
 *             buffer and n must stay below 2^31 elements.
 *   hip_stream a hipStream_t for all device work of the context (NULL: the
 *             null stream); hf_set_stream changes it later.
 *   out       receives the context.  Returns HF_EINVAL on bad arguments.
 * No device call is made; the context holds no device memory.
 */
int hf_create(const int32_t* dims, int32_t n_dims, int32_t act, int32_t prec,
              int64_t max_batch, void* hip_stream, hf_ctx** out);

/* Free a context (host memory, events, pinned host staging).  NULL is ok. */
int hf_destroy(hf_ctx* ctx);

/* Stream (a hipStream_t) for all later device work; NULL = null stream. */
int hf_set_stream(hf_ctx* ctx, void* hip_stream);

/* n = sum_l d_l (d_{l-1} + 1), or -1 for a NULL context. */
int64_t hf_num_params(const hf_ctx* ctx);

/* Bytes of device workspace for calls of up to `batch` rows (batch <= 0:
 * max_batch).  0 for a NULL context or batch > max_batch.  Grows with
 * batch. */
size_t hf_workspace_bytes(const hf_ctx* ctx, int64_t batch);

/* Hand the context a device workspace, 256-byte aligned, of `bytes` bytes.
 * The context lays it out for the largest batch b <= max_batch with
 * hf_workspace_bytes(ctx, b) <= bytes; later calls with more than b rows
 * return HF_EWORKSPACE (as does a workspace too small for one row).  The
 * caller keeps ownership and must keep it alive while the context uses it,
 * and must not write to it meanwhile.  Contents need no initialisation: the
 * call clears what needs clearing (for HF_BF16_INPUTS, the operand padding)
 * and synchronises the device.  A new workspace discards the old one's
 * contents (such as the cache of a solve). */
int hf_set_workspace(hf_ctx* ctx, void* dev_ptr, size_t bytes);

/*
 * hf_loss_grad: f and g = grad f at theta = W on the batch (X, y) of B rows
 * (Alg. 1 step 1; the per-node gradient of Alg. 2).
 *   W     device, n fp32 (parameter layout above)
 *   X, y  device, B x d_0 fp32 and B int32
 *   loss  device, 1 fp32: f = (1/B) sum_i [logsumexp(z_i) - z_{i,y_i}]
 *   grad  device, n fp32
 * Asynchronous.  A label outside [0, d_L) raises a device flag reported as
 * HF_ELABEL by the next hf_check or hf_cg.
 */
int hf_loss_grad(hf_ctx* ctx, const float* W, const float* X,
                 const int32_t* y, int64_t B, float* loss, float* grad);

/*
 * hf_hvp: one curvature-vector product on the batch (X, y) of B rows,
 * without damping (Sec. 2.1, paragraph after Alg. 1; the per-node product of
 * Alg. 2):
 *   mode HF_HESSIAN      out = H v, exact Hessian of f by the R-operator
 *   mode HF_GAUSS_NEWTON out = G v = J^T H_L J v (labels unused; y may be NULL)
 *   v, out device, n fp32.  Asynchronous.
 */
int hf_hvp(hf_ctx* ctx, const float* W, const float* X, const int32_t* y,
           int64_t B, const float* v, int32_t mode, float* out);

/* Result of hf_cg (host struct). */
typedef struct hf_cg_info {
  int32_t iters;      /* completed updates of the iterate                   */
  int32_t products;   /* curvature products evaluated                       */
  int32_t neg_curv;   /* 1 if the solve stopped on p^T B_k p <= 0           */
  int32_t neg_iter;   /* CG iteration j of the detection, else -1           */
  double pBp;         /* p^T B_k p at the detection (kappa)                 */
  double pHp;         /* p^T A p = kappa - lambda ||p||^2 at the detection  */
  double gTd;         /* g^T d~ for the returned direction (<= 0)           */
  double rr0;         /* ||g||^2                                            */
  double rr_final;    /* ||r||^2 at exit                                    */
  int32_t status;     /* HF_OK, HF_ENUMERIC or HF_ELABEL                    */
  int32_t replayed;   /* 1 if the iterations were replayed from one captured
                         graph of an iteration (no kernel timing, kept
                         iterates or trace on the context), else 0          */
} hf_cg_info;

/*
 * hf_cg: CG-Minimize(B_k, -g) with B_k = A + lambda I, A = H or G on the
 * fixed curvature batch (Xc, yc) of Bc rows at theta = W (Alg. 1 steps 3-4;
 * Alg. 2 builds the operator from one minibatch).
 *   g          device, n fp32: the gradient (may come from a larger batch)
 *   damping    lambda >= 0
 *   max_iters  fixed iteration budget >= 0 (Sec. 2.2)
 *   rel_tol    stop when ||r||^2 <= rel_tol^2 ||g||^2; 0 disables
 *   step       device, n fp32: the iterate at exit; -g when negative
 *              curvature is met at the first iteration (Sec. 2.1)
 *   neg_dir    device, n fp32: d~ = -sgn(g^T p) p for the detected p
 *              (Sec. 2.2), zeros when there was no detection
 *   info       host struct, filled on return
 * Starts from x_0 = 0.  The loop runs on the device with device-resident
 * scalars; the call synchronises the stream before it returns.
 */
int hf_cg(hf_ctx* ctx, const float* W, const float* Xc, const int32_t* yc,
          int64_t Bc, const float* g, float damping, int32_t max_iters,
          float rel_tol, int32_t mode, float* step, float* neg_dir,
          hf_cg_info* info);

/*
 * hf_pcg: hf_cg preconditioned by the diagonal M (the pre-conditioning of
 * Martens' HF that Sec. 2.1 lists): z = M^-1 r, p_0 = -z_0,
 * alpha = r.z / p^T B_k p, beta = r'.z' / r.z, p = -z' + beta p.  The
 * detection test p^T B_k p <= 0, the returned step (-g at the first
 * iteration), the orientation of d~ and the relative stop on |r| / |g| are
 * those of hf_cg.
 *   minv   device, n fp32 (parameter layout), the diagonal of M^-1, > 0;
 *          e.g. (F + lambda)^(-3/4) with F from hf_fisher_diag
 * Other arguments, outputs and errors as for hf_cg.
 */
int hf_pcg(hf_ctx* ctx, const float* W, const float* Xc, const int32_t* yc,
           int64_t Bc, const float* g, float damping, int32_t max_iters,
           float rel_tol, int32_t mode, const float* minv, float* step,
           float* neg_dir, hf_cg_info* info);

/*
 * hf_fisher_diag: out = (1/B) sum_b grad l_b (.) grad l_b, the batch average
 * of the squared per-example gradients of the cross-entropy l_b of example
 * b (parameter layout; the diagonal Martens' preconditioner is built from).
 * One forward and one backward pass; the weight blocks are the weight-
 * gradient contraction of squared operands (HF_BF16_INPUTS: of the bf16
 * operands squared and rounded to bf16 again, accumulated in fp32).
 * X, y, B as for hf_loss_grad; out device, n fp32.  Asynchronous on the
 * context's stream.
 */
int hf_fisher_diag(hf_ctx* ctx, const float* W, const float* X,
                   const int32_t* y, int64_t B, float* out);

/*
 * hf_bicgstab: Bi-CG-STAB (Alg. 3; the solver behind the paper's results,
 * Sec. 2.1 footnote) for B_k d = -g with B_k = A + lambda I, A = H or G on
 * the fixed curvature batch (Xc, yc) of Bc rows at theta = W, from d = 0
 * with r0* = r0 (Alg. 2: "starting point 0").  Two curvature products per
 * iteration.  Every iterate x is a candidate direction (Sec. 2.2): its
 * curvature x^T A x (from x^T B x = -(g, x) - (r, x), r being the residual)
 * marks it Newton-type (> 0) or negative-curvature (< 0).
 *   step      device, n fp32: the final iterate (the Newton-system solution)
 *   neg_dir   device, n fp32: the FIRST negative-curvature candidate,
 *             oriented d~ = -sgn(g^T x) x, or zeros if none was met
 *   info      iters = completed iterations, products = curvature products,
 *             neg_curv / neg_iter = whether and at which iteration the first
 *             negative-curvature candidate appeared, pBp = d~^T B d~,
 *             pHp = d~^T A d~ (< 0), gTd = g^T d~ (< 0), rr0 = |g|^2,
 *             rr_final = |r|^2 at exit
 * The solve runs max_iters iterations unless the relative residual falls
 * below rel_tol (0 disables) or a denominator of the recurrences vanishes
 * ((A p, r0*) = 0 or (r, r0*) = 0; A s = 0 takes gamma = 0).  Arguments as
 * for hf_cg; the call synchronises the stream before it returns.
 */
int hf_bicgstab(hf_ctx* ctx, const float* W, const float* Xc, const int32_t* yc,
                int64_t Bc, const float* g, float damping, int32_t max_iters,
                float rel_tol, int32_t mode, float* step, float* neg_dir,
                hf_cg_info* info);

/*
 * hf_pbicgstab: hf_bicgstab preconditioned on the right by the diagonal M
 * (Martens' pre-conditioning, listed in Sec. 2.1, applied to Alg. 3; the
 * paper gives no preconditioned form, and right preconditioning is the one
 * that keeps the residual of the original system).  It is Bi-CG-STAB on
 * B_k M^-1 y = -g with d = M^-1 y: the two products of an iteration are
 * taken of M^-1 p and M^-1 s, and the iterate advances along them,
 * x += alpha M^-1 p + gamma M^-1 s.  r stays -g - B_k x, so the candidate
 * curvature, the breakdown tests and the relative stop on |r| / |g| are
 * those of hf_bicgstab.
 *   minv   device, n fp32 (parameter layout), the diagonal of M^-1, > 0
 * Other arguments, outputs and errors as for hf_bicgstab.
 */
int hf_pbicgstab(hf_ctx* ctx, const float* W, const float* Xc,
                 const int32_t* yc, int64_t Bc, const float* g, float damping,
                 int32_t max_iters, float rel_tol, int32_t mode,
                 const float* minv, float* step, float* neg_dir,
                 hf_cg_info* info);

/*
 * hf_loss: the objective alone, f = (1/B) sum_i [logsumexp(z_i) - z_{i,y_i}]
 * at theta = W on the batch (X, y) of B rows (the forward pass only; the
 * line search of Alg. 2 evaluates it at trial points).
 *   loss  device, 1 fp32.  Asynchronous; labels checked as in hf_loss_grad.
 */
int hf_loss(hf_ctx* ctx, const float* W, const float* X, const int32_t* y,
            int64_t B, float* loss);

/* Parameters of hf_iterate (host struct). */
typedef struct hf_iter_params {
  int32_t solver;         /* HF_SOLVER_CG or HF_SOLVER_BICGSTAB              */
  int32_t curvature;      /* HF_HESSIAN, HF_GAUSS_NEWTON or HF_HYBRID         */
  float damping;          /* lambda >= 0                                      */
  int32_t max_iters;      /* solver iteration budget >= 0 (Sec. 2.2)         */
  float rel_tol;          /* relative residual stop against |g|, 0 = off     */
  float eta;              /* warm start x0 = eta * delta; 0 starts from 0    */
  float armijo_c;         /* c of the Armijo condition, in (0, 1)            */
  float shrink;           /* step reduction per rejected trial, in (0, 1)    */
  int32_t max_backtracks; /* reductions tried per candidate, >= 0            */
  int32_t adapt_damping;  /* 1: compute rho and the next lambda (LM rule)   */
  int32_t keep_cap;       /* CG-backtracking: iterates kept, 0 = off        */
  float* keep_buf;        /* device, keep_cap * n fp32, caller-owned         */
  int32_t precondition;   /* 1: preconditioned solve, M = (F + lambda)^xi   */
  float precond_exp;      /* xi >= 0 (Martens: 3/4)                          */
} hf_iter_params;

/* Result of hf_iterate (host struct). */
typedef struct hf_iter_info {
  hf_cg_info solve;       /* the solve; products include the warm start's   */
  int32_t mode_used;      /* HF_HESSIAN or HF_GAUSS_NEWTON                    */
  int32_t direction;      /* 0 the solver's step, 1 the negative-curvature
                             direction, -1 no candidate accepted            */
  int32_t accepted;       /* 1 if a step satisfied the Armijo condition      */
  int32_t evals;          /* objective evaluations in the line searches      */
  double f0, f1;          /* f before and after (f1 = f0 if none accepted)   */
  double alpha;           /* accepted step length, 0 if none                */
  double gTd;             /* g^T delta for the chosen direction             */
  int32_t backtrack_iter; /* solver iterate chosen by backtracking, -1 off  */
  double rho;             /* reduction ratio (-inf: undefined; nan: off)    */
  double damping_next;    /* lambda for the next iteration                  */
} hf_iter_info;

/*
 * hf_iterate: one iteration of the distributed HF method on one worker's
 * share (Alg. 2, one k; Alg. 1):
 *   1. f and g at theta = W on the batch (X, y) of B rows;
 *   2. the curvature on the batch (Xc, yc) of Bc rows: H, G, or HF_HYBRID:
 *      H, except in the iteration right after a Hessian solve that met
 *      negative curvature, which uses G (Sec. 3); *hybrid_state carries
 *      this between calls (in/out, 0 initially; ignored otherwise);
 *   3. the Newton system (A + lambda I) d = -g by CG-Minimize (Alg. 1) or
 *      Bi-CG-STAB (Alg. 3), from 0 or from eta * delta (Alg. 2);
 *   4. the candidate directions (Sec. 2.2): the solver's step if
 *      g^T step < 0, and the oriented negative-curvature direction if one
 *      was met, rescaled to the step's length (to |g| if the step is 0);
 *   5. for each candidate, Armijo backtracking (Alg. 2): alpha = 1, then
 *      alpha *= shrink until f(W + alpha d) <= f + c alpha g^T d, at most
 *      max_backtracks reductions; the candidate reaching the lower f wins;
 *   6. W += alpha d in place, and delta = d (zeros if none was accepted).
 * CG-backtracking (keep_cap > 0; Sec. 2.2 takes the solver's iterates as
 * candidates for it, after Martens 2010): the solver keeps its iterate after
 * j updates for j = 1, then j <- max(j + 1, ceil(13 j / 10)), j < max_iters,
 * the latest keep_cap of them, in keep_buf (keep_cap consecutive vectors of
 * n floats, overwritten).  f is then evaluated from the final iterate
 * backwards while it decreases; the last iterate before it rises replaces
 * the solver's step in 4., and its f serves as the Armijo trial at
 * alpha = 1.  Damping (adapt_damping = 1; Alg. 1 adjusts lambda in its
 * second step): rho = (f1 - f0) / (m(p) - m(0)) for the accepted update
 * p = alpha d, with m the damped quadratic model of eq. (1) and B p from one
 * stateless curvature product at the old W; damping_next = 3/2 lambda if
 * rho < 1/4 (also when nothing was accepted or m(p) >= m(0), reported as
 * rho = -inf), 2/3 lambda if rho > 3/4, else lambda.  Without it rho is NaN
 * and damping_next = damping.  Preconditioning (precondition = 1;
 * damping > 0 only): the gradient pass of 1. also forms F as hf_fisher_diag
 * does on (X, y), and the solve of 3. is hf_pcg or hf_pbicgstab with
 * M^-1 = (F + lambda)^(-xi).
 *   W      device, n fp32, in/out.  X, y / Xc, yc as for hf_loss_grad /
 *          hf_cg (yc may be NULL only for HF_GAUSS_NEWTON).
 *   delta  device, n fp32, in/out: delta_{k-1} in, delta_k out.
 * The objective values that decide the line search are reduced in fp64.
 * Synchronises the stream; uses the workspace's solver vectors.
 */
int hf_iterate(hf_ctx* ctx, float* W, const float* X, const int32_t* y,
               int64_t B, const float* Xc, const int32_t* yc, int64_t Bc,
               const hf_iter_params* params, int32_t* hybrid_state,
               float* delta, hf_iter_info* info);

/*
 * hf_set_trace: lock-step diagnostic of the solvers' curvature products.
 * Every later solve on ctx (hf_cg, hf_pcg, hf_bicgstab, hf_pbicgstab and
 * the solve inside hf_iterate) copies the operand v (for hf_pbicgstab
 * M^-1 p and M^-1 s) and the undamped result A v of each of its first
 * `cap` curvature products k into buf: slot 2k (n floats at
 * buf + 2k n) gets v, slot 2k + 1 gets A v (A = H or G of the solve, on its
 * cached curvature batch; the product B_k v of Alg. 1 step 3 is A v +
 * lambda v).  Products are numbered in the order the solve evaluates them:
 * a warm start's product is k = 0; CG's iteration j is k = j (+1 after a
 * warm start); Bi-CG-STAB's iteration j is k = 2j (on p) and 2j + 1 (on s).
 * Slots of products the solve did not evaluate are left untouched.
 *   buf  device, 2 cap n fp32, 16-byte aligned, caller-owned; it must stay
 *        alive while tracing is on.  cap = 0 (buf ignored) turns it off.
 * Returns HF_EINVAL for cap < 0 or a NULL / misaligned buffer with cap > 0.
 * Costs two vector copies per traced product.
 */
int hf_set_trace(hf_ctx* ctx, float* buf, int32_t cap);

/* SHA-256 (hex) of the sources the library was built from. */
const char* hf_build_id(void);

/* Bytes of the device scratch that hf_hvp_noalloc uses in place of a
 * workspace: one array per GPU, held until the process ends. */
#define HF_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/*
 * hf_hvp_noalloc: hf_hvp for callers that cannot allocate device memory or
 * hand over a workspace (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  It computes what hf_hvp computes, with
 * the same kernels, but its scratch is a static device array of
 * HF_NOALLOC_SCRATCH_BYTES per GPU instead of the context's workspace
 * (none needs to be set).  It makes no allocating call (no hipMalloc,
 * hipFree, memset node or host-side device allocation), is asynchronous on
 * the context's stream, and can be captured into a graph.
 *   label_err  device int32 or NULL: set to 0 by the call, then to 1 if a
 *              label outside [0, d_L) was seen (hf_hvp reports this through
 *              hf_check instead; without label_err it is not reported).
 * The scratch holds the activations, deltas and split-K partials of one
 * product at B rows (less than hf_workspace_bytes(ctx, B), which also
 * holds the solvers' vectors); a batch whose layout needs more than
 * HF_NOALLOC_SCRATCH_BYTES returns HF_EWORKSPACE before any device work.  Every call on one GPU shares that GPU's scratch and leaves
 * its contents there: calls that may overlap on one GPU (other streams,
 * other threads, other contexts) race and must be serialised by the caller.
 * The context's workspace, if any, is not touched.  Other arguments and
 * errors as for hf_hvp; the context's kernel profiler does not time it.
 */
int hf_hvp_noalloc(hf_ctx* ctx, const float* W, const float* X,
                   const int32_t* y, int64_t B, const float* v, int32_t mode,
                   float* out, int32_t* label_err);

/* Synchronise the stream and report a device-detected error (HF_ELABEL)
 * raised since the last hf_check; clears the flag. */
int hf_check(hf_ctx* ctx);

/* Message for the last failed call on ctx ("" if none); static text for a
 * NULL context. */
const char* hf_last_error(const hf_ctx* ctx);

/* Static name of an HF_* code. */
const char* hf_strerror(int32_t code);

/*
 * Kernel timing.  When enabled, every kernel launch carries a start/stop HIP
 * event pair bound to its dispatch on the context's stream, and its
 * algorithmic work (flops for the contractions, bytes for memory-bound
 * kernels) is accumulated per kernel name.  hf_prof_get synchronises the
 * stream.  hf_prof_only restricts the events to the launches of one kernel
 * name (NULL or "": every kernel; HF_EINVAL while timing is off) until it
 * is called again or timing is turned off (hf_prof_reset keeps it);
 * launches and work are still counted for every name, the others' times
 * stay 0.
 * Events cost time of their own (a few microseconds per launch), which
 * matters for small kernels.
 */
int hf_prof_enable(hf_ctx* ctx, int32_t on);
int hf_prof_only(hf_ctx* ctx, const char* name);
int hf_prof_reset(hf_ctx* ctx);
int32_t hf_prof_count(hf_ctx* ctx);
int hf_prof_get(hf_ctx* ctx, int32_t i, const char** name, int64_t* launches,
                double* total_ms, double* flops, double* bytes);

#ifdef __cplusplus
}
#endif
#endif /* HF_H */
