// Internal declarations shared by the host driver and the gfx950 kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace hfk {

// ---------------------------------------------------------------- profiling
// Every launch goes through a Launch object; when profiling is on it brackets
// the kernel with HIP events on the same stream and records its algorithmic
// work under the kernel's name.
struct Profiler;

struct Launch {
  hipStream_t stream;
  Profiler* prof;   // null when profiling is off
};

// Kernel timing: prof_begin takes a start/stop event pair for the next
// launch, which passes prof_a(L) and prof_b(L) to hipExtLaunchKernelGGL (the
// events are bound to the kernel's own dispatch, with no marker packets of
// their own); prof_end files the pair for collection.  Null events when
// profiling is off.
void prof_begin(const Launch& L, const char* name);
hipEvent_t prof_a(const Launch& L);
hipEvent_t prof_b(const Launch& L);
void prof_end(const Launch& L, const char* name, double flops, double bytes);

// ------------------------------------------------------------------- GEMM
// C[m][n] = sum_k X(m, k) * Y(n, k), where
//   X(m, k) = XK ? X[m * ldx + k] : X[k * ldx + m]
//   Y(n, k) = YK ? Y[n * ldy + k] : Y[k * ldy + n]
// Modes:
//   single  acc  = sum_{s < nseg} X[s] * Y[s]                  (K-concatenation)
//   dual    acc0 = X[0] * Y[0],  acc1 = X[1] * Y[0] + X[0] * Y[1]
//   dual0   acc0 = X[0] * Y[0],  acc1 = X[0] * Y[1]
struct GemmShape {
  int M, N, K;
  const float* X[2];
  const float* Y[2];
  int ldx, ldy;
  int nseg;          // single mode
  int splits;        // split-K factor (grid z), single mode only
  const int* skip;   // if non-null and *skip != 0 the kernel does nothing
};

enum Act { ACT_SIGMOID = 0, ACT_TANH = 1, ACT_RELU = 2 };

// Epilogue arguments (one struct; each kernel uses the fields it needs).
struct EpiArgs {
  int act;
  int hidden;            // 1: hidden layer (apply phi), 0: output layer
  const float* bias;     // b_l (forward)
  const float* rbias;    // c_l, the bias part of v (R-forward)
  float* out0;           // primary output
  float* out1;           // secondary output
  float* out2;           // tertiary output
  int ldo;               // leading dimension of out0/out1/out2
  const float* aux0;     // A_{l-1} (activation of the previous layer)
  const float* aux1;     // RZ_{l-1}
  const float* aux2;     // E_{l-1} * phi''(A_{l-1})
  int lda;               // leading dimension of aux0..aux2
  long long split_stride;  // split-K partial stride (elements)
  // weight gradient only: column sums of the first K-segment's X operand
  // (the bias part of the gradient or product): written to bias_out when
  // there is one split, else per split to bias_part[z * M + m]
  float* bias_out;
  double* bias_part;
  // scratch for split-K of the batch-row GEMMs (partials of the single-
  // product kernels when the output has too few tiles for the chip), and
  // its capacity in floats; null: never split
  float* split_buf;
  long long split_cap;
};

// Output tile (128 or 64 rows and columns) of the single-product GEMMs
// for an M x N output over K (all segments): 64 when an output side is at
// most 64 wide, or when 128 x 128 tiles could not give every compute unit a
// workgroup even split along K (at most 32 splits of at least 128).  The
// split-K choice of the weight gradients counts tiles of this size.
int gemm_tile(int M, int N, int K);


// Forward:  out0 = phi(acc + bias) (hidden) or acc + bias (logits);
// the weights come transposed (Y row-contiguous: Y[k * ldy + n])
void gemm_fwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// Forward + R-forward (dual / dual0):
//   hidden: out0 = A = phi(acc0 + b), out1 = RZ = acc1 + c,
//           out2 = RA = phi'(A) RZ;   output: out0 = acc0 + b, out1 = acc1 + c
void gemm_fwd_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// R-forward on cached activations aux0 = A_l, weights and direction
// transposed (Y row-contiguous):
//   out1 = RZ = acc + c; hidden: out2 = RA = phi'(A) RZ
void gemm_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// Backward data for the gradient: out0 = delta = acc * phi'(aux0);
//   if out2: out2 = acc * phi''(aux0) (cache for the Hessian product)
void gemm_bwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// Backward + R-backward (dual): out0 = delta = acc0 phi'(a),
//   out1 = Rdelta = acc1 phi'(a) + acc0 phi''(a) RZ  (a = aux0, RZ = aux1)
void gemm_bwd_rbwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// R-backward on the cache: out1 = acc phi'(aux0) + aux2 * aux1
void gemm_rbwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// Gauss-Newton backward: out1 = acc * phi'(aux0)
void gemm_gnbwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// Weight gradient (XK = YK = false): out0[z * split_stride + m * ldo + n] = acc,
// plus the bias sums sum_k X[0](m, k) (see EpiArgs::bias_out / bias_part)
void gemm_wgrad(const Launch& L, const GemmShape& s, const EpiArgs& e);
// The same with every operand element squared (sum_k X^2 Y^2; bias sums of
// X[0]^2)
void gemm_wgrad_sq(const Launch& L, const GemmShape& s, const EpiArgs& e);

// ------------------------------------------------- narrow-net product
// The cached curvature product up to the weight gradients in one launch
// (or two: layer 1 in tiles, then the row-local rest), for nets with
// 2 <= L <= NARROW_MAX_LAYERS, at most NARROW_MAX_INPUT inputs, hidden
// layers at most NARROW_MAX_HIDDEN wide and at most 64 classes
// (narrow.hip): 16 or 4 batch rows per workgroup with every intermediate
// row in LDS.  Writes Rdelta_l
// (l = 1..L, leading dimensions ld[l]) and, for the Hessian, RA_l
// (l = 1..L-1), which the weight-gradient GEMMs then read.  Pointers per
// layer index l; the cache (A_l, P, delta_l, E2_l) is that of a solve.
constexpr int NARROW_MAX_HIDDEN = 128;
constexpr int NARROW_MAX_LAYERS = 4;
constexpr int NARROW_MAX_INPUT = 1024;     // d_0 (the rows of X sit in LDS)
struct NarrowArgs {
  int L, B, act, hess;
  int d[NARROW_MAX_LAYERS + 1];
  int ld[NARROW_MAX_LAYERS + 1];
  long long offW[NARROW_MAX_LAYERS + 1], offB[NARROW_MAX_LAYERS + 1];
  const float* X;                         // B x d_0, row-major
  const float* W;                         // parameters
  const float* v;                         // direction
  const float* A[NARROW_MAX_LAYERS + 1];  // A_l, l = 1..L-1
  const float* P;                         // softmax probabilities
  const float* D[NARROW_MAX_LAYERS + 1];  // delta_l, l = 2..L (Hessian)
  const float* E2[NARROW_MAX_LAYERS + 1]; // E2_l, l = 1..L-1 (Hessian)
  float* RA[NARROW_MAX_LAYERS + 1];       // out: RA_l (Hessian)
  float* RD[NARROW_MAX_LAYERS + 1];       // out: Rdelta_l
  float* RZ1;                             // RZ_1 (B x ld[1]): the 4-row form
                                          // writes it, then reads it
  int ldRA, ldRD;                         // their leading dimensions (0: ld[l])
  float invB;
  const int* skip;
};
// most per-block partials of a CG vector kernel (its largest grid)
constexpr int CG_MAX_GRID = 1024;
// The weight gradients of every layer from one GEMM over concatenated
// columns: Rdelta_1 .. Rdelta_L side by side (column offset roff[l], width
// ldr) against X, A_1 .. A_{L-1} side by side (offset yoff[l - 1], width
// ldy), and for the Hessian delta_l against RA_{l-1} likewise; layer l's
// gradient is the diagonal block (roff[l], yoff[l - 1]).  narrow_scatter
// sums the GEMM's split-K partials of the diagonal blocks (and the bias
// partials of their rows) in split order and writes them in the parameter
// layout.
struct NarrowCat {
  int L, M, N;                            // M = ldr, N = ldy
  int d[NARROW_MAX_LAYERS + 1];
  int roff[NARROW_MAX_LAYERS + 1], yoff[NARROW_MAX_LAYERS + 1];
  long long offW[NARROW_MAX_LAYERS + 2], offB[NARROW_MAX_LAYERS + 1];
  long long n;                            // parameters
};
// out[i], i < n, from `splits` partials (part: splits x M x N, bpart:
// splits x M doubles).  With dot (a CG iteration's product q = out of the
// direction p) the kernel also does the work of the iteration's first
// vector kernel: the per-block partials of p.q and p.p and, for an iteration
// replayed from a graph (j = -1), the publication of its index.  Returns
// the number of partials written (0 without dot).
struct CgState;
struct CgDotFuse {
  const float* p;
  double* part;      // p.q partials at part[b], p.p at part[CG_MAX_GRID + b]
  CgState* st;
  int j;
};
int narrow_scatter(const Launch& L, const float* part, const double* bpart,
                   int splits, const NarrowCat& nc, float* out, const int* skip,
                   const CgDotFuse* dot = nullptr);
// Copies column blocks of B rows: dst_k[r * ldd + c] = src_k[r * lds_k + c]
// for c < cols_k (one launch for up to 2 NARROW_MAX_LAYERS blocks).
struct NarrowGather {
  int nblk, B, ldd[2];
  const float* src[2 * NARROW_MAX_LAYERS];
  int lds[2 * NARROW_MAX_LAYERS], cols[2 * NARROW_MAX_LAYERS];
  float* dst[2 * NARROW_MAX_LAYERS];
  int which[2 * NARROW_MAX_LAYERS];       // index into ldd
};
void narrow_gather(const Launch& L, const NarrowGather& g);
// Whether the layer widths and the alignment of X and v (16 bytes, d_0 a
// multiple of 4) admit the narrow kernel.
bool narrow_eligible(int L, const int* d, const float* X, const float* v);
void narrow_product(const Launch& L, const NarrowArgs& a);
// The cache of a solve (the activations, p and, for the Hessian, delta_l and
// E2_l) for the same nets at up to 64 x 16 rows, in two launches: A_1 in
// tiles, then 4 batch rows per workgroup through the rest; X, A_l and delta_l
// also into the concatenated columns of the weight-gradient GEMM (Ycat,
// Dcat; null: not written).  A label outside [0, C) sets *err (Hessian).
struct NarrowFwdArgs {
  int L, B, act, hess;
  int d[NARROW_MAX_LAYERS + 1];
  int ld[NARROW_MAX_LAYERS + 1];
  long long offW[NARROW_MAX_LAYERS + 1], offB[NARROW_MAX_LAYERS + 1];
  const float* X;                         // B x d_0, row-major
  const float* W;                         // parameters
  const int32_t* y;                       // labels (Hessian)
  float* A[NARROW_MAX_LAYERS + 1];        // out: A_l, l = 1..L-1 (A_1 by
                                          // the layer-1 kernel, always)
  float* P;                               // out: softmax probabilities; null:
                                          // neither P nor A_2 .. A_{L-1} stored
  float* D[NARROW_MAX_LAYERS + 1];        // out: delta_l, l = 2..L (Hessian)
  float* E2[NARROW_MAX_LAYERS + 1];       // out: E2_l, l = 1..L-1 (Hessian)
  float* Ycat;                            // out: X, A_l at column yoff[l]
  int ldy;
  int yoff[NARROW_MAX_LAYERS + 1];
  float* Dcat;                            // out: delta_l at column roff[l]
  int ldr;
  int roff[NARROW_MAX_LAYERS + 1];
  float invB;
  int* err;
  // the gradient instead (Alg. 1 step 1): delta_1 .. delta_L into Dcat; no
  // E2
  int grad;
  // non-null: labels checked and the per-row loss summed into one fp64
  // partial per 4 rows, as the softmax row kernel does (the gradient, and
  // the loss alone with hess = grad = 0)
  double* loss_part;
};
void narrow_forward(const Launch& L, const NarrowFwdArgs& a);

// --------------------------------------------------------- bf16-input GEMM
// Precision HF_BF16_INPUTS: every GEMM operand is a bf16 copy (stored as
// uint16_t, rounded to nearest even from fp32), the MFMAs accumulate in fp32
// and the epilogues compute in fp32.  Every operand is K-contiguous:
//   X(m, k) = X[m * ldx + k],  Y(n, k) = Y[n * ldy + k]
// and the kernels read without bounds checks, so each operand buffer must
// have: a leading dimension that is a multiple of 64, zeros in columns
// K .. ld, 256-byte alignment, and rows up to M (or N) rounded up to 256.
// Modes as above.
typedef uint16_t bf16_t;

struct GemmShapeH {
  int M, N, K;
  const bf16_t* X[2];
  const bf16_t* Y[2];
  int ldx, ldy;
  int nseg;
  int splits;
  const int* skip;
};

// Epilogue arguments of the bf16-input kernels.  A bf16 result is written
// row-major to h* (leading dimension ldo) and, where t* is given, transposed
// to t* (t[col * ldt + row]), the batch-contiguous copy the weight gradient
// contracts over; t* also gets zeros in rows M .. (M rounded up to 64).
// fp32 results (logits, RZ, the phi'' cache, weight gradients) go to f*
// with leading dimension ldf.  Aux buffers must have rows up to M rounded
// up to 256 (they are read unchecked and masked).
struct EpiH {
  int act;
  int hidden;
  const float* bias;
  const float* rbias;
  bf16_t* h0; bf16_t* h1; bf16_t* h2;
  bf16_t* t0; bf16_t* t1; bf16_t* t2;
  float* f0; float* f1; float* f2;
  int ldo, ldt, ldf;
  const bf16_t* a0;      // A_{l-1} (bf16, leading dimension ldo)
  const float* a1;       // RZ_{l-1} (fp32, ldf)
  const float* a2;       // E_{l-1} * phi''(A_{l-1}) (fp32, ldf)
  long long split_stride;
  float* bias_out;
  double* bias_part;
};

// Same contractions and epilogue formulas as the fp32 kernels above, with
// the outputs placed as follows:
//   fwd        hidden: A -> h0/t0; output layer: logits -> f0
//   fwd_rfwd   RZ -> f1; hidden: A -> h0/t0, RA -> h2/t2; output: logits -> f0
//              (f1 and t2 may be null for a hidden layer, as for rfwd)
//   rfwd       RZ -> f1; hidden: RA = phi'(a0) RZ -> h2/t2 (f1 and t2 may
//              be null for a hidden layer: neither is then stored)
//   bwd        delta -> h0/t0; if f2: E phi''(a0) -> f2
//   bwd_rbwd   delta -> h0/t0, Rdelta -> h1/t1
//   rbwd       Rdelta = acc phi'(a0) + a2 a1 -> h1/t1
//   gnbwd      Rdelta = acc phi'(a0) -> h1/t1
//   wgrad      acc -> f0 (+ split stride), bias sums as for gemm_wgrad
void hgemm_fwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_fwd_rfwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_rfwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_bwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_bwd_rbwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_rbwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_gnbwd(const Launch& L, const GemmShapeH& s, const EpiH& e);
void hgemm_wgrad(const Launch& L, const GemmShapeH& s, const EpiH& e);
// out[r * ldo + c] = bf16(in[r * ldi + c]), outT[c * ldt + r] = the same
// for r < R and 0 for R <= r < Rpad (R x C; either output may be null)
void cvt_bf16(const Launch& L, const float* in, int R, int C, int ldi,
              bf16_t* out, int ldo, bf16_t* outT, int ldt, int Rpad,
              const int* skip);
// outT[c * ldt + r] = in[r * ldi + c] for r < R, 0 for R <= r < Rpad (bf16
// R x C in, its transposed copy out)
void transpose_bf16(const Launch& L, const bf16_t* in, int R, int C, int ldi,
                    bf16_t* outT, int ldt, int Rpad, const int* skip);
// p[i] = bf16(p[i]^2), i < n, in place (p 16-byte aligned)
void square_bf16(const Launch& L, bf16_t* p, long long n);

// --------------------------------------------------------------- row ops
// Softmax cross-entropy over rows of Z (B x C, leading dimension ld):
//   P = softmax(Z); if y: D = (P - onehot(y)) / B and per-block loss partials
//   (double, one per 4 rows) into loss_part; bad labels set *err_flag.
void softmax_xent(const Launch& L, const float* Z, const int32_t* y, int B,
                  int C, int ld, float* P, float* D, double* loss_part,
                  int* err_flag);
// loss = sum(loss_part[0 .. nparts)) / B, in a fixed order, to loss (fp32)
// and loss64 (fp64); either may be null.
void loss_finalize(const Launch& L, const double* loss_part, int nparts,
                   int B, float* loss, double* loss64 = nullptr);
// Rdelta_L = P * (RZ - rowsum(P * RZ)) / B.
void softmax_rop(const Launch& L, const float* P, const float* RZ, int B,
                 int C, int ld, float* RD, const int* skip);
// The same written as bf16 (round to nearest even; leading dimension ldo),
// columns below C only.
void softmax_rop_h(const Launch& L, const float* P, const float* RZ, int B,
                   int C, int ld, bf16_t* RD, int ldo, const int* skip);
// Up to 16 row-major blocks transposed in one launch:
// out[i][c * ldo[i] + r] = in[i][r * ldi[i] + c] (R[i] x C[i] -> C[i] x R[i]).
struct TransposeBatch {
  static constexpr int MAX = 16;
  const float* in[MAX];
  float* out[MAX];
  int R[MAX], C[MAX], ldi[MAX], ldo[MAX];
  int n;
};
void transpose_batch(const Launch& L, const TransposeBatch& b, const int* skip);
// out[m * ldo + n] = sum_z part[z * M * N + m * N + n] and
// bout[m] = sum_z bpart[z * M + m], both in split order
void splitk_reduce(const Launch& L, const float* part, const double* bpart,
                   int splits, int M, int N, float* out, int ldo, float* bout,
                   const int* skip);

// ------------------------------------------------------------------- CG
struct CgState {
  double rr[2];        // r.r, slot = iteration parity
  double rz[2];        // r.z, z = M^-1 r (preconditioned CG), same slots
  double rr0, kappa, alpha, beta, pp, pq, gp;
  double lambda, tol2;
  int done, neg, neg_iter, iters, products, status;
  // iteration index kept on the device, for an iteration replayed from a
  // graph (the kernels then take j = -1): the dot kernel copies jn to jc,
  // the kernels after it read jc, and the direction kernel sets jn = jc + 1
  int jc, jn;
  // iteration budget (> 0): the direction kernel of iteration
  // max_iters - 1 sets done, so that iterations replayed past the budget
  // do nothing
  int max_iters;
};

int cg_grid(long long n);
int cg_part_doubles();
// x = 0, r = g, p = -g; or, from a warm start x0 with q = A x0, x = x0,
// r = g + q + lambda x0, p = -r.  neg_dir = 0; state initialised with
// rr = |r|^2 and rr0 = |g|^2.  x0 and q may be null (start from 0).
void cg_init(const Launch& L, const float* g, const float* x0, const float* q,
             float* x, float* r, float* p, float* neg_dir, long long n,
             double lambda, double tol2, double* part, CgState* st,
             const float* minv = nullptr, int max_iters = 0);
// One CG iteration j after the product q = A p has been formed:
// kappa = p.q + lambda p.p and the stop test; x += alpha p,
// r += alpha (q + lambda p); at a detection d~ = -sgn(g.p) p and, at j = 0,
// x = -g; beta = rr'/rr and p = -r + beta p.  j = -1 takes the index from
// the state (an iteration captured once and replayed); then, if hflag is
// not null (host-visible memory), the last kernel of the iteration stores
// st->done there.
// dot_blocks > 0: the product already wrote that many partials of p.q and
// p.p (and published the index), so the dot kernel is not launched.
void cg_iteration(const Launch& L, float* x, float* r, float* p, const float* q,
                  const float* g, float* neg_dir, long long n, int j,
                  double* part, CgState* st, const float* minv = nullptr,
                  int* hflag = nullptr, int dot_blocks = 0);
// With minv (device, n floats, the diagonal of M^-1) cg_init and
// cg_iteration run preconditioned CG: z = minv r, p = -z at the start,
// alpha = r.z / kappa, beta = r'.z' / r.z, p = -z' + beta p.
// minv = (F + lambda)^(-xi), elementwise in fp64
void precond_inverse(const Launch& L, const float* F, double lambda, double xi,
                     float* minv, long long n);

// ----------------------------------------------------------- Bi-CG-STAB
struct BicgState {
  double rho[2];       // (r_j, r0*), slot = iteration parity
  double rr0, rr, alpha, gamma, beta;
  double lambda, tol2;
  double dBd, dHd, gTd, coef;   // first negative-curvature candidate
  int done, status, iters, products, neg, neg_iter;
};

// y += a x (the damping term of B = A + lambda I)
void axpy(const Launch& L, float* y, const float* x, float a, long long n,
          const int* skip);
// x = 0, r = r0* = p = -g; or, from a warm start x0 with q = A x0,
// x = x0, r = r0* = p = -g - (q + lambda x0).  neg_dir = 0; state
// initialised with rho = |r0|^2 and rr0 = |g|^2.  x0, q may be null.
void bicg_init(const Launch& L, const float* g, const float* x0,
               const float* q, float* x, float* r, float* rs, float* p,
               float* neg_dir, long long n, double lambda, double tol2,
               double* part, BicgState* st, const float* minv = nullptr,
               float* ph = nullptr);
// first half of iteration j, after Ap = B p: alpha and s = r - alpha Ap
void bicg_half(const Launch& L, const float* r, const float* rs,
               const float* Ap, float* s, long long n, int j, double* part,
               BicgState* st, const float* minv = nullptr, float* sh = nullptr);
// second half, after t = B s: gamma, x, r, candidate curvature, beta, p,
// and the oriented candidate at the first negative curvature
void bicg_rest(const Launch& L, float* x, float* r, const float* rs, float* p,
               const float* Ap, const float* s, const float* t, const float* g,
               float* neg_dir, long long n, int j, double* part,
               BicgState* st, const float* minv = nullptr, float* ph = nullptr,
               const float* sh = nullptr);
// With minv (device, n floats, the diagonal of M^-1) the three run
// Bi-CG-STAB preconditioned on the right: init and rest write
// ph = minv p and half writes sh = minv s, the vectors the curvature
// products are taken of, and the iterate advances along them.

// ------------------------------------------------------------ outer step
// out = w + a d, in fp64 (w null: out = a d)
void waxpy(const Launch& L, float* out, const float* w, double a,
           const float* d, long long n);
// dst = src unless *skip (device flag of a solve that has stopped)
void keep_iterate(const Launch& L, float* dst, const float* src, long long n,
                  const int* skip);
// ------------------------------------------------ no-allocation scratch
// Device address of this GPU's HF_NOALLOC_SCRATCH_BYTES scratch array,
// looked up on the first call on each device (the current device).
hipError_t noalloc_scratch(void** out);
// Zero bytes (a multiple of 4) at p with a fill kernel on L.stream.
void fill_zero(const Launch& L, void* p, size_t bytes);

// out[k] = a[k] . b[k] for k < 4 (device doubles), fixed summation order;
// uses the first 4 partial regions of part
void dots4(const Launch& L, const float* const a[4], const float* const b[4],
           long long n, double* part, double* out);

}  // namespace hfk
