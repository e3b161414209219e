// Internal declarations shared by the host driver and the gfx950 kernels.
#pragma once

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

void prof_begin(const Launch& L, const char* name);
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
};

// Forward:  out0 = phi(acc + bias) (hidden) or acc + bias (logits)
void gemm_fwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// Forward + R-forward (dual / dual0):
//   hidden: out0 = A = phi(acc0 + b), out1 = RZ = acc1 + c,
//           out2 = RA = phi'(A) RZ;   output: out0 = acc0 + b, out1 = acc1 + c
void gemm_fwd_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e);
// R-forward on cached activations aux0 = A_l:
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
// Weight gradient (XK = YK = false): out0[z * split_stride + m * ldo + n] = acc
void gemm_wgrad(const Launch& L, const GemmShape& s, const EpiArgs& e);

// --------------------------------------------------------------- row ops
// Softmax cross-entropy over rows of Z (B x C, leading dimension ld):
//   P = softmax(Z); if y: D = (P - onehot(y)) / B and per-block loss partials
//   (double, one per 4 rows) into loss_part; bad labels set *err_flag.
void softmax_xent(const Launch& L, const float* Z, const int32_t* y, int B,
                  int C, int ld, float* P, float* D, double* loss_part,
                  int* err_flag);
// loss = sum(loss_part[0 .. nparts)) / B, in a fixed order.
void loss_finalize(const Launch& L, const double* loss_part, int nparts,
                   int B, float* loss);
// Rdelta_L = P * (RZ - rowsum(P * RZ)) / B.
void softmax_rop(const Launch& L, const float* P, const float* RZ, int B,
                 int C, int ld, float* RD, const int* skip);
// out[c] = sum_r D[r * ld + c] for c < cols (deterministic two-pass);
// part must hold colsum_chunks(rows) * cols doubles.
int colsum_chunks(int rows);
void colsum(const Launch& L, const float* D, int rows, int cols, int ld,
            double* part, float* out, const int* skip);
// out[m * ldo + n] = sum_z part[z * M * N + m * N + n]
void splitk_reduce(const Launch& L, const float* part, int splits, int M,
                   int N, float* out, int ldo, const int* skip);

// ------------------------------------------------------------------- CG
struct CgState {
  double rr, rr0, kappa, alpha, beta, pp, pq, gp;
  double lambda, tol2;
  int done, neg, neg_pending, neg_iter;
  int iters, products, status, j;
  unsigned int counter[4];
  int pad[4];
};

int cg_grid(long long n);
// x = 0, r = g, p = -g, neg_dir = 0, rr = rr0 = |g|^2 (state initialised)
void cg_init(const Launch& L, const float* g, float* x, float* r, float* p,
             float* neg_dir, long long n, double lambda, double tol2,
             double* part, CgState* st);
// kappa = p.q + lambda p.p; detection; alpha
void cg_curv_dot(const Launch& L, const float* p, const float* q, long long n,
                 int j, double* part, CgState* st);
// on a pending detection: gp = g.p; neg_dir = -sgn(gp) p; step = -g at j = 0
void cg_neg(const Launch& L, const float* g, const float* p, float* x,
            float* neg_dir, long long n, double* part, CgState* st);
// x += alpha p; r += alpha (q + lambda p); rr' = r.r; beta; tolerance
void cg_update(const Launch& L, float* x, float* r, const float* p,
               const float* q, long long n, double* part, CgState* st);
// p = -r + beta p
void cg_dir(const Launch& L, const float* r, float* p, long long n,
            CgState* st);

}  // namespace hfk
