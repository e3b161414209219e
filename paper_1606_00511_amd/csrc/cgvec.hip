// Vector kernels of CG-Minimize on the damped operator B_k = A + lambda I
// (Alg. 1 steps 3-4), with the negative-curvature exit of Sec. 2.1 (text
// after eq. (1)) and the orientation d~ = -sgn(g^T p) p of Sec. 2.2.
//
// The recurrences are textbook linear CG from x_0 = 0:
//   kappa = p.(A p) + lambda p.p;  stop if kappa <= 0
//   alpha = rr / kappa;  x += alpha p;  r += alpha (A p + lambda p)
//   rr' = r.r;  beta = rr' / rr;  p = -r + beta p
//
// Kernel schedule of iteration j (all on one stream):
//   dot     per-block partials of p.q and p.p
//   update  every block sums the dot partials in block order (so all blocks
//           hold the same kappa), takes the stop decision, and if it goes on
//           updates x and r and writes per-block partials of r.r; at a
//           detection it writes per-block partials of g.p instead
//   dir     every block sums the r.r partials in block order, forms beta
//           and updates p; at a detection in this iteration it sums the g.p
//           partials and writes d~ and the step instead
// Block 0 of update and dir records the scalars in a CgState in device
// memory; rr is kept in two slots indexed by the iteration's parity so that
// no block reads a slot that another block of the same kernel writes.  No
// fences or atomics are needed, every sum has a fixed order, and repeated
// solves are bit-identical.  Once `done` is set every kernel returns at once.
#include "hf_internal.h"

namespace hfk {
namespace {

constexpr int NT = 256;
constexpr int MAX_GRID = CG_MAX_GRID;

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Fixed-order block sum; the result is returned to every thread.
__device__ __forceinline__ double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

// Fixed-order total of nb per-block partials (same value in every block).
__device__ __forceinline__ double total(const double* part, int nb, double* sh) {
  double s = 0.0;
  for (int b = threadIdx.x; b < nb; b += NT) s += part[b];
  return block_sum(s, sh);
}

__device__ __forceinline__ bool is_fin(double x) { return isfinite(x); }

// Vector updates apply their (fp64) scalars in fp64 and round once on the
// store: near a breakdown of the Bi-CG-STAB recurrences, casting the scalars
// to fp32 and updating in fp32 amplified rounding by orders of magnitude.
struct d4 { double v[4]; };
__device__ __forceinline__ d4 up(f32x4 a) {
  d4 r; r.v[0] = a[0]; r.v[1] = a[1]; r.v[2] = a[2]; r.v[3] = a[3]; return r;
}
__device__ __forceinline__ f32x4 down(const d4& a) {
  f32x4 r = {(float)a.v[0], (float)a.v[1], (float)a.v[2], (float)a.v[3]};
  return r;
}

__device__ __forceinline__ double dot4(f32x4 a, f32x4 b) {
  return ((double)a[0] * b[0] + (double)a[1] * b[1]) +
         ((double)a[2] * b[2] + (double)a[3] * b[3]);
}

}  // namespace

extern "C" __global__ void hf_cg_reset(CgState* __restrict__ st) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    CgState z = {};
    *st = z;
  }
}

// PC: preconditioned CG with z = minv r; p = -z and the partials of r.z too.
template <bool PC>
__device__ __forceinline__ void cg_init_body(
    const float* __restrict__ g, const float* __restrict__ x0,
    const float* __restrict__ q, double lambda, float* __restrict__ x,
    float* __restrict__ r, float* __restrict__ p, float* __restrict__ nd,
    long long n, double* __restrict__ part_rr, double* __restrict__ part_gg,
    const float* __restrict__ minv, double* __restrict__ part_rz) {
  __shared__ double sh[4];
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  double srr = 0.0, sgg = 0.0, srz = 0.0;
  for (long long i = t0; i < n; i += stride) {
    const float gv = g[i];
    float xv = 0.f, rv = gv;
    if (x0) {
      xv = x0[i];
      rv = (float)((double)gv + (double)q[i] + lambda * (double)xv);
    }
    const float zv = PC ? (float)((double)minv[i] * (double)rv) : rv;
    x[i] = xv; r[i] = rv; p[i] = -zv; nd[i] = 0.f;
    srr += (double)rv * rv;
    sgg += (double)gv * gv;
    if (PC) srz += (double)rv * zv;
  }
  srr = block_sum(srr, sh);
  sgg = block_sum(sgg, sh);
  if (PC) srz = block_sum(srz, sh);
  if (threadIdx.x == 0) {
    part_rr[blockIdx.x] = srr;
    part_gg[blockIdx.x] = sgg;
    if (PC) part_rz[blockIdx.x] = srz;
  }
}

// From x0 = 0: x = 0, r = g, p = -g.  From a warm start x0 (with q = A x0):
// x = x0, r = g + q + lambda x0 (the gradient of the model at x0), p = -r.
// d~ = 0.  Partials of r.r and of g.g (the relative stop is against |g|).
extern "C" __global__ __launch_bounds__(256) void hf_cg_init(
    const float* __restrict__ g, const float* __restrict__ x0,
    const float* __restrict__ q, double lambda, float* __restrict__ x,
    float* __restrict__ r, float* __restrict__ p, float* __restrict__ nd,
    long long n, double* __restrict__ part_rr, double* __restrict__ part_gg) {
  cg_init_body<false>(g, x0, q, lambda, x, r, p, nd, n, part_rr, part_gg,
                      nullptr, nullptr);
}
// the same for preconditioned CG: p = -minv r and partials of r.(minv r)
extern "C" __global__ __launch_bounds__(256) void hf_pcg_init(
    const float* __restrict__ g, const float* __restrict__ x0,
    const float* __restrict__ q, double lambda, float* __restrict__ x,
    float* __restrict__ r, float* __restrict__ p, float* __restrict__ nd,
    long long n, double* __restrict__ part_rr, double* __restrict__ part_gg,
    const float* __restrict__ minv, double* __restrict__ part_rz) {
  cg_init_body<true>(g, x0, q, lambda, x, r, p, nd, n, part_rr, part_gg, minv,
                     part_rz);
}

template <bool PC>
__device__ __forceinline__ void cg_init_fin_body(
    const double* __restrict__ part_rr, const double* __restrict__ part_gg,
    const double* __restrict__ part_rz, int nb, double lambda, double tol2,
    int max_iters, CgState* __restrict__ st) {
  __shared__ double sh[4];
  const double rr = total(part_rr, nb, sh);
  const double gg = total(part_gg, nb, sh);
  const double rz = PC ? total(part_rz, nb, sh) : rr;
  if (threadIdx.x == 0) {
    st->rr[0] = rr;
    st->rr[1] = rr;
    st->rz[0] = rz;
    st->rz[1] = rz;
    st->rr0 = gg;
    st->lambda = lambda;
    st->tol2 = tol2;
    st->max_iters = max_iters;
    st->neg_iter = -1;
    const bool fin = is_fin(rr) && is_fin(rz);
    st->status = fin ? 0 : -5;
    st->done = (rr == 0.0 || !fin) ? 1 : 0;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_init_fin(
    const double* __restrict__ part_rr, const double* __restrict__ part_gg,
    int nb, double lambda, double tol2, int max_iters, CgState* __restrict__ st) {
  cg_init_fin_body<false>(part_rr, part_gg, nullptr, nb, lambda, tol2,
                          max_iters, st);
}
extern "C" __global__ __launch_bounds__(256) void hf_pcg_init_fin(
    const double* __restrict__ part_rr, const double* __restrict__ part_gg,
    const double* __restrict__ part_rz, int nb, double lambda, double tol2,
    int max_iters, CgState* __restrict__ st) {
  cg_init_fin_body<true>(part_rr, part_gg, part_rz, nb, lambda, tol2,
                         max_iters, st);
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_dot(
    const float* __restrict__ p, const float* __restrict__ q, long long n,
    double* __restrict__ part, CgState* __restrict__ st, int j) {
  // an iteration replayed from a graph: this is its first vector kernel, and
  // the kernels after it read the index it publishes (no block of this
  // kernel reads jc); -1 once the solve has stopped, so that no later
  // kernel takes a replayed iteration for the one that stopped
  if (j < 0 && blockIdx.x == 0 && threadIdx.x == 0) st->jc = st->done ? -1 : st->jn;
  if (st->done) return;
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  double pq = 0.0, pp = 0.0;
  long long i = t0;
  for (; i + stride < n4; i += 2 * stride) {
    const f32x4 a0 = ((const f32x4*)p)[i], a1 = ((const f32x4*)p)[i + stride];
    const f32x4 b0 = ((const f32x4*)q)[i], b1 = ((const f32x4*)q)[i + stride];
    pq += dot4(a0, b0) + dot4(a1, b1);
    pp += dot4(a0, a0) + dot4(a1, a1);
  }
  for (; i < n4; i += stride) {
    const f32x4 a = ((const f32x4*)p)[i], b = ((const f32x4*)q)[i];
    pq += dot4(a, b);
    pp += dot4(a, a);
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    pq += (double)p[e] * q[e];
    pp += (double)p[e] * p[e];
  }
  pq = block_sum(pq, sh);
  pp = block_sum(pp, sh);
  if (threadIdx.x == 0) {
    part[blockIdx.x] = pq;
    part[MAX_GRID + blockIdx.x] = pp;
  }
}

// PC: alpha = r.z / kappa, and per-block partials of r'.(minv r') as well
template <bool PC>
__device__ __forceinline__ void cg_update_body(
    float* __restrict__ x, float* __restrict__ r, const float* __restrict__ p,
    const float* __restrict__ q, long long n, int j,
    const double* __restrict__ dpart, double* __restrict__ rpart,
    CgState* __restrict__ st, const float* __restrict__ minv,
    double* __restrict__ zpart, const float* __restrict__ g,
    double* __restrict__ gpart, int ndp) {
  if (st->done) return;
  if (j < 0) j = st->jc;
  __shared__ double sh[4];
  // the partials of p.q and p.p: one per block of the dot kernel (its grid
  // is this one), or ndp from the product that formed them
  const int nb = ndp > 0 ? ndp : (int)gridDim.x;
  const double pq = total(dpart, nb, sh);
  const double pp = total(dpart + MAX_GRID, nb, sh);
  const double lam = st->lambda;
  const double kappa = pq + lam * pp;
  const double rr = PC ? st->rz[j & 1] : st->rr[j & 1];
  const bool stop = !is_fin(kappa) || kappa <= 0.0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->kappa = kappa;
    st->pq = pq;
    st->pp = pp;
    st->products = j + 1;
    if (!is_fin(kappa)) {
      st->status = -5;
      st->done = 1;
    } else if (kappa <= 0.0) {
      st->neg = 1;
      st->neg_iter = j;
      st->done = 1;
    } else {
      st->alpha = rr / kappa;
    }
  }
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  if (stop) {
    if (!is_fin(kappa)) return;
    // detection: partials of g.p for the orientation of d~
    double gp = 0.0;
    for (long long i = t0; i < n4; i += stride)
      gp += dot4(((const f32x4*)g)[i], ((const f32x4*)p)[i]);
    for (long long e = n4 * 4 + t0; e < n; e += stride) gp += (double)g[e] * p[e];
    gp = block_sum(gp, sh);
    if (threadIdx.x == 0) gpart[blockIdx.x] = gp;
    return;
  }
  const double alpha = rr / kappa;
  double s = 0.0, sz = 0.0;
  for (long long i = t0; i < n4; i += stride) {
    const d4 pv = up(((const f32x4*)p)[i]);
    const d4 qv = up(((const f32x4*)q)[i]);
    d4 xv = up(((f32x4*)x)[i]);
    d4 rv = up(((f32x4*)r)[i]);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      xv.v[k] += alpha * pv.v[k];
      rv.v[k] += alpha * (qv.v[k] + lam * pv.v[k]);
    }
    const f32x4 r4 = down(rv);
    ((f32x4*)x)[i] = down(xv);
    ((f32x4*)r)[i] = r4;
    s += dot4(r4, r4);
    if (PC) {
      const f32x4 m4 = ((const f32x4*)minv)[i];
#pragma unroll
      for (int k = 0; k < 4; ++k) sz += (double)r4[k] * (double)(float)((double)m4[k] * (double)r4[k]);
    }
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    const double pv = p[e];
    x[e] = (float)((double)x[e] + alpha * pv);
    const float rv = (float)((double)r[e] + alpha * ((double)q[e] + lam * pv));
    r[e] = rv;
    s += (double)rv * rv;
    if (PC) sz += (double)rv * (double)(float)((double)minv[e] * (double)rv);
  }
  s = block_sum(s, sh);
  if (PC) sz = block_sum(sz, sh);
  if (threadIdx.x == 0) {
    rpart[blockIdx.x] = s;
    if (PC) zpart[blockIdx.x] = sz;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_update(
    float* __restrict__ x, float* __restrict__ r, const float* __restrict__ p,
    const float* __restrict__ q, long long n, int j,
    const double* __restrict__ dpart, double* __restrict__ rpart,
    CgState* __restrict__ st, const float* __restrict__ g,
    double* __restrict__ gpart, int ndp) {
  cg_update_body<false>(x, r, p, q, n, j, dpart, rpart, st, nullptr, nullptr,
                        g, gpart, ndp);
}
extern "C" __global__ __launch_bounds__(256) void hf_pcg_update(
    float* __restrict__ x, float* __restrict__ r, const float* __restrict__ p,
    const float* __restrict__ q, long long n, int j,
    const double* __restrict__ dpart, double* __restrict__ rpart,
    CgState* __restrict__ st, const float* __restrict__ minv,
    double* __restrict__ zpart, const float* __restrict__ g,
    double* __restrict__ gpart, int ndp) {
  cg_update_body<true>(x, r, p, q, n, j, dpart, rpart, st, minv, zpart, g,
                       gpart, ndp);
}

// PC: beta = r'.z' / r.z and p = -minv r + beta p.
// At a detection in iteration j: d~ = -sgn(g.p) p with sgn(0) = +1, and the
// step is -g when the detection happened at the first iteration, else the
// current iterate.
template <bool PC>
__device__ __forceinline__ void cg_dir_body(
    const float* __restrict__ r, float* __restrict__ p, long long n, int j,
    const double* __restrict__ rpart, CgState* __restrict__ st,
    const float* __restrict__ minv, const double* __restrict__ zpart,
    int* __restrict__ hflag, const float* __restrict__ g,
    float* __restrict__ x, float* __restrict__ nd,
    const double* __restrict__ gpart) {
  const bool lead = blockIdx.x == 0 && threadIdx.x == 0;
  const bool replay = j < 0;
  if (replay) j = st->jc;
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  if (st->done) {
    if (st->neg && st->neg_iter == j) {
      const double gp = total(gpart, gridDim.x, sh);
      if (lead) st->gp = gp;
      const float coef = gp >= 0.0 ? -1.0f : 1.0f;
      const bool first = j == 0;
      for (long long i = t0; i < n4; i += stride) {
        ((f32x4*)nd)[i] = coef * ((const f32x4*)p)[i];
        if (first) ((f32x4*)x)[i] = -((const f32x4*)g)[i];
      }
      for (long long e = n4 * 4 + t0; e < n; e += stride) {
        nd[e] = coef * p[e];
        if (first) x[e] = -g[e];
      }
    }
    if (hflag && lead) *(volatile int*)hflag = 1;
    return;
  }
  const double rr_new = total(rpart, gridDim.x, sh);
  const double rz_new = PC ? total(zpart, gridDim.x, sh) : rr_new;
  const double rz = PC ? st->rz[j & 1] : st->rr[j & 1];
  const double beta = rz_new / rz;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->rr[(j + 1) & 1] = rr_new;
    if (PC) st->rz[(j + 1) & 1] = rz_new;
    st->iters = j + 1;
    st->beta = beta;
    if (!is_fin(rr_new) || !is_fin(rz_new)) {
      st->status = -5;
      st->done = 1;
    } else if (st->tol2 > 0.0 && rr_new <= st->tol2 * st->rr0) {
      st->done = 1;
    } else if (st->max_iters > 0 && j + 1 >= st->max_iters) {
      st->done = 1;
    }
    if (replay) st->jn = j + 1;
    if (hflag) *(volatile int*)hflag = st->done;
  }
  for (long long i = t0; i < n4; i += stride) {
    d4 pv = up(((const f32x4*)p)[i]);
    d4 zv = up(((const f32x4*)r)[i]);
    if (PC) {
      const f32x4 m4 = ((const f32x4*)minv)[i];
#pragma unroll
      for (int k = 0; k < 4; ++k) zv.v[k] = (double)(float)((double)m4[k] * zv.v[k]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) pv.v[k] = beta * pv.v[k] - zv.v[k];
    ((f32x4*)p)[i] = down(pv);
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    const double zv = PC ? (double)(float)((double)minv[e] * (double)r[e]) : (double)r[e];
    p[e] = (float)(beta * (double)p[e] - zv);
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_dir(
    const float* __restrict__ r, float* __restrict__ p, long long n, int j,
    const double* __restrict__ rpart, CgState* __restrict__ st,
    int* __restrict__ hflag, const float* __restrict__ g,
    float* __restrict__ x, float* __restrict__ nd,
    const double* __restrict__ gpart) {
  cg_dir_body<false>(r, p, n, j, rpart, st, nullptr, nullptr, hflag, g, x, nd,
                     gpart);
}
extern "C" __global__ __launch_bounds__(256) void hf_pcg_dir(
    const float* __restrict__ r, float* __restrict__ p, long long n, int j,
    const double* __restrict__ rpart, CgState* __restrict__ st,
    const float* __restrict__ minv, const double* __restrict__ zpart,
    int* __restrict__ hflag, const float* __restrict__ g,
    float* __restrict__ x, float* __restrict__ nd,
    const double* __restrict__ gpart) {
  cg_dir_body<true>(r, p, n, j, rpart, st, minv, zpart, hflag, g, x, nd, gpart);
}

// ------------------------------------------------------------- launchers
// One float4 per thread and block pass, up to MAX_GRID blocks: the vectors
// of the small nets (below a million parameters) are latency-bound, and a
// grid of a few dozen blocks left each thread a chain of dependent passes
// (784-100-10 net: update and direction kernels 6 -> 5 us each).
int cg_grid(long long n) {
  long long b = (n + NT * 4 - 1) / (NT * 4);
  if (b < 1) b = 1;
  if (b > MAX_GRID) b = MAX_GRID;
  return (int)b;
}

int cg_part_doubles() { return 10 * MAX_GRID; }

void cg_init(const Launch& L, const float* g, const float* x0, const float* q,
             float* x, float* r, float* p, float* neg_dir, long long n,
             double lambda, double tol2, double* part, CgState* st,
             const float* minv, int max_iters) {
  const int nb = cg_grid(n);
  hipLaunchKernelGGL(hf_cg_reset, dim3(1), dim3(64), 0, L.stream, st);
  if (minv) {
    prof_begin(L, "hf_pcg_init");
    hipExtLaunchKernelGGL(hf_pcg_init, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, g, x0, q,
                       lambda, x, r, p, neg_dir, n, part + 4 * MAX_GRID,
                       part + 5 * MAX_GRID, minv, part + 6 * MAX_GRID);
    prof_end(L, "hf_pcg_init", 0.0, (x0 ? 8.0 : 6.0) * 4.0 * n);
    hipLaunchKernelGGL(hf_pcg_init_fin, dim3(1), dim3(NT), 0, L.stream,
                       part + 4 * MAX_GRID, part + 5 * MAX_GRID,
                       part + 6 * MAX_GRID, nb, lambda, tol2, max_iters, st);
    return;
  }
  prof_begin(L, "hf_cg_init");
  hipExtLaunchKernelGGL(hf_cg_init, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, g, x0, q,
                     lambda, x, r, p, neg_dir, n, part + 4 * MAX_GRID,
                     part + 5 * MAX_GRID);
  prof_end(L, "hf_cg_init", 0.0, (x0 ? 7.0 : 5.0) * 4.0 * n);
  hipLaunchKernelGGL(hf_cg_init_fin, dim3(1), dim3(NT), 0, L.stream,
                     part + 4 * MAX_GRID, part + 5 * MAX_GRID, nb, lambda, tol2,
                     max_iters, st);
}

void cg_iteration(const Launch& L, float* x, float* r, float* p, const float* q,
                  const float* g, float* neg_dir, long long n, int j,
                  double* part, CgState* st, const float* minv, int* hflag,
                  int dot_blocks) {
  const int nb = cg_grid(n);
  double* dpart = part;                  // 2 * MAX_GRID: p.q, p.p
  double* rpart = part + 2 * MAX_GRID;   // r.r
  double* gpart = part + 3 * MAX_GRID;   // g.p
  double* zpart = part + 6 * MAX_GRID;   // r.z (preconditioned)
  if (dot_blocks <= 0) {
    prof_begin(L, "hf_cg_dot");
    hipExtLaunchKernelGGL(hf_cg_dot, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, p, q,
                          n, dpart, st, j);
    prof_end(L, "hf_cg_dot", 0.0, 2.0 * 4.0 * n);
  }
  if (minv) {
    prof_begin(L, "hf_pcg_update");
    hipExtLaunchKernelGGL(hf_pcg_update, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, x, r, p,
                       q, n, j, dpart, rpart, st, minv, zpart, g, gpart, dot_blocks);
    prof_end(L, "hf_pcg_update", 0.0, 7.0 * 4.0 * n);
  } else {
    prof_begin(L, "hf_cg_update");
    hipExtLaunchKernelGGL(hf_cg_update, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, x, r, p,
                       q, n, j, dpart, rpart, st, g, gpart, dot_blocks);
    prof_end(L, "hf_cg_update", 0.0, 6.0 * 4.0 * n);
  }
  if (minv) {
    prof_begin(L, "hf_pcg_dir");
    hipExtLaunchKernelGGL(hf_pcg_dir, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, r, p, n, j,
                       rpart, st, minv, zpart, hflag, g, x, neg_dir, gpart);
    prof_end(L, "hf_pcg_dir", 0.0, 4.0 * 4.0 * n);
  } else {
    prof_begin(L, "hf_cg_dir");
    hipExtLaunchKernelGGL(hf_cg_dir, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, r, p, n, j,
                       rpart, st, hflag, g, x, neg_dir, gpart);
    prof_end(L, "hf_cg_dir", 0.0, 3.0 * 4.0 * n);
  }
}

// ========================================================== Bi-CG-STAB
// Alg. 3 on B_k d = -g, B_k = A + lambda I, from d = 0 with r0* = r0.
// Iteration j, with its two curvature products (Ap = B p_j, t = B s_j):
//   bicg_dot1    partials of (Ap, r0*)
//   bicg_s       alpha = rho_j / (Ap, r0*) (every block sums the partials);
//                s = r - alpha Ap
//   bicg_dot2    partials of (s, t) and (t, t)
//   bicg_update  gamma = (s, t) / (t, t) (0 if t = 0); x += alpha p + gamma s;
//                r = s - gamma t; partials of (r, r0*), (r, r), (g, x),
//                (r, x), (x, x)
//   bicg_dir     the candidate x_{j+1}: since r = -g - B x, its curvature is
//                x^T B x = -(g, x) - (r, x) and x^T A x = x^T B x - lambda (x, x);
//                beta = (rho_{j+1} / rho_j)(alpha / gamma); p = r + beta (p - gamma Ap)
//   bicg_negw    at the first negative-curvature candidate: d~ = -sgn(g, x) x
// Preconditioned (minv = the diagonal of M^-1 given): Bi-CG-STAB
// preconditioned on the right.  The products are taken of p^ = M^-1 p and
// s^ = M^-1 s, written beside p and s by the kernels that form them, and
// x advances along them (x += alpha p^ + gamma s^); r stays the residual of
// the original system, so every test and the candidate curvature are
// unchanged.
// Scalars stay in a BicgState; as for CG, blocks that need a reduced value
// each sum the per-block partials in block order, and block 0 records it.
namespace {
constexpr int PA = 0;                 // (Ap, r0*)
constexpr int PB = 1 * MAX_GRID;      // (s, t), (t, t)
constexpr int PC = 3 * MAX_GRID;      // five dots of bicg_update
constexpr int PI = 8 * MAX_GRID;      // (r0, r0) and (g, g) of the init
}  // namespace

extern "C" __global__ void hf_bicg_reset(BicgState* __restrict__ st) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    BicgState z = {};
    *st = z;
  }
}

// From 0: x = 0, r = r0* = p = -g.  From a warm start x0 (q = A x0):
// x = x0, r = r0* = p = -g - (q + lambda x0).  d~ = 0.  Partials of r.r
// (= (r0, r0*)) and of g.g (the relative stop is against |g|).
extern "C" __global__ __launch_bounds__(256) void hf_bicg_init(
    const float* __restrict__ g, const float* __restrict__ x0,
    const float* __restrict__ q, double lambda, float* __restrict__ x,
    float* __restrict__ r, float* __restrict__ rs, float* __restrict__ p,
    float* __restrict__ nd, long long n, double* __restrict__ part,
    const float* __restrict__ minv, float* __restrict__ ph) {
  __shared__ double sh[4];
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  double srr = 0.0, sgg = 0.0;
  for (long long i = t0; i < n; i += stride) {
    const float gv = g[i];
    float xv = 0.f, rv = -gv;
    if (x0) {
      xv = x0[i];
      rv = (float)(-(double)gv - ((double)q[i] + lambda * (double)xv));
    }
    x[i] = xv; r[i] = rv; rs[i] = rv; p[i] = rv; nd[i] = 0.f;
    if (minv) ph[i] = (float)((double)minv[i] * (double)rv);
    srr += (double)rv * rv;
    sgg += (double)gv * gv;
  }
  srr = block_sum(srr, sh);
  sgg = block_sum(sgg, sh);
  if (threadIdx.x == 0) {
    part[PI + blockIdx.x] = srr;
    part[PI + MAX_GRID + blockIdx.x] = sgg;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_bicg_init_fin(
    const double* __restrict__ part, int nb, double lambda, double tol2,
    BicgState* __restrict__ st) {
  __shared__ double sh[4];
  const double rr = total(part + PI, nb, sh);
  const double gg = total(part + PI + MAX_GRID, nb, sh);
  if (threadIdx.x == 0) {
    st->rho[0] = rr;          // (r0, r0*) = |r0|^2
    st->rr0 = gg;
    st->rr = rr;
    st->lambda = lambda;
    st->tol2 = tol2;
    st->neg_iter = -1;
    st->status = is_fin(rr) ? 0 : -5;
    st->done = (rr == 0.0 || !is_fin(rr)) ? 1 : 0;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_bicg_dot1(
    const float* __restrict__ Ap, const float* __restrict__ rs, long long n,
    double* __restrict__ part, const BicgState* __restrict__ st) {
  if (st->done) return;
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  double a = 0.0;
  for (long long i = t0; i < n4; i += stride)
    a += dot4(((const f32x4*)Ap)[i], ((const f32x4*)rs)[i]);
  for (long long e = n4 * 4 + t0; e < n; e += stride) a += (double)Ap[e] * rs[e];
  a = block_sum(a, sh);
  if (threadIdx.x == 0) part[PA + blockIdx.x] = a;
}

extern "C" __global__ __launch_bounds__(256) void hf_bicg_s(
    const float* __restrict__ r, const float* __restrict__ Ap,
    float* __restrict__ s, long long n, int j, const double* __restrict__ part,
    BicgState* __restrict__ st, const float* __restrict__ minv,
    float* __restrict__ shat) {
  if (st->done) return;
  __shared__ double sh[4];
  const double den = total(part + PA, gridDim.x, sh);
  const double alpha = st->rho[j & 1] / den;
  const bool stop = den == 0.0 || !is_fin(alpha);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->products = 2 * j + 1;
    st->alpha = alpha;
    if (stop) {
      if (!is_fin(den)) st->status = -5;
      st->done = 1;
    }
  }
  if (stop) return;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  for (long long i = t0; i < n4; i += stride) {
    d4 rv = up(((const f32x4*)r)[i]);
    const d4 av = up(((const f32x4*)Ap)[i]);
#pragma unroll
    for (int k = 0; k < 4; ++k) rv.v[k] -= alpha * av.v[k];
    const f32x4 s4 = down(rv);
    ((f32x4*)s)[i] = s4;
    if (minv) {
      const f32x4 m4 = ((const f32x4*)minv)[i];
      f32x4 h4;
#pragma unroll
      for (int k = 0; k < 4; ++k) h4[k] = (float)((double)m4[k] * (double)s4[k]);
      ((f32x4*)shat)[i] = h4;
    }
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    const float sv = (float)((double)r[e] - alpha * (double)Ap[e]);
    s[e] = sv;
    if (minv) shat[e] = (float)((double)minv[e] * (double)sv);
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_bicg_dot2(
    const float* __restrict__ s, const float* __restrict__ t, long long n,
    double* __restrict__ part, const BicgState* __restrict__ st) {
  if (st->done) return;
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  double st_ = 0.0, tt = 0.0;
  for (long long i = t0; i < n4; i += stride) {
    const f32x4 a = ((const f32x4*)s)[i], b = ((const f32x4*)t)[i];
    st_ += dot4(a, b);
    tt += dot4(b, b);
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    st_ += (double)s[e] * t[e];
    tt += (double)t[e] * t[e];
  }
  st_ = block_sum(st_, sh);
  tt = block_sum(tt, sh);
  if (threadIdx.x == 0) {
    part[PB + blockIdx.x] = st_;
    part[PB + MAX_GRID + blockIdx.x] = tt;
  }
}

// ph, shat: the vectors the products were taken of (p and s themselves
// without a preconditioner)
extern "C" __global__ __launch_bounds__(256) void hf_bicg_update(
    float* __restrict__ x, float* __restrict__ r, const float* __restrict__ rs,
    const float* __restrict__ ph, const float* __restrict__ s,
    const float* __restrict__ shat, const float* __restrict__ t,
    const float* __restrict__ g, long long n, int j, double* __restrict__ part,
    BicgState* __restrict__ st) {
  if (st->done) return;
  __shared__ double sh[4];
  const double stv = total(part + PB, gridDim.x, sh);
  const double tt = total(part + PB + MAX_GRID, gridDim.x, sh);
  const double gamma = tt != 0.0 ? stv / tt : 0.0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->gamma = gamma;
    st->products = 2 * j + 2;
    st->iters = j + 1;
  }
  const double a = st->alpha, c = gamma;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  double e0 = 0.0, e1 = 0.0, e2 = 0.0, e3 = 0.0, e4 = 0.0;
  for (long long i = t0; i < n4; i += stride) {
    const d4 sv = up(((const f32x4*)s)[i]), tv = up(((const f32x4*)t)[i]);
    const d4 pv = up(((const f32x4*)ph)[i]), shv = up(((const f32x4*)shat)[i]);
    d4 xv = up(((f32x4*)x)[i]), rv;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      xv.v[k] += a * pv.v[k] + c * shv.v[k];
      rv.v[k] = sv.v[k] - c * tv.v[k];
    }
    const f32x4 x4 = down(xv), r4 = down(rv);
    ((f32x4*)x)[i] = x4;
    ((f32x4*)r)[i] = r4;
    e0 += dot4(r4, ((const f32x4*)rs)[i]);
    e1 += dot4(r4, r4);
    e2 += dot4(((const f32x4*)g)[i], x4);
    e3 += dot4(r4, x4);
    e4 += dot4(x4, x4);
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    const float xv = (float)((double)x[e] + a * (double)ph[e] + c * (double)shat[e]);
    const float rv = (float)((double)s[e] - c * (double)t[e]);
    x[e] = xv;
    r[e] = rv;
    e0 += (double)rv * rs[e];
    e1 += (double)rv * rv;
    e2 += (double)g[e] * xv;
    e3 += (double)rv * xv;
    e4 += (double)xv * xv;
  }
  const double d0 = block_sum(e0, sh);
  const double d1 = block_sum(e1, sh);
  const double d2 = block_sum(e2, sh);
  const double d3 = block_sum(e3, sh);
  const double d4s = block_sum(e4, sh);
  if (threadIdx.x == 0) {
    part[PC + blockIdx.x] = d0;
    part[PC + MAX_GRID + blockIdx.x] = d1;
    part[PC + 2 * MAX_GRID + blockIdx.x] = d2;
    part[PC + 3 * MAX_GRID + blockIdx.x] = d3;
    part[PC + 4 * MAX_GRID + blockIdx.x] = d4s;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_bicg_dir(
    float* __restrict__ p, const float* __restrict__ r,
    const float* __restrict__ Ap, long long n, int j,
    const double* __restrict__ part, BicgState* __restrict__ st,
    const float* __restrict__ minv, float* __restrict__ ph) {
  if (st->done) return;
  __shared__ double sh[4];
  const int nb = gridDim.x;
  const double rho1 = total(part + PC, nb, sh);
  const double rr = total(part + PC + MAX_GRID, nb, sh);
  const double gx = total(part + PC + 2 * MAX_GRID, nb, sh);
  const double rx = total(part + PC + 3 * MAX_GRID, nb, sh);
  const double xx = total(part + PC + 4 * MAX_GRID, nb, sh);
  const double rho = st->rho[j & 1];
  const double gamma = st->gamma;
  const double xBx = -gx - rx;
  const double xHx = xBx - st->lambda * xx;
  const bool bad = !is_fin(rr) || !is_fin(rho1) || !is_fin(xBx);
  const bool stop = bad || (st->tol2 > 0.0 && rr <= st->tol2 * st->rr0) ||
                    rho1 == 0.0 || gamma == 0.0;
  const double beta = stop ? 0.0 : (rho1 / rho) * (st->alpha / gamma);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->rr = rr;
    st->rho[(j + 1) & 1] = rho1;
    st->beta = beta;
    if (xHx < 0.0 && st->neg_iter < 0) {
      st->neg = 1;
      st->neg_iter = j;
      st->dHd = xHx;
      st->dBd = xBx;
      st->coef = gx >= 0.0 ? -1.0 : 1.0;     // d~ = -sgn(g.x) x
      st->gTd = st->coef * gx;
    }
    if (bad) st->status = -5;
    if (stop) st->done = 1;
  }
  if (stop) return;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  for (long long i = t0; i < n4; i += stride) {
    d4 pv = up(((const f32x4*)p)[i]);
    const d4 rv = up(((const f32x4*)r)[i]), av = up(((const f32x4*)Ap)[i]);
#pragma unroll
    for (int k = 0; k < 4; ++k) pv.v[k] = rv.v[k] + beta * (pv.v[k] - gamma * av.v[k]);
    const f32x4 p4 = down(pv);
    ((f32x4*)p)[i] = p4;
    if (minv) {
      const f32x4 m4 = ((const f32x4*)minv)[i];
      f32x4 h4;
#pragma unroll
      for (int k = 0; k < 4; ++k) h4[k] = (float)((double)m4[k] * (double)p4[k]);
      ((f32x4*)ph)[i] = h4;
    }
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride) {
    const float pv = (float)((double)r[e] + beta * ((double)p[e] - gamma * (double)Ap[e]));
    p[e] = pv;
    if (minv) ph[e] = (float)((double)minv[e] * (double)pv);
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_bicg_negw(
    const float* __restrict__ x, float* __restrict__ nd, long long n, int j,
    const BicgState* __restrict__ st) {
  if (st->neg_iter != j) return;
  const float c = (float)st->coef;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  for (long long i = t0; i < n4; i += stride)
    ((f32x4*)nd)[i] = c * ((const f32x4*)x)[i];
  for (long long e = n4 * 4 + t0; e < n; e += stride) nd[e] = c * x[e];
}

extern "C" __global__ __launch_bounds__(256) void hf_axpy(
    float* __restrict__ y, const float* __restrict__ x, double a, long long n,
    const int* __restrict__ skip) {
  if (skip && *skip) return;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  const long long t0 = (long long)blockIdx.x * NT + threadIdx.x;
  for (long long i = t0; i < n4; i += stride) {
    d4 yv = up(((const f32x4*)y)[i]);
    const d4 xv = up(((const f32x4*)x)[i]);
#pragma unroll
    for (int k = 0; k < 4; ++k) yv.v[k] += a * xv.v[k];
    ((f32x4*)y)[i] = down(yv);
  }
  for (long long e = n4 * 4 + t0; e < n; e += stride)
    y[e] = (float)((double)y[e] + a * (double)x[e]);
}

void axpy(const Launch& L, float* y, const float* x, float a, long long n,
          const int* skip) {
  prof_begin(L, "hf_axpy");
  hipExtLaunchKernelGGL(hf_axpy, dim3(cg_grid(n)), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, y, x,
                     (double)a, n, skip);
  prof_end(L, "hf_axpy", 0.0, 3.0 * 4.0 * n);
}

void bicg_init(const Launch& L, const float* g, const float* x0,
               const float* q, float* x, float* r, float* rs, float* p,
               float* neg_dir, long long n, double lambda, double tol2,
               double* part, BicgState* st, const float* minv, float* ph) {
  const int nb = cg_grid(n);
  hipLaunchKernelGGL(hf_bicg_reset, dim3(1), dim3(64), 0, L.stream, st);
  prof_begin(L, "hf_bicg_init");
  hipExtLaunchKernelGGL(hf_bicg_init, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, g, x0, q,
                     lambda, x, r, rs, p, neg_dir, n, part, minv, ph);
  prof_end(L, "hf_bicg_init", 0.0, ((x0 ? 8.0 : 6.0) + (minv ? 2.0 : 0.0)) * 4.0 * n);
  hipLaunchKernelGGL(hf_bicg_init_fin, dim3(1), dim3(NT), 0, L.stream, part, nb,
                     lambda, tol2, st);
}

void bicg_half(const Launch& L, const float* r, const float* rs,
               const float* Ap, float* s, long long n, int j, double* part,
               BicgState* st, const float* minv, float* sh) {
  const int nb = cg_grid(n);
  prof_begin(L, "hf_bicg_dot1");
  hipExtLaunchKernelGGL(hf_bicg_dot1, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, Ap, rs, n,
                     part, st);
  prof_end(L, "hf_bicg_dot1", 0.0, 2.0 * 4.0 * n);
  prof_begin(L, "hf_bicg_s");
  hipExtLaunchKernelGGL(hf_bicg_s, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, r, Ap, s, n, j,
                     part, st, minv, sh);
  prof_end(L, "hf_bicg_s", 0.0, (minv ? 5.0 : 3.0) * 4.0 * n);
}

void bicg_rest(const Launch& L, float* x, float* r, const float* rs, float* p,
               const float* Ap, const float* s, const float* t, const float* g,
               float* neg_dir, long long n, int j, double* part,
               BicgState* st, const float* minv, float* ph, const float* sh) {
  if (!minv) {
    ph = p;
    sh = s;
  }
  const int nb = cg_grid(n);
  prof_begin(L, "hf_bicg_dot2");
  hipExtLaunchKernelGGL(hf_bicg_dot2, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, s, t, n,
                     part, st);
  prof_end(L, "hf_bicg_dot2", 0.0, 2.0 * 4.0 * n);
  prof_begin(L, "hf_bicg_update");
  hipExtLaunchKernelGGL(hf_bicg_update, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, x, r, rs,
                     ph, s, sh, t, g, n, j, part, st);
  prof_end(L, "hf_bicg_update", 0.0, (minv ? 9.0 : 8.0) * 4.0 * n);
  prof_begin(L, "hf_bicg_dir");
  hipExtLaunchKernelGGL(hf_bicg_dir, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, p, r, Ap, n,
                     j, part, st, minv, ph);
  prof_end(L, "hf_bicg_dir", 0.0, (minv ? 6.0 : 4.0) * 4.0 * n);
  prof_begin(L, "hf_bicg_negw");
  hipExtLaunchKernelGGL(hf_bicg_negw, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, x, neg_dir,
                     n, j, st);
  prof_end(L, "hf_bicg_negw", 0.0, 2.0 * 4.0 * n);
}


// ============================================================ outer step
// out = w + a d (w may be null: out = a d), applied in fp64
extern "C" __global__ __launch_bounds__(256) void hf_waxpy(
    float* __restrict__ out, const float* __restrict__ w, double a,
    const float* __restrict__ d, long long n) {
  const long long stride = (long long)gridDim.x * NT;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride)
    out[i] = (float)((w ? (double)w[i] : 0.0) + a * (double)d[i]);
}

// dst = src, unless the solve has stopped (*skip != 0): keeps a solver
// iterate for CG-backtracking only if the iteration that formed it ran
extern "C" __global__ __launch_bounds__(256) void hf_keep_iterate(
    float* __restrict__ dst, const float* __restrict__ src, long long n,
    const int* __restrict__ skip) {
  if (skip && *skip) return;
  const long long stride = (long long)gridDim.x * NT;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

// per-block partials of the four dot products a_k . b_k
extern "C" __global__ __launch_bounds__(256) void hf_dots4(
    const float* __restrict__ a0, const float* __restrict__ b0,
    const float* __restrict__ a1, const float* __restrict__ b1,
    const float* __restrict__ a2, const float* __restrict__ b2,
    const float* __restrict__ a3, const float* __restrict__ b3, long long n,
    double* __restrict__ part) {
  __shared__ double sh[4];
  const long long stride = (long long)gridDim.x * NT;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride) {
    s0 += (double)a0[i] * b0[i];
    s1 += (double)a1[i] * b1[i];
    s2 += (double)a2[i] * b2[i];
    s3 += (double)a3[i] * b3[i];
  }
  s0 = block_sum(s0, sh);
  s1 = block_sum(s1, sh);
  s2 = block_sum(s2, sh);
  s3 = block_sum(s3, sh);
  if (threadIdx.x == 0) {
    part[blockIdx.x] = s0;
    part[MAX_GRID + blockIdx.x] = s1;
    part[2 * MAX_GRID + blockIdx.x] = s2;
    part[3 * MAX_GRID + blockIdx.x] = s3;
  }
}

// out[k] = sum of the partials of dot k, in block order
extern "C" __global__ __launch_bounds__(256) void hf_dots4_fin(
    const double* __restrict__ part, int nb, double* __restrict__ out) {
  __shared__ double sh[4];
  for (int k = 0; k < 4; ++k) {
    const double t = total(part + k * MAX_GRID, nb, sh);
    if (threadIdx.x == 0) out[k] = t;
  }
}

void waxpy(const Launch& L, float* out, const float* w, double a,
           const float* d, long long n) {
  const int nb = cg_grid(n);
  prof_begin(L, "hf_waxpy");
  hipExtLaunchKernelGGL(hf_waxpy, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, out, w, a, d, n);
  prof_end(L, "hf_waxpy", 0.0, (w ? 3.0 : 2.0) * 4.0 * n);
}

void keep_iterate(const Launch& L, float* dst, const float* src, long long n,
                  const int* skip) {
  const int nb = cg_grid(n);
  prof_begin(L, "hf_keep_iterate");
  hipExtLaunchKernelGGL(hf_keep_iterate, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, dst, src,
                     n, skip);
  prof_end(L, "hf_keep_iterate", 0.0, 2.0 * 4.0 * n);
}

void dots4(const Launch& L, const float* const a[4], const float* const b[4],
           long long n, double* part, double* out) {
  const int nb = cg_grid(n);
  prof_begin(L, "hf_dots4");
  hipExtLaunchKernelGGL(hf_dots4, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, a[0], b[0], a[1],
                     b[1], a[2], b[2], a[3], b[3], n, part);
  prof_end(L, "hf_dots4", 0.0, 8.0 * 4.0 * n);
  hipLaunchKernelGGL(hf_dots4_fin, dim3(1), dim3(NT), 0, L.stream, part, nb, out);
}

// minv = (F + lambda)^(-xi): the diagonal of M^-1 for Martens' M = (F + lambda)^xi
extern "C" __global__ __launch_bounds__(256) void hf_precond_inv(
    const float* __restrict__ F, double lambda, double xi, float* __restrict__ minv,
    long long n) {
  const long long stride = (long long)gridDim.x * NT;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride)
    minv[i] = (float)pow((double)F[i] + lambda, -xi);
}

void precond_inverse(const Launch& L, const float* F, double lambda, double xi,
                     float* minv, long long n) {
  const int nb = cg_grid(n);
  prof_begin(L, "hf_precond_inv");
  hipExtLaunchKernelGGL(hf_precond_inv, dim3(nb), dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, F, lambda,
                     xi, minv, n);
  prof_end(L, "hf_precond_inv", 0.0, 2.0 * 4.0 * n);
}

}  // namespace hfk
