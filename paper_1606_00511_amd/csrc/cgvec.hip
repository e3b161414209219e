// Vector kernels of CG-Minimize on the damped operator B_k = A + lambda I
// (Alg. 1 steps 3-4), with the negative-curvature exit of Sec. 2.1 (text
// after eq. (1)) and the orientation d~ = -sgn(g^T p) p of Sec. 2.2.
//
// The recurrences are textbook linear CG from x_0 = 0:
//   kappa = p.(A p) + lambda p.p;  stop if kappa <= 0
//   alpha = rr / kappa;  x += alpha p;  r += alpha (A p + lambda p)
//   rr' = r.r;  beta = rr' / rr;  p = -r + beta p
//
// The scalars live in a CgState in device memory and never travel to the
// host inside the loop.  Each dot product is a grid of blocks that reduce
// float data in double precision (wave shuffles, then LDS across the 4
// waves); the last block to finish (atomic ticket) sums the per-block
// partials in block order and updates the state, so every sum has a fixed
// order and repeated solves are bit-identical.  After a stop every kernel
// reads `done` and returns at once.
#include "hf_internal.h"

namespace hfk {
namespace {

constexpr int NT = 256;
constexpr int MAX_GRID = 1024;

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over the block in a fixed order; the result is valid in thread 0.
__device__ __forceinline__ double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) r = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  __syncthreads();
  return r;
}

// Publish this block's partials, then report whether it is the last block.
template <int K>
__device__ __forceinline__ bool publish(const double (&v)[K], double* part,
                                        unsigned int* counter, double* sh) {
  __shared__ bool last;
  double r[K];
#pragma unroll
  for (int k = 0; k < K; ++k) r[k] = block_sum(v[k], sh);
  if (threadIdx.x == 0) {
#pragma unroll
    for (int k = 0; k < K; ++k) part[(size_t)k * MAX_GRID + blockIdx.x] = r[k];
    __threadfence();
    const unsigned int t = atomicAdd(counter, 1u);
    last = (t == gridDim.x - 1);
  }
  __syncthreads();
  if (last) __threadfence();
  return last;
}

// In the last block: the fixed-order total of partial k over all blocks.
__device__ __forceinline__ double gather(const double* part, int k,
                                         double* sh) {
  double s = 0.0;
  for (int b = threadIdx.x; b < (int)gridDim.x; b += NT)
    s += part[(size_t)k * MAX_GRID + b];
  return block_sum(s, sh);
}

__device__ __forceinline__ bool is_fin(double x) { return isfinite(x); }

}  // namespace

extern "C" __global__ void hf_cg_reset(CgState* __restrict__ st) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    CgState z = {};
    *st = z;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_init(
    const float* __restrict__ g, float* __restrict__ x, float* __restrict__ r,
    float* __restrict__ p, float* __restrict__ nd, long long n, double lambda,
    double tol2, double* __restrict__ part, CgState* __restrict__ st) {
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  double s = 0.0;
  const f32x4 z4 = {0.f, 0.f, 0.f, 0.f};
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n4; i += stride) {
    const f32x4 gv = ((const f32x4*)g)[i];
    ((f32x4*)x)[i] = z4;
    ((f32x4*)r)[i] = gv;
    ((f32x4*)p)[i] = -gv;
    ((f32x4*)nd)[i] = z4;
    s += (double)gv[0] * gv[0] + (double)gv[1] * gv[1] +
         (double)gv[2] * gv[2] + (double)gv[3] * gv[3];
  }
  for (long long i = n4 * 4 + (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride) {
    const float gv = g[i];
    x[i] = 0.f; r[i] = gv; p[i] = -gv; nd[i] = 0.f;
    s += (double)gv * gv;
  }
  const double v[1] = {s};
  if (!publish<1>(v, part, &st->counter[0], sh)) return;
  const double rr = gather(part, 0, sh);
  if (threadIdx.x == 0) {
    st->rr = rr;
    st->rr0 = rr;
    st->lambda = lambda;
    st->tol2 = tol2;
    st->kappa = st->alpha = st->beta = st->pp = st->pq = st->gp = 0.0;
    st->neg = 0;
    st->neg_pending = 0;
    st->neg_iter = -1;
    st->iters = 0;
    st->products = 0;
    st->j = 0;
    st->status = is_fin(rr) ? 0 : -5;
    st->done = (rr == 0.0 || !is_fin(rr)) ? 1 : 0;
    st->counter[0] = 0;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_curv_dot(
    const float* __restrict__ p, const float* __restrict__ q, long long n,
    int j, double* __restrict__ part, CgState* __restrict__ st) {
  if (st->done) return;
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  double pq = 0.0, pp = 0.0;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n4; i += stride) {
    const f32x4 a = ((const f32x4*)p)[i];
    const f32x4 b = ((const f32x4*)q)[i];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      pq += (double)a[c] * b[c];
      pp += (double)a[c] * a[c];
    }
  }
  for (long long i = n4 * 4 + (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride) {
    pq += (double)p[i] * q[i];
    pp += (double)p[i] * p[i];
  }
  const double v[2] = {pq, pp};
  if (!publish<2>(v, part, &st->counter[1], sh)) return;
  const double tpq = gather(part, 0, sh);
  const double tpp = gather(part, 1, sh);
  if (threadIdx.x == 0) {
    const double kappa = tpq + st->lambda * tpp;
    st->pq = tpq;
    st->pp = tpp;
    st->kappa = kappa;
    st->products = j + 1;
    st->j = j;
    if (!is_fin(kappa)) {
      st->status = -5;
      st->done = 1;
    } else if (kappa <= 0.0) {
      st->neg = 1;
      st->neg_pending = 1;
      st->neg_iter = j;
      st->done = 1;
    } else {
      st->alpha = st->rr / kappa;
    }
    st->counter[1] = 0;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_neg_dot(
    const float* __restrict__ g, const float* __restrict__ p, long long n,
    double* __restrict__ part, CgState* __restrict__ st) {
  if (!st->neg_pending) return;
  __shared__ double sh[4];
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  double gp = 0.0;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n4; i += stride) {
    const f32x4 a = ((const f32x4*)g)[i];
    const f32x4 b = ((const f32x4*)p)[i];
    gp += (double)a[0] * b[0] + (double)a[1] * b[1] + (double)a[2] * b[2] +
          (double)a[3] * b[3];
  }
  for (long long i = n4 * 4 + (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride)
    gp += (double)g[i] * p[i];
  const double v[1] = {gp};
  if (!publish<1>(v, part, &st->counter[2], sh)) return;
  const double t = gather(part, 0, sh);
  if (threadIdx.x == 0) {
    st->gp = t;
    st->counter[2] = 0;
  }
}

// d~ = -sgn(g.p) p with sgn(0) = +1; the step is -g when the detection
// happened at the first iteration, else the current iterate.
extern "C" __global__ __launch_bounds__(256) void hf_cg_neg_write(
    const float* __restrict__ g, const float* __restrict__ p,
    float* __restrict__ x, float* __restrict__ nd, long long n,
    CgState* __restrict__ st) {
  if (!st->neg_pending) return;
  const float coef = st->gp >= 0.0 ? -1.0f : 1.0f;
  const bool first = st->neg_iter == 0;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n4; i += stride) {
    ((f32x4*)nd)[i] = coef * ((const f32x4*)p)[i];
    if (first) ((f32x4*)x)[i] = -((const f32x4*)g)[i];
  }
  for (long long i = n4 * 4 + (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride) {
    nd[i] = coef * p[i];
    if (first) x[i] = -g[i];
  }
  __shared__ bool last;
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    last = atomicAdd(&st->counter[3], 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (last && threadIdx.x == 0) {
    st->neg_pending = 0;
    st->counter[3] = 0;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_update(
    float* __restrict__ x, float* __restrict__ r, const float* __restrict__ p,
    const float* __restrict__ q, long long n, double* __restrict__ part,
    CgState* __restrict__ st) {
  if (st->done) return;
  __shared__ double sh[4];
  const float alpha = (float)st->alpha;
  const float lam = (float)st->lambda;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  double rr = 0.0;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n4; i += stride) {
    const f32x4 pv = ((const f32x4*)p)[i];
    const f32x4 qv = ((const f32x4*)q)[i];
    f32x4 xv = ((f32x4*)x)[i];
    f32x4 rv = ((f32x4*)r)[i];
    xv += alpha * pv;
    rv += alpha * (qv + lam * pv);
    ((f32x4*)x)[i] = xv;
    ((f32x4*)r)[i] = rv;
    rr += (double)rv[0] * rv[0] + (double)rv[1] * rv[1] +
          (double)rv[2] * rv[2] + (double)rv[3] * rv[3];
  }
  for (long long i = n4 * 4 + (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride) {
    const float pv = p[i];
    x[i] += alpha * pv;
    const float rv = r[i] + alpha * (q[i] + lam * pv);
    r[i] = rv;
    rr += (double)rv * rv;
  }
  const double v[1] = {rr};
  if (!publish<1>(v, part, &st->counter[0], sh)) return;
  const double t = gather(part, 0, sh);
  if (threadIdx.x == 0) {
    st->iters = st->j + 1;
    if (!is_fin(t)) {
      st->status = -5;
      st->done = 1;
    } else {
      st->beta = t / st->rr;
      st->rr = t;
      if (st->tol2 > 0.0 && t <= st->tol2 * st->rr0) st->done = 1;
    }
    st->counter[0] = 0;
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_cg_dir(
    const float* __restrict__ r, float* __restrict__ p, long long n,
    const CgState* __restrict__ st) {
  if (st->done) return;
  const float beta = (float)st->beta;
  const long long n4 = n >> 2;
  const long long stride = (long long)gridDim.x * NT;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n4; i += stride)
    ((f32x4*)p)[i] = beta * ((const f32x4*)p)[i] - ((const f32x4*)r)[i];
  for (long long i = n4 * 4 + (long long)blockIdx.x * NT + threadIdx.x; i < n; i += stride)
    p[i] = beta * p[i] - r[i];
}

// ------------------------------------------------------------- launchers
int cg_grid(long long n) {
  long long b = (n + NT * 4 * 4 - 1) / (NT * 4 * 4);
  if (b < 1) b = 1;
  if (b > MAX_GRID) b = MAX_GRID;
  return (int)b;
}

void cg_init(const Launch& L, const float* g, float* x, float* r, float* p,
             float* neg_dir, long long n, double lambda, double tol2,
             double* part, CgState* st) {
  hipLaunchKernelGGL(hf_cg_reset, dim3(1), dim3(64), 0, L.stream, st);
  prof_begin(L, "hf_cg_init");
  hipLaunchKernelGGL(hf_cg_init, dim3(cg_grid(n)), dim3(NT), 0, L.stream, g, x,
                     r, p, neg_dir, n, lambda, tol2, part, st);
  prof_end(L, "hf_cg_init", 0.0, 5.0 * 4.0 * n);
}

void cg_curv_dot(const Launch& L, const float* p, const float* q, long long n,
                 int j, double* part, CgState* st) {
  prof_begin(L, "hf_cg_curv_dot");
  hipLaunchKernelGGL(hf_cg_curv_dot, dim3(cg_grid(n)), dim3(NT), 0, L.stream,
                     p, q, n, j, part, st);
  prof_end(L, "hf_cg_curv_dot", 0.0, 2.0 * 4.0 * n);
}

void cg_neg(const Launch& L, const float* g, const float* p, float* x,
            float* neg_dir, long long n, double* part, CgState* st) {
  prof_begin(L, "hf_cg_neg_dot");
  hipLaunchKernelGGL(hf_cg_neg_dot, dim3(cg_grid(n)), dim3(NT), 0, L.stream, g,
                     p, n, part, st);
  prof_end(L, "hf_cg_neg_dot", 0.0, 0.0);
  prof_begin(L, "hf_cg_neg_write");
  hipLaunchKernelGGL(hf_cg_neg_write, dim3(cg_grid(n)), dim3(NT), 0, L.stream,
                     g, p, x, neg_dir, n, st);
  prof_end(L, "hf_cg_neg_write", 0.0, 0.0);
}

void cg_update(const Launch& L, float* x, float* r, const float* p,
               const float* q, long long n, double* part, CgState* st) {
  prof_begin(L, "hf_cg_update");
  hipLaunchKernelGGL(hf_cg_update, dim3(cg_grid(n)), dim3(NT), 0, L.stream, x,
                     r, p, q, n, part, st);
  prof_end(L, "hf_cg_update", 0.0, 6.0 * 4.0 * n);
}

void cg_dir(const Launch& L, const float* r, float* p, long long n,
            CgState* st) {
  prof_begin(L, "hf_cg_dir");
  hipLaunchKernelGGL(hf_cg_dir, dim3(cg_grid(n)), dim3(NT), 0, L.stream, r, p,
                     n, st);
  prof_end(L, "hf_cg_dir", 0.0, 3.0 * 4.0 * n);
}

}  // namespace hfk
