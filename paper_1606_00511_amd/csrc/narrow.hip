// The cached curvature product of a narrow net in one launch (Sec. 2.1:
// R-forward, the output layer's R-operator, R-backward or the Gauss-Newton
// backward), for nets whose hidden layers are at most 128 wide and whose
// output layer is at most 64 wide.
//
// Every step of the product except the weight gradients is row-local: the
// R-forward of a batch row needs only that row, the softmax R-operator acts
// on one row of logits, and the backward step to layer l - 1 needs only the
// row's Rdelta_l.  A workgroup therefore takes 16 batch rows and all of
// their hidden units, keeps every intermediate row in LDS, and writes out
// only what the weight-gradient GEMMs that follow read: Rdelta_l for every
// layer and, for the Hessian, RA_l.  On small batches this replaces the
// transposes of v, 2L - 1 GEMMs with their split-K passes and the softmax
// R-operator kernel, whose launch latency, not their work, set the time.
//
// Arithmetic per element is that of the epilogues of the separate kernels:
//   RZ_l = RA_{l-1} W_l^T + A_{l-1} V_l^T + c_l  (RZ_1 = X V_1^T + c_1)
//   RA_l = phi'(A_l) RZ_l
//   Rdelta_L = p (RZ_L - p.RZ_L) / B
//   Rdelta_{l-1} = (Rdelta_l W_l [+ delta_l V_l]) phi'(A_{l-1})
//                  [+ E2_{l-1} RZ_{l-1}]     (bracketed terms: Hessian)
// with v16x16x4 fp32 MFMAs; the K order within a block of 16 is permuted
// identically for both operands.
#include "act.h"
#include "hf_internal.h"

namespace hfk {
namespace {

constexpr int RW = 16;       // batch rows per workgroup
constexpr int NW = 8;        // waves; wave w owns output columns 16w .. 16w + 15
constexpr int NT = 64 * NW;
constexpr int LDR = 132;     // LDS row stride (floats): 16-byte row shift
constexpr int MAXH = NARROW_MAX_HIDDEN;
constexpr int MAXL = NARROW_MAX_LAYERS;
constexpr int LDX = NARROW_MAX_INPUT + 4;   // X rows in LDS: 16-byte row shift

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace

extern "C" __global__ __launch_bounds__(512) void hf_narrow_product(NarrowArgs g) {
  if (g.skip && *g.skip) return;
  __shared__ __attribute__((aligned(16))) float sA[MAXL - 1][RW][LDR];   // A_l
  __shared__ __attribute__((aligned(16))) float sRA[2][RW][LDR];         // RA_l
  __shared__ __attribute__((aligned(16))) float sRZ[MAXL - 1][RW][LDR];  // RZ_l (H)
  __shared__ __attribute__((aligned(16))) float sRD[2][RW][LDR];         // RZ_L, Rdelta
  __shared__ __attribute__((aligned(16))) float sX[RW][LDX];             // X rows
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, g16 = lane >> 4;
  const int r0 = blockIdx.x * RW;
  const int L = g.L;
  const int act = g.act;
  const bool hess = g.hess != 0;

  // the cached activations of this workgroup's rows, zero past B and past
  // d_l (columns up to MAXH are read as the next layer's K padding)
  for (int l = 1; l < L; ++l) {
    const float* A = g.A[l];
    const int dl = g.d[l], ldl = g.ld[l];
    for (int e = tid; e < RW * MAXH; e += NT) {
      const int r = e / MAXH, c = e - r * MAXH;
      sA[l - 1][r][c] = (r0 + r < g.B && c < dl) ? A[(size_t)(r0 + r) * ldl + c] : 0.0f;
    }
  }

  // the workgroup's rows of X, read once (the waves share them), with
  // zeros past B and from d_0 to the next multiple of 16
  {
    const int d0 = g.d[0];
    const int q4 = (d0 + 15) >> 2 & ~3;    // float4s per row, K padded to 16
    for (int e = tid; e < RW * q4; e += NT) {
      const int r = e / q4, c = 4 * (e - r * q4);
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      if (r0 + r < g.B && c < d0) x = *(const f32x4*)(g.X + (size_t)(r0 + r) * d0 + c);
      *(f32x4*)&sX[r][c] = x;
    }
  }
  __syncthreads();

  // ---- layer 1: RZ_1 = X V_1^T + c_1 over K = d_0 (16-byte loads; the
  // host checks d_0 % 4 == 0, d_0 <= NARROW_MAX_INPUT and 16-byte alignment
  // of X and v)
  {
    const int d0 = g.d[0], d1 = g.d[1];
    const int n0 = 16 * wave;
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
    if (n0 < d1) {
      const bool vr = n0 + i16 < d1;
      const float* xs = &sX[i16][4 * g16];
      const float* vp = g.v + g.offW[1] + (size_t)(vr ? n0 + i16 : 0) * d0 + 4 * g16;
      // Full K blocks of v in stages of U blocks: the next stage's U loads
      // are issued before the current stage's 4U MFMAs, with no branch
      // around them, so that the MFMAs wait only for their own stage.  A
      // column past d_1 reads column 0's row instead: it feeds only outputs
      // that are never stored.  X comes from LDS.
      const int nfull = d0 >> 4;
      constexpr int U = 8;
      const int nst = nfull / U;
      f32x4 va[U];
      auto load = [&](int b0, f32x4 (&w)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) w[u] = *(const f32x4*)(vp + 16 * (b0 + u));
      };
      if (nst > 0) load(0, va);
      for (int st = 0; st < nst; ++st) {
        // the last stage reloads itself (in bounds, unused)
        const int nb = (st + 1 < nst ? st + 1 : st) * U;
        f32x4 vn[U];
        load(nb, vn);
        // keep the scheduler from sinking these loads to their uses
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const f32x4 xa = *(const f32x4*)(xs + 16 * (st * U + u));
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (u & 1) acc1 = mfma16(xa[q], va[u][q], acc1);
            else acc0 = mfma16(xa[q], va[u][q], acc0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u) va[u] = vn[u];
      }
      // the remaining full blocks, their loads issued together
      {
        const int b0 = nst * U;
        f32x4 vr2[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int b = b0 + u < nfull ? b0 + u : 0;
          vr2[u] = *(const f32x4*)(vp + 16 * b);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (b0 + u < nfull) {
            const f32x4 xa = *(const f32x4*)(xs + 16 * (b0 + u));
#pragma unroll
            for (int q = 0; q < 4; ++q) acc0 = mfma16(xa[q], vr2[u][q], acc0);
          }
      }
      const int k0 = nfull << 4;
      if (k0 < d0) {     // ragged last block: LDS holds zeros past d_0
        const f32x4 xa = *(const f32x4*)(xs + k0);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = k0 + 4 * g16 + q;
          const float b = k < d0 ? vp[k0 + q] : 0.0f;
          acc0 = mfma16(xa[q], b, acc0);
        }
      }
      // lane (i16, g16) holds rows 4 g16 .. 4 g16 + 3 of column n0 + i16
      const int n = n0 + i16;
      const bool nv = n < d1;
      const float cb = nv ? g.v[g.offB[1] + n] : 0.0f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 4 * g16 + r;
        const float rz = acc0[r] + acc1[r] + cb;
        const float ra = nv ? act_d1(act, sA[0][row][n]) * rz : 0.0f;
        sRA[0][row][n] = ra;
        if (hess) {
          sRZ[0][row][n] = nv ? rz : 0.0f;
          if (nv && r0 + row < g.B)
            g.RA[1][(size_t)(r0 + row) * (g.ldRA ? g.ldRA : g.ld[1]) + n] = ra;
        }
      }
    }
  }
  __syncthreads();

  // ---- layers 2 .. L: RZ_l = RA_{l-1} W_l^T + A_{l-1} V_l^T + c_l over
  // K = d_{l-1} <= 128; A operands from LDS, weights K-contiguous rows
  for (int l = 2; l <= L; ++l) {
    const int dk = g.d[l - 1], dn = g.d[l];
    const int kpad = (dk + 15) & ~15;
    const int n0 = 16 * wave;
    const float(*xr)[LDR] = sRA[(l - 2) & 1];
    const float(*xa)[LDR] = sA[l - 2];
    if (n0 < dn) {
      const int n = n0 + i16;
      const bool nv = n < dn;
      const float* wrow = g.W + g.offW[l] + (size_t)(nv ? n : 0) * dk;
      const float* vrow = g.v + g.offW[l] + (size_t)(nv ? n : 0) * dk;
      // every weight value this lane feeds, loaded before the first MFMA
      constexpr int NB = MAXH / 16;
      float bw[NB][4], bv[NB][4];
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = 16 * b + 4 * g16 + q;
          const bool kv = nv && k < dk;
          bw[b][q] = kv ? wrow[k] : 0.0f;
          bv[b][q] = kv ? vrow[k] : 0.0f;
        }
      f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (16 * b < kpad) {
          const f32x4 a0 = *(const f32x4*)&xr[i16][16 * b + 4 * g16];
          const f32x4 a1 = *(const f32x4*)&xa[i16][16 * b + 4 * g16];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc0 = mfma16(a0[q], bw[b][q], acc0);
            acc1 = mfma16(a1[q], bv[b][q], acc1);
          }
        }
      }
      const float cb = nv ? g.v[g.offB[l] + n] : 0.0f;
      if (l < L) {
        float(*yo)[LDR] = sRA[(l - 1) & 1];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 4 * g16 + r;
          const float rz = acc0[r] + acc1[r] + cb;
          const float ra = nv ? act_d1(act, sA[l - 1][row][n]) * rz : 0.0f;
          yo[row][n] = ra;
          if (hess) {
            sRZ[l - 1][row][n] = nv ? rz : 0.0f;
            if (nv && r0 + row < g.B)
              g.RA[l][(size_t)(r0 + row) * (g.ldRA ? g.ldRA : g.ld[l]) + n] = ra;
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) sRD[0][4 * g16 + r][n] = nv ? acc0[r] + acc1[r] + cb : 0.0f;
      }
    }
    __syncthreads();
  }

  // ---- output layer: Rdelta_L = p (RZ_L - p.RZ_L) / B, one wave per row
  // (columns lane < C <= 64), rows 2 wave and 2 wave + 1
  {
    const int C = g.d[L], ldL = g.ld[L];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rr = 2 * wave + h;
      const int row = r0 + rr;
      const bool cv = lane < C, rv = row < g.B;
      const float p = (cv && rv) ? g.P[(size_t)row * ldL + lane] : 0.0f;
      const float rz = cv ? sRD[0][rr][lane] : 0.0f;
      const float dot = wave_sum(p * rz);
      const float rd = p * (rz - dot) * g.invB;
      sRD[1][rr][lane] = rd;
      if (cv && rv) g.RD[L][(size_t)row * (g.ldRD ? g.ldRD : ldL) + lane] = rd;
    }
  }
  __syncthreads();

  // ---- backward, l = L .. 2: Rdelta_{l-1} = (Rdelta_l W_l [+ delta_l V_l])
  // phi'(A_{l-1}) [+ E2_{l-1} RZ_{l-1}] over K = d_l; the weights enter as
  // W_l[k][n] (n contiguous)
  int cur = 1;
  for (int l = L; l >= 2; --l) {
    const int dk = g.d[l], dn = g.d[l - 1];
    const int kpad = (dk + 15) & ~15;
    const int n0 = 16 * wave;
    const float(*xr)[LDR] = sRD[cur];
    float(*yo)[LDR] = sRD[cur ^ 1];
    if (n0 < dn) {
      const int n = n0 + i16;
      const bool nv = n < dn;
      const float* wcol = g.W + g.offW[l] + (nv ? n : 0);
      const float* vcol = g.v + g.offW[l] + (nv ? n : 0);
      const bool dr = r0 + i16 < g.B;
      const float* drow = hess ? g.D[l] + (size_t)(dr ? r0 + i16 : 0) * g.ld[l] : nullptr;
      // every weight (and delta_l) value this lane feeds, loaded first
      constexpr int NB = MAXH / 16;
      float bw[NB][4], bv[NB][4], ad[NB][4];
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = 16 * b + 4 * g16 + q;
          const bool kv = k < dk;
          bw[b][q] = (kv && nv) ? wcol[(size_t)k * dn] : 0.0f;
          bv[b][q] = (hess && kv && nv) ? vcol[(size_t)k * dn] : 0.0f;
          ad[b][q] = (hess && kv && dr) ? drow[k] : 0.0f;
        }
      f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (16 * b < kpad) {
          const f32x4 a0 = *(const f32x4*)&xr[i16][16 * b + 4 * g16];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc0 = mfma16(a0[q], bw[b][q], acc0);
            if (hess) acc1 = mfma16(ad[b][q], bv[b][q], acc1);
          }
        }
      }
      const float* e2 = hess ? g.E2[l - 1] : nullptr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 4 * g16 + r;
        const bool rv = r0 + row < g.B;
        float rd = (acc0[r] + acc1[r]) * act_d1(act, sA[l - 2][row][n]);
        if (hess)
          rd += ((nv && rv) ? e2[(size_t)(r0 + row) * g.ld[l - 1] + n] : 0.0f) *
                sRZ[l - 2][row][n];
        rd = nv ? rd : 0.0f;
        yo[row][n] = rd;
        if (nv && rv)
          g.RD[l - 1][(size_t)(r0 + row) * (g.ldRD ? g.ldRD : g.ld[l - 1]) + n] = rd;
      }
    }
    __syncthreads();
    cur ^= 1;
  }
}

// out[i] for parameter i: a weight of layer l at (m, k) is the diagonal
// block's element (roff[l] + m, yoff[l - 1] + k), a bias of layer l its row
// roff[l] + m; both summed over the splits in split order (fp64).  With dpart
// (a CG iteration's product, p its direction): the block's partials of p.q
// and p.p, q being the stored fp32 out, summed in fp64 in a fixed order.
extern "C" __global__ __launch_bounds__(256) void hf_narrow_scatter(
    const float* __restrict__ part, const double* __restrict__ bpart, int S,
    NarrowCat nc, float* __restrict__ out, const int* __restrict__ skip,
    const float* __restrict__ p, double* __restrict__ dpart,
    CgState* __restrict__ st, int j) {
  // an iteration replayed from a graph: publish its index for the vector
  // kernels after this one, -1 once the solve has stopped
  if (dpart && j < 0 && blockIdx.x == 0 && threadIdx.x == 0)
    st->jc = st->done ? -1 : st->jn;
  if (skip && *skip) return;
  const size_t mn = (size_t)nc.M * nc.N;
  double pq = 0.0, pp = 0.0;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < nc.n;
       i += (long long)gridDim.x * 256) {
    int l = 1;
    while (l < nc.L && i >= nc.offW[l + 1]) ++l;
    double t = 0.0;
    if (i < nc.offB[l]) {
      const long long loc = i - nc.offW[l];
      const int dk = nc.d[l - 1];
      const int m = (int)(loc / dk), k = (int)(loc - (long long)m * dk);
      const float* src = part + (size_t)(nc.roff[l] + m) * nc.N + nc.yoff[l - 1] + k;
      for (int z0 = 0; z0 < S; z0 += 8) {
        float v[8];
#pragma unroll
        for (int z = 0; z < 8; ++z) v[z] = z0 + z < S ? src[(size_t)(z0 + z) * mn] : 0.0f;
#pragma unroll
        for (int z = 0; z < 8; ++z)
          if (z0 + z < S) t += (double)v[z];
      }
    } else {
      const int m = (int)(i - nc.offB[l]);
      for (int z = 0; z < S; ++z) t += bpart[(size_t)z * nc.M + nc.roff[l] + m];
    }
    const float q = (float)t;
    out[i] = q;
    if (dpart) {
      const double pv = p[i];
      pq += pv * (double)q;
      pp += pv * pv;
    }
  }
  if (!dpart) return;
  __shared__ double sh[2][4];
  pq = wave_sum_d(pq);
  pp = wave_sum_d(pp);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh[0][w] = pq;
    sh[1][w] = pp;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    dpart[blockIdx.x] = (sh[0][0] + sh[0][1]) + (sh[0][2] + sh[0][3]);
    dpart[CG_MAX_GRID + blockIdx.x] = (sh[1][0] + sh[1][1]) + (sh[1][2] + sh[1][3]);
  }
}

extern "C" __global__ __launch_bounds__(256) void hf_narrow_gather(NarrowGather g) {
  const int k = blockIdx.y;
  if (k >= g.nblk) return;
  const float* __restrict__ src = g.src[k];
  float* __restrict__ dst = g.dst[k];
  const int cols = g.cols[k], lds = g.lds[k], ldd = g.ldd[g.which[k]];
  const long long tot = (long long)g.B * cols;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < tot;
       e += (long long)gridDim.x * 256) {
    const int r = (int)(e / cols), c = (int)(e - (long long)r * cols);
    dst[(size_t)r * ldd + c] = src[(size_t)r * lds + c];
  }
}

int narrow_scatter(const Launch& Lc, const float* part, const double* bpart,
                   int splits, const NarrowCat& nc, float* out, const int* skip,
                   const CgDotFuse* dot) {
  const int nb = (int)std::min<long long>((nc.n + 255) / 256, CG_MAX_GRID);
  prof_begin(Lc, "hf_narrow_scatter");
  hipExtLaunchKernelGGL(hf_narrow_scatter, dim3((unsigned)nb), dim3(256), 0, Lc.stream,
                        prof_a(Lc), prof_b(Lc), 0, part, bpart, splits, nc, out, skip,
                        dot ? dot->p : nullptr, dot ? dot->part : nullptr,
                        dot ? dot->st : nullptr, dot ? dot->j : 0);
  prof_end(Lc, "hf_narrow_scatter", 0.0, 4.0 * (splits + 1 + (dot ? 1 : 0)) * (double)nc.n);
  return dot ? nb : 0;
}

void narrow_gather(const Launch& Lc, const NarrowGather& g) {
  long long most = 0;
  for (int k = 0; k < g.nblk; ++k) most = std::max<long long>(most, (long long)g.B * g.cols[k]);
  const long long nb = std::max<long long>(1, std::min<long long>((most + 255) / 256, 256));
  prof_begin(Lc, "hf_narrow_gather");
  hipExtLaunchKernelGGL(hf_narrow_gather, dim3((unsigned)nb, (unsigned)g.nblk), dim3(256), 0,
                        Lc.stream, prof_a(Lc), prof_b(Lc), 0, g);
  double by = 0.0;
  for (int k = 0; k < g.nblk; ++k) by += 8.0 * g.B * g.cols[k];
  prof_end(Lc, "hf_narrow_gather", 0.0, by);
}

bool narrow_eligible(int L, const int* d, const float* X, const float* v) {
  if (L < 2 || L > NARROW_MAX_LAYERS) return false;
  for (int l = 1; l < L; ++l)
    if (d[l] > NARROW_MAX_HIDDEN) return false;
  if (d[L] > 64) return false;
  if (d[0] % 4 || d[0] > NARROW_MAX_INPUT) return false;
  if (((uintptr_t)X & 15u) || ((uintptr_t)v & 15u)) return false;
  return true;
}

void narrow_product(const Launch& Lc, const NarrowArgs& a) {
  const int nb = (a.B + RW - 1) / RW;
  // algorithmic work: the GEMM flops of the replaced passes
  double fl = 2.0 * a.B * a.d[0] * a.d[1];
  for (int l = 2; l <= a.L; ++l)
    fl += 2.0 * a.B * a.d[l - 1] * a.d[l] * (a.hess ? 4.0 : 3.0);
  prof_begin(Lc, "hf_narrow_product");
  hipExtLaunchKernelGGL(hf_narrow_product, dim3(nb), dim3(NT), 0, Lc.stream,
                        prof_a(Lc), prof_b(Lc), 0, a);
  prof_end(Lc, "hf_narrow_product", fl, 4.0 * a.B * (a.d[0] + 4.0 * a.d[1]));
}

}  // namespace hfk
