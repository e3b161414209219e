// The narrow nets' passes (Sec. 2.1 and Alg. 1 step 1), for nets with 2 to 4
// weight layers whose hidden layers are at most 128 wide and whose output
// layer is at most 64 wide: the cached curvature product (R-forward, the
// output layer's R-operator, R-backward or the Gauss-Newton backward), the
// solve's cache (forward pass, softmax and, for the Hessian, the backward
// pass of delta and of the phi'' term) and the gradient's passes, each up
// to the weight gradients; then every layer's weight gradient from one GEMM
// over concatenated columns, whose diagonal blocks hf_narrow_scatter writes
// out in the parameter layout.
//
// Every step except the weight gradients is row-local: the R-forward of a
// batch row needs only that row, the softmax and its R-operator act on one
// row of logits, and the backward step to layer l - 1 needs only the row's
// delta_l or Rdelta_l.  A workgroup therefore takes a few batch rows and all
// of their hidden units, keeps every intermediate row in LDS, and writes out
// only what the weight-gradient GEMM reads.  On small batches this replaces
// chains of GEMMs with their split-K passes and row kernels, whose launch
// latency, not their work, set the time.  The first layer, whose K is the
// input width, is a kernel of its own below 1,025 rows (hf_narrow_layer1,
// in tiles); above, hf_narrow_product holds 16 rows per workgroup and does
// it inside.
//
// The product's arithmetic per element is that of the epilogues of the
// separate kernels:
//   RZ_l = RA_{l-1} W_l^T + A_{l-1} V_l^T + c_l  (RZ_1 = X V_1^T + c_1)
//   RA_l = phi'(A_l) RZ_l
//   Rdelta_L = p (RZ_L - p.RZ_L) / B
//   Rdelta_{l-1} = (Rdelta_l W_l [+ delta_l V_l]) phi'(A_{l-1})
//                  [+ E2_{l-1} RZ_{l-1}]     (bracketed terms: Hessian)
// The 16-row kernel uses v16x16x4 fp32 MFMAs, the K order within a block of
// 16 permuted identically for both operands.
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
  // the wave index in a scalar register: the loops and branches on it are
  // uniform
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i16 = lane & 15, g16 = lane >> 4;
  const int r0 = blockIdx.x * RW;
  const int L = g.L;
  const int act = g.act;
  const bool hess = g.hess != 0;
  const int d0 = g.d[0], d1 = g.d[1];

  // Layer 1's slots of V_1 (below) are requested first, then the rows of
  // the cached activations and of X; every load is issued before any is
  // used (a clamped index where the value is not wanted), so the workgroup
  // waits on memory once.
  const int n0 = 16 * wave;
  const bool l1 = n0 < d1;                       // this wave has layer-1 columns
  const int nfull = d0 >> 4;
  // a column past d_1 reads column 0's row: it feeds only outputs that are
  // never stored
  const float* vp = g.v + g.offW[1] + (size_t)(n0 + i16 < d1 ? n0 + i16 : 0) * d0 + 4 * g16;
  constexpr int U = 8;                           // K blocks in flight
  f32x4 vs[U];
  auto vload = [&](int b, int u) {
    vs[u] = *(const f32x4*)(vp + 16 * (b < nfull ? b : nfull - 1));
  };
  if (l1 && nfull > 0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      vload(u, u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  {
    // the cached activations of this workgroup's rows, zero past B and past
    // d_l (columns up to MAXH are read as the next layer's K padding)
    constexpr int PE = RW * MAXH / NT;           // elements per thread and layer
    float qa[MAXL - 1][PE];
#pragma unroll
    for (int l = 1; l < MAXL; ++l)
#pragma unroll
      for (int j = 0; j < PE; ++j) {
        const int e = tid + NT * j, r = e / MAXH, c = e - r * MAXH;
        const bool ok = l < L && r0 + r < g.B && c < g.d[l < L ? l : 1];
        qa[l - 1][j] = (l < L ? g.A[l] : g.X)[ok ? (size_t)(r0 + r) * g.ld[l] + c : 0];
      }
    // the workgroup's rows of X, read once (the waves share them), with
    // zeros past B and from d_0 to the next multiple of 16: at most
    // RW * NARROW_MAX_INPUT / 4 = 8 NT float4s
    constexpr int PX = RW * NARROW_MAX_INPUT / 4 / NT;
    const int q4 = (d0 + 15) >> 2 & ~3;          // float4s per row, K padded to 16
    f32x4 qx[PX];
#pragma unroll
    for (int j = 0; j < PX; ++j) {
      const int e = tid + NT * j, r = e / q4, c = 4 * (e - r * q4);
      const bool ok = e < RW * q4 && r0 + r < g.B && c < d0;
      qx[j] = *(const f32x4*)(g.X + (ok ? (size_t)(r0 + r) * d0 + c : 0));
    }
#pragma unroll
    for (int l = 1; l < MAXL; ++l)
#pragma unroll
      for (int j = 0; j < PE; ++j) {
        const int e = tid + NT * j, r = e / MAXH, c = e - r * MAXH;
        const bool ok = l < L && r0 + r < g.B && c < g.d[l < L ? l : 1];
        if (l < L) sA[l - 1][r][c] = ok ? qa[l - 1][j] : 0.0f;
      }
#pragma unroll
    for (int j = 0; j < PX; ++j) {
      const int e = tid + NT * j, r = e / q4, c = 4 * (e - r * q4);
      const bool ok = e < RW * q4 && r0 + r < g.B && c < d0;
      if (e < RW * q4) *(f32x4*)&sX[r][c] = ok ? qx[j] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  __syncthreads();

  // ---- layer 1: RZ_1 = X V_1^T + c_1 over K = d_0 (16-byte loads; the
  // host checks d_0 % 4 == 0, d_0 <= NARROW_MAX_INPUT and 16-byte alignment
  // of X and v)
  {
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
    if (l1) {
      const float* xs = &sX[i16][4 * g16];
      // The full K blocks, U in flight: slot u holds block t0 + u and, once
      // its MFMAs have read it, is reloaded with block t0 + u + U (the last
      // full block again past the end: in bounds, unused).  No branch
      // around the loads and no copy between registers (either would make
      // the compiler wait for loads in flight).  X comes from LDS.
      for (int t0 = 0; t0 < nfull; t0 += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (t0 + u < nfull) {
            const f32x4 xa = *(const f32x4*)(xs + 16 * (t0 + u));
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (u & 1) acc1 = mfma16(xa[q], vs[u][q], acc1);
              else acc0 = mfma16(xa[q], vs[u][q], acc0);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
          vload(t0 + u + U, u);
          __builtin_amdgcn_sched_barrier(0);
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
      // every weight value this lane feeds, loaded before the first MFMA;
      // past d_{l-1} the loads read the row's first weight, unmasked (the A
      // operands are zero there up to the block's end)
      constexpr int NB = MAXH / 16;
      float bw[NB][4], bv[NB][4];
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = 16 * b + 4 * g16 + q;
          const int kc = k < dk ? k : 0;
          bw[b][q] = wrow[kc];
          bv[b][q] = vrow[kc];
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
      // every weight (and delta_l) value this lane feeds, loaded first;
      // past d_l the weight loads read the column's first weight, unmasked
      // (Rdelta_l is zero there up to the block's end), and delta_l is
      // masked to zero (its partner, V_l, is not)
      constexpr int NB = MAXH / 16;
      float bw[NB][4], bv[NB][4], ad[NB][4];
      const float* dsrc = hess ? drow : wcol;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = 16 * b + 4 * g16 + q;
          const bool kv = k < dk;
          const size_t kc = kv ? (size_t)k * dn : 0;
          bw[b][q] = wcol[kc];
          bv[b][q] = vcol[kc];
          const float dv = dsrc[kv && dr ? k : 0];
          ad[b][q] = hess && kv && dr ? dv : 0.0f;
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

// ------------------------------------------------------------------------
// The same product in two launches, for batches whose 16-row grid leaves
// most compute units idle: hf_narrow_layer1 (below) forms RZ_1 in
// tiles that each read only part of V_1, and hf_narrow_product4 does the
// rest with 4 batch rows per workgroup.  (A workgroup holding all hidden
// units of its rows must stream all of V_1, which costs a compute unit
// several microseconds at the 784-input widths.)  The row-local steps use
// v4x4x1 fp32 MFMAs with the A operand broadcast to all 16 blocks: one
// instruction multiplies the 4 rows' values at one k by 64 output columns'
// values at that k, so a wave covers 64 columns and a run of K; the 8 waves
// split the columns into groups of 64 and K into slices, and their partial
// sums are added in LDS in a fixed order.
namespace {

constexpr int R4 = 4;                             // batch rows per workgroup
constexpr int LR4 = NARROW_MAX_HIDDEN + 16;       // LDS row stride: k + 16 i
static_assert(NT == R4 * MAXH, "one thread per (row, column) of a layer");
// acc += sum_a x(a) b[a]: x(a) is the A operand of lanes 4a .. 4a + 3 (row
// i = lane & 3 at k = a), b[a] this lane's column value at k = a
#define HF_M4(a) acc = __builtin_amdgcn_mfma_f32_4x4x1f32(xa, b[a], acc, 4, a, 0);
__device__ __forceinline__ f32x4 mfma4x16(float xa, const float (&b)[16], f32x4 acc) {
  HF_M4(0) HF_M4(1) HF_M4(2) HF_M4(3) HF_M4(4) HF_M4(5) HF_M4(6) HF_M4(7)
  HF_M4(8) HF_M4(9) HF_M4(10) HF_M4(11) HF_M4(12) HF_M4(13) HF_M4(14) HF_M4(15)
  return acc;
}
#undef HF_M4

}  // namespace

extern "C" __global__ __launch_bounds__(512) void hf_narrow_product4(NarrowArgs g) {
  if (g.skip && *g.skip) return;
  constexpr int ML = MAXL - 1;
  __shared__ __attribute__((aligned(16))) float sA[ML][R4][LR4];   // A_l
  __shared__ __attribute__((aligned(16))) float sRA[2][R4][LR4];   // RA_l
  __shared__ __attribute__((aligned(16))) float sRZ[ML][R4][LR4];  // RZ_l (H)
  __shared__ __attribute__((aligned(16))) float sRD[2][R4][LR4];   // RZ_L, Rdelta
  __shared__ __attribute__((aligned(16))) float sD[ML][R4][LR4];   // delta_l (H)
  __shared__ __attribute__((aligned(16))) float sE2[ML][R4][LR4];  // E2_l (H)
  __shared__ __attribute__((aligned(16))) float sP[R4][64];        // p
  __shared__ __attribute__((aligned(16))) float red[NW][R4][64];   // partials
  // the wave index in a scalar register: the loops and branches on it are
  // uniform
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int xi = lane & 3, xk = lane >> 2;   // A operand: row, k within 16
  const int r0 = blockIdx.x * R4;
  const int L = g.L;
  const int act = g.act;
  const bool hess = g.hess != 0;

  // Weight values of layer l for this lane, for the forward step (fw: W_l
  // and V_l at [c][k], c an output column) or the backward step (W_l and
  // V_l at [k][c]): wave (column group cg, K slice sl) takes the blocks sl
  // and sl + nks of 16 k.  Past the layer's widths the loads read the
  // layer's first weight, unmasked (masking the value would wait for the
  // load): past d_k they meet the zero K padding of the LDS rows, and a
  // column past d_n feeds only outputs that are never stored.
  auto weights = [&](int l, bool fw, float (&bw)[2][16], float (&bv)[2][16]) {
    const int dk = fw ? g.d[l - 1] : g.d[l], dn = fw ? g.d[l] : g.d[l - 1];
    const int ncg = (dn + 63) >> 6, nks = NW / ncg;
    const int cg = wave % ncg, sl = wave / ncg;
    const int c = 64 * cg + lane;
    const bool cv = c < dn;
    const float* w = g.W + g.offW[l];
    const float* vv = g.v + g.offW[l];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const int k = 16 * (sl + h * nks) + a;
        const bool kv = cv && k < dk;
        const size_t o = kv ? (fw ? (size_t)c * dk + k : (size_t)k * dn + c) : 0;
        bw[h][a] = w[o];
        bv[h][a] = vv[o];
      }
  };
  // the first forward and the first backward step's weights, requested
  // with the rows below
  float fw2[2][16], fv2[2][16], bwL[2][16], bvL[2][16];
  weights(2, true, fw2, fv2);
  weights(L, false, bwL, bvL);

  // the workgroup's rows of the cached operands and of RZ_1, zero past B
  // and past the layer's width (read as K padding up to the next multiple
  // of 16); every load issued (an operand the net or the mode does not
  // have reads X[0] instead, and its value is not used)
  {
    const int pr = tid / MAXH, pc = tid - pr * MAXH;   // NT = R4 * MAXH
    const bool prv = r0 + pr < g.B;
    const int prow = prv ? r0 + pr : 0;
    float qa[ML], qe[ML], qd[ML], qp, qz;
#pragma unroll
    for (int l = 1; l <= ML; ++l) {
      const bool has = l < L, hd = hess && l + 1 <= L;
      const bool ok = prv && has && pc < g.d[l];
      const bool okd = prv && hd && pc < g.d[hd ? l + 1 : 1];
      const size_t o = ok ? (size_t)prow * g.ld[l] + pc : 0;
      qa[l - 1] = (has ? g.A[l] : g.X)[o];
      qe[l - 1] = (has && hess ? g.E2[l] : g.X)[o];
      qd[l - 1] = (hd ? g.D[l + 1] : g.X)[okd ? (size_t)prow * g.ld[l + 1] + pc : 0];
    }
    {
      const bool ok = prv && pc < g.d[L] && pc < 64;
      qp = g.P[ok ? (size_t)prow * g.ld[L] + pc : 0];
    }
    const bool okz = prv && pc < g.d[1];
    qz = g.RZ1[okz ? (size_t)prow * g.ld[1] + pc : 0];
#pragma unroll
    for (int l = 1; l <= ML; ++l) {
      const bool ok = prv && pc < g.d[l];
      if (l < L) sA[l - 1][pr][pc] = ok ? qa[l - 1] : 0.0f;
      if (hess && l < L) sE2[l - 1][pr][pc] = ok ? qe[l - 1] : 0.0f;
      if (hess && l + 1 <= L) sD[l - 1][pr][pc] = (prv && pc < g.d[l + 1]) ? qd[l - 1] : 0.0f;
    }
    if (pc < 64) sP[pr][pc] = (prv && pc < g.d[L]) ? qp : 0.0f;
    // RA_1 = phi'(A_1) RZ_1
    const float rz = okz ? qz : 0.0f;
    const float ra = okz ? act_d1(act, qa[0]) * rz : 0.0f;
    sRA[0][pr][pc] = ra;
    if (hess) {
      sRZ[0][pr][pc] = rz;
      if (okz) g.RA[1][(size_t)prow * (g.ldRA ? g.ldRA : g.ld[1]) + pc] = ra;
    }
  }
  __syncthreads();

  // Cross-wave sum of the partial tiles in red (wave = slice * ncg + cg):
  // thread (row tid / 128, column tid % 128) gets its column's total.
  auto total = [&](int ncg, int nks, int i, int c) {
    float s = 0.0f;
    for (int k = 0; k < nks; ++k) s += red[k * ncg + (c >> 6)][i][c & 63];
    return s;
  };

  // ---- layers 2 .. L: RZ_l = RA_{l-1} W_l^T + A_{l-1} V_l^T + c_l over
  // K = d_{l-1} <= 128 (at most 8 blocks: a wave takes blocks sl, sl + nks)
  for (int l = 2; l <= L; ++l) {
    const int dk = g.d[l - 1], dn = g.d[l];
    const int ncg = (dn + 63) >> 6, nks = NW / ncg;
    const int sl = wave / ncg;
    const int nblk = (dk + 15) >> 4;
    float bw[2][16], bv[2][16];
    if (l == 2) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          bw[h][a] = fw2[h][a];
          bv[h][a] = fv2[h][a];
        }
    } else {
      weights(l, true, bw, bv);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int b = sl + h * nks;
      if (b < nblk) {
        acc = mfma4x16(sRA[(l - 2) & 1][xi][16 * b + xk], bw[h], acc);
        acc = mfma4x16(sA[l - 2][xi][16 * b + xk], bv[h], acc);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    {
      const int i = tid >> 7, cc = tid & (MAXH - 1);
      float rz = 0.0f;
      if (cc < dn) rz = total(ncg, nks, i, cc) + g.v[g.offB[l] + cc];
      if (l < L) {
        const float ra = cc < dn ? act_d1(act, sA[l - 1][i][cc]) * rz : 0.0f;
        sRA[(l - 1) & 1][i][cc] = ra;
        if (hess) {
          sRZ[l - 1][i][cc] = rz;
          if (cc < dn && r0 + i < g.B)
            g.RA[l][(size_t)(r0 + i) * (g.ldRA ? g.ldRA : g.ld[l]) + cc] = ra;
        }
      } else {
        sRD[0][i][cc] = rz;
      }
    }
    __syncthreads();
  }

  // ---- output layer: Rdelta_L = p (RZ_L - p.RZ_L) / B, wave i < 4 takes
  // row i (columns lane < C <= 64)
  if (wave < R4) {
    const int i = wave, C = g.d[L];
    const bool cv = lane < C;
    const float p = sP[i][lane];
    const float rz = cv ? sRD[0][i][lane] : 0.0f;
    const float dot = wave_sum(p * rz);
    const float rd = cv ? p * (rz - dot) * g.invB : 0.0f;
    sRD[1][i][lane] = rd;
    if (cv && r0 + i < g.B)
      g.RD[L][(size_t)(r0 + i) * (g.ldRD ? g.ldRD : g.ld[L]) + lane] = rd;
  }
  __syncthreads();

  // ---- backward, l = L .. 2: Rdelta_{l-1} = (Rdelta_l W_l [+ delta_l V_l])
  // phi'(A_{l-1}) [+ E2_{l-1} RZ_{l-1}] over K = d_l
  int cur = 1;
  for (int l = L; l >= 2; --l) {
    const int dk = g.d[l], dn = g.d[l - 1];
    const int ncg = (dn + 63) >> 6, nks = NW / ncg;
    const int sl = wave / ncg;
    const int nblk = (dk + 15) >> 4;
    float bw[2][16], bv[2][16];
    if (l == L) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          bw[h][a] = bwL[h][a];
          bv[h][a] = bvL[h][a];
        }
    } else {
      weights(l, false, bw, bv);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int b = sl + h * nks;
      if (b < nblk) {
        acc = mfma4x16(sRD[cur][xi][16 * b + xk], bw[h], acc);
        if (hess) acc = mfma4x16(sD[l - 2][xi][16 * b + xk], bv[h], acc);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    {
      const int i = tid >> 7, cc = tid & (MAXH - 1);
      float rd = 0.0f;
      if (cc < dn) {
        rd = total(ncg, nks, i, cc) * act_d1(act, sA[l - 2][i][cc]);
        if (hess) rd += sE2[l - 2][i][cc] * sRZ[l - 2][i][cc];
        if (r0 + i < g.B)
          g.RD[l - 1][(size_t)(r0 + i) * (g.ldRD ? g.ldRD : g.ld[l - 1]) + cc] = rd;
      }
      sRD[cur ^ 1][i][cc] = rd;
    }
    __syncthreads();
    cur ^= 1;
  }
}

// ------------------------------------------------------------------------
// Layer 1 of the narrow product on its own: RZ_1 = X V_1^T + c_1 in tiles
// of 16 batch rows x 32 hidden units, so that a workgroup streams only its
// 32 rows of V_1 (a workgroup holding all hidden units of its rows would
// stream all of V_1).  Four waves split K into quarters of whole 16-blocks
// and add their partial tiles in LDS in a fixed order.  v16x16x4 fp32
// MFMAs, the K order within a block of 16 permuted identically for both
// operands; 16-byte loads (the host checks d_0 % 4 == 0 and the 16-byte
// alignment of X and v).  With act >= 0 (v = W, c = b) it is the forward
// layer instead: A_1 = phi(X W_1^T + b_1).
namespace {
constexpr int T1R = 16, T1C = 32;                 // tile: rows x hidden units
constexpr int NT1 = 256;
constexpr int U1 = 4;                             // 16-blocks per load stage
}  // namespace

extern "C" __global__ __launch_bounds__(256) void hf_narrow_layer1(
    const float* __restrict__ X, const float* __restrict__ v, int B, int d0,
    int d1, long long offW1, long long offB1, float* __restrict__ rz, int ldrz,
    int act, const int* __restrict__ skip) {
  if (skip && *skip) return;
  __shared__ f32x4 red[4][2][64];                  // per wave, subtile, lane
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i16 = lane & 15, g16 = lane >> 4;
  const int r0 = blockIdx.x * T1R, n0 = blockIdx.y * T1C;
  // a row past B or a hidden unit past d_1 reads row 0: it feeds only
  // outputs that are never stored
  const int xr = r0 + i16 < B ? r0 + i16 : 0;
  const float* xp = X + (size_t)xr * d0 + 4 * g16;
  const float* vp[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int n = n0 + 16 * s + i16;
    vp[s] = v + offW1 + (size_t)(n < d1 ? n : 0) * d0 + 4 * g16;
  }
  const int nblk = (d0 + 15) >> 4, nfull = d0 >> 4;
  const int b0 = wave * nblk / 4, b1 = (wave + 1) * nblk / 4;
  const int fe = b1 < nfull ? b1 : nfull;          // full blocks [b0, fe)
  f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  auto mma = [&](const f32x4& a, const f32x4& b0v, const f32x4& b1v) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[q], b0v[q], acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[q], b1v[q], acc[1], 0, 0, 0);
    }
  };
  // the full blocks [b0, fe), U1 of them in flight: slot u holds block
  // t0 + u and, once its MFMAs have read it, is reloaded with block
  // t0 + u + U1 (the last full block again past the end: in bounds,
  // unused).  No branch around the loads and no copy between registers
  // (either would make the compiler wait for loads in flight).
  if (fe > b0) {
    f32x4 xs[U1], ws[U1][2];
    auto load = [&](int b, int u) {
      const int bb = b < fe ? b : fe - 1;
      xs[u] = *(const f32x4*)(xp + 16 * bb);
      ws[u][0] = *(const f32x4*)(vp[0] + 16 * bb);
      ws[u][1] = *(const f32x4*)(vp[1] + 16 * bb);
    };
    // (issued in slot order, as in the loop: the compiler's wait for the
    // oldest slot then covers both ways into the loop)
#pragma unroll
    for (int u = 0; u < U1; ++u) {
      load(b0 + u, u);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int t0 = b0; t0 < fe; t0 += U1) {
#pragma unroll
      for (int u = 0; u < U1; ++u) {
        if (t0 + u < fe) mma(xs[u], ws[u][0], ws[u][1]);
        __builtin_amdgcn_sched_barrier(0);
        load(t0 + u + U1, u);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // the ragged last block (d_0 % 16 != 0), in this wave's range: float4s
  // past d_0 are zero
  if (nfull < nblk && nfull >= b0 && nfull < b1) {
    const int k = 16 * nfull + 4 * g16;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    const bool kv = k < d0;
    const f32x4 a = kv ? *(const f32x4*)(xp + 16 * nfull) : z;
    const f32x4 w0 = kv ? *(const f32x4*)(vp[0] + 16 * nfull) : z;
    const f32x4 w1 = kv ? *(const f32x4*)(vp[1] + 16 * nfull) : z;
    mma(a, w0, w1);
  }
  red[wave][0][lane] = acc[0];
  red[wave][1][lane] = acc[1];
  __syncthreads();
  // lane (i16, g16) of a subtile holds rows 4 g16 .. 4 g16 + 3 of column
  // i16; thread t adds the four waves' values of subtile t / 64 (fixed order)
  if (tid < 128) {
    const int s = tid >> 6, l = tid & 63;
    const int n = n0 + 16 * s + (l & 15);
    f32x4 t = red[0][s][l];
#pragma unroll
    for (int w = 1; w < 4; ++w) t += red[w][s][l];
    if (n < d1) {
      const float cb = v[offB1 + n];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = r0 + 4 * (l >> 4) + r;
        if (row < B) rz[(size_t)row * ldrz + n] = act >= 0 ? act_f(act, t[r] + cb) : t[r] + cb;
      }
    }
  }
}

// ------------------------------------------------------------------------
// The cache of a solve for a narrow net in two launches (Alg. 1 step 1 and
// the backward pass of Sec. 2.1): hf_narrow_layer1 with the activation
// forms A_1 = phi(X W_1^T + b_1) in tiles, then this kernel takes 4 batch
// rows per workgroup through the later layers, the softmax and, for the
// Hessian, the backward pass of delta and of E2 = (delta_l W_l) phi''.
// Arithmetic per element is that of the forward and backward epilogues and
// of the softmax row kernel; the contractions are those of
// hf_narrow_product4 with W in place of v.  With loss_part and no backward
// pass (hess = grad = 0, P null) it is the loss-only forward of the line
// search: only the per-row losses leave the workgroup.
extern "C" __global__ __launch_bounds__(512) void hf_narrow_forward4(NarrowFwdArgs g) {
  constexpr int ML = MAXL - 1;
  __shared__ __attribute__((aligned(16))) float sA[ML][R4][LR4];   // A_l
  __shared__ __attribute__((aligned(16))) float sD[2][R4][LR4];    // delta_l
  __shared__ __attribute__((aligned(16))) float sZ[R4][64];        // logits
  __shared__ __attribute__((aligned(16))) float red[NW][R4][64];   // partials
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int xi = lane & 3, xk = lane >> 2;   // A operand: row, k within 16
  const int r0 = blockIdx.x * R4;
  const int L = g.L;
  const int act = g.act;
  const bool hess = g.hess != 0, grad = g.grad != 0;
  const bool delta = hess || grad;       // the backward pass of delta runs
  const bool loss = g.loss_part != nullptr;
  const bool keep = g.P != nullptr;      // A_l and P are stored

  // Weight values of W_l for this lane (forward: [c][k]; backward: [k][c]),
  // blocks sl and sl + nks of 16 k; past the widths the loads read W_l's
  // first weight, unmasked (the A operands are zero there, and columns past
  // d_n are never stored)
  auto weights = [&](int l, bool fw, float (&bw)[2][16]) {
    const int dk = fw ? g.d[l - 1] : g.d[l], dn = fw ? g.d[l] : g.d[l - 1];
    const int ncg = (dn + 63) >> 6, nks = NW / ncg;
    const int c = 64 * (wave % ncg) + lane, sl = wave / ncg;
    const bool cv = c < dn;
    const float* w = g.W + g.offW[l];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const int k = 16 * (sl + h * nks) + a;
        const bool kv = cv && k < dk;
        bw[h][a] = w[kv ? (fw ? (size_t)c * dk + k : (size_t)k * dn + c) : 0];
      }
  };
  float fw2[2][16], bwL[2][16];
  weights(2, true, fw2);
  weights(L, false, bwL);

  // A_1 rows (zero past B and d_1), also into the concatenated columns;
  // the workgroup's rows of X into the concatenated columns
  {
    const int pr = tid / MAXH, pc = tid - pr * MAXH;   // NT = R4 * MAXH
    const bool prv = r0 + pr < g.B;
    const int prow = prv ? r0 + pr : 0;
    const bool ok = prv && pc < g.d[1];
    const float a = g.A[1][ok ? (size_t)prow * g.ld[1] + pc : 0];
    // X: at most R4 * NARROW_MAX_INPUT / 4 = 2 NT float4s
    const int d0 = g.d[0], q4 = d0 >> 2;
    f32x4 xv[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int e = tid + NT * h, r = e / (q4 ? q4 : 1), c = 4 * (e - r * q4);
      const bool xok = g.Ycat && e < R4 * q4 && r0 + r < g.B;
      xv[h] = *(const f32x4*)(g.X + (xok ? (size_t)(r0 + r) * d0 + c : 0));
    }
    sA[0][pr][pc] = ok ? a : 0.0f;
    if (g.Ycat && ok) g.Ycat[(size_t)prow * g.ldy + g.yoff[1] + pc] = a;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int e = tid + NT * h, r = e / (q4 ? q4 : 1), c = 4 * (e - r * q4);
      if (g.Ycat && e < R4 * q4 && r0 + r < g.B)
        *(f32x4*)(g.Ycat + (size_t)(r0 + r) * g.ldy + c) = xv[h];
    }
  }
  __syncthreads();

  auto total = [&](int ncg, int nks, int i, int c) {
    float s = 0.0f;
    for (int k = 0; k < nks; ++k) s += red[k * ncg + (c >> 6)][i][c & 63];
    return s;
  };

  // ---- layers 2 .. L: Z_l = A_{l-1} W_l^T + b_l; A_l = phi(Z_l) below L
  for (int l = 2; l <= L; ++l) {
    const int dk = g.d[l - 1], dn = g.d[l];
    const int ncg = (dn + 63) >> 6, nks = NW / ncg;
    const int sl = wave / ncg;
    const int nblk = (dk + 15) >> 4;
    float bw[2][16];
    if (l == 2) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int a = 0; a < 16; ++a) bw[h][a] = fw2[h][a];
    } else {
      weights(l, true, bw);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int b = sl + h * nks;
      if (b < nblk) acc = mfma4x16(sA[l - 2][xi][16 * b + xk], bw[h], acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    {
      const int i = tid >> 7, cc = tid & (MAXH - 1);
      const bool cv = cc < dn, rv = r0 + i < g.B;
      const float z = cv ? total(ncg, nks, i, cc) + g.W[g.offB[l] + cc] : 0.0f;
      if (l < L) {
        const float a = cv ? act_f(act, z) : 0.0f;
        sA[l - 1][i][cc] = a;
        if (cv && rv) {
          if (keep) g.A[l][(size_t)(r0 + i) * g.ld[l] + cc] = a;
          if (g.Ycat) g.Ycat[(size_t)(r0 + i) * g.ldy + g.yoff[l] + cc] = a;
        }
      } else if (cc < 64) {
        sZ[i][cc] = z;
      }
    }
    __syncthreads();
  }

  // ---- softmax of the logits, wave i < 4 on row i (columns lane < C <= 64);
  // with labels a label outside [0, C) flagged, delta_L = (p - e_y) / B, and
  // for the loss the row's log(sum exp z) - z_y
  __shared__ float wl[R4];
  if (wave < R4) {
    const int i = wave, C = g.d[L], row = r0 + i;
    const bool cv = lane < C, rv = row < g.B;
    const float z = cv ? sZ[i][lane] : -INFINITY;
    float m = z;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    const float e = cv ? expf(z - m) : 0.0f;
    const float sum = wave_sum(e);
    const float p = e * (1.0f / sum);
    if (keep && cv && rv) g.P[(size_t)row * g.ld[L] + lane] = p;
    if (delta || loss) {
      int yi = rv ? g.y[row] : -1;
      if (rv && (yi < 0 || yi >= C)) {
        if (lane == 0) *g.err = 1;
        yi = -1;
      }
      if (delta) {
        const float dl = cv ? (lane == yi ? p - 1.0f : p) * g.invB : 0.0f;
        sD[0][i][lane] = dl;
        if (cv && rv) {
          if (hess) g.D[L][(size_t)row * g.ld[L] + lane] = dl;
          if (g.Dcat) g.Dcat[(size_t)row * g.ldr + g.roff[L] + lane] = dl;
        }
      }
      if (loss && lane == 0) {
        const float zy = yi >= 0 ? sZ[i][yi] : 0.0f;
        wl[i] = yi >= 0 ? (m + logf(sum)) - zy : 0.0f;
      }
    }
  }
  __syncthreads();
  if (loss && tid == 0)
    g.loss_part[blockIdx.x] = ((double)wl[0] + (double)wl[1]) + ((double)wl[2] + (double)wl[3]);
  if (!delta) return;

  // ---- backward, l = L .. 2: t = delta_l W_l over K = d_l;
  // delta_{l-1} = t phi'(A_{l-1}); for the Hessian E2_{l-1} = t phi''(A_{l-1})
  // (delta_1 only for the gradient)
  int cur = 0;
  for (int l = L; l >= 2; --l) {
    const int dk = g.d[l], dn = g.d[l - 1];
    const int ncg = (dn + 63) >> 6, nks = NW / ncg;
    const int sl = wave / ncg;
    const int nblk = (dk + 15) >> 4;
    float bw[2][16];
    if (l == L) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int a = 0; a < 16; ++a) bw[h][a] = bwL[h][a];
    } else {
      weights(l, false, bw);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int b = sl + h * nks;
      if (b < nblk) acc = mfma4x16(sD[cur][xi][16 * b + xk], bw[h], acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    {
      const int i = tid >> 7, cc = tid & (MAXH - 1);
      const bool cv = cc < dn, rv = r0 + i < g.B;
      float dl = 0.0f;
      if (cv) {
        const float t = total(ncg, nks, i, cc), a = sA[l - 2][i][cc];
        dl = t * act_d1(act, a);
        if (rv) {
          const size_t o = (size_t)(r0 + i) * g.ld[l - 1] + cc;
          if (hess) {
            g.E2[l - 1][o] = t * act_d2(act, a);
            if (l > 2) g.D[l - 1][o] = dl;
          }
          if (g.Dcat && (grad || l > 2))
            g.Dcat[(size_t)(r0 + i) * g.ldr + g.roff[l - 1] + cc] = dl;
        }
      }
      sD[cur ^ 1][i][cc] = dl;
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
  // (a narrow net has far fewer than 2^31 parameters: 32-bit index
  // arithmetic)
  const size_t mn = (size_t)nc.M * nc.N;
  const int n = (int)nc.n;
  double pq = 0.0, pp = 0.0;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) {
    int l = 1;
    while (l < nc.L && i >= (int)nc.offW[l + 1]) ++l;
    double t = 0.0;
    if (i < (int)nc.offB[l]) {
      const int loc = i - (int)nc.offW[l];
      const int dk = nc.d[l - 1];
      const int m = loc / dk, k = loc - m * dk;
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
      const int m = i - (int)nc.offB[l];
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
  // The layer-1 tiles and the 4-row workgroups up to 64 workgroups of 16
  // rows, the 16-row form above: CG on G measured 10-15% faster on each
  // side of the switch (nets 784-100-10, 784-128-64 and 256-64-64-10 at
  // 500 to 8,000 rows; the forms meet between 1,000 and 1,500 rows).
  const bool four = (a.B + RW - 1) / RW <= 64;
  // algorithmic work: the GEMM flops of the replaced passes
  const double f1 = 2.0 * a.B * a.d[0] * a.d[1];
  double fr = 0.0;
  for (int l = 2; l <= a.L; ++l)
    fr += 2.0 * a.B * a.d[l - 1] * a.d[l] * (a.hess ? 4.0 : 3.0);
  if (four) {
    const dim3 g1((unsigned)((a.B + T1R - 1) / T1R), (unsigned)((a.d[1] + T1C - 1) / T1C));
    prof_begin(Lc, "hf_narrow_layer1");
    hipExtLaunchKernelGGL(hf_narrow_layer1, g1, dim3(NT1), 0, Lc.stream, prof_a(Lc),
                          prof_b(Lc), 0, a.X, a.v, a.B, a.d[0], a.d[1], a.offW[1], a.offB[1],
                          a.RZ1, a.ld[1], -1, a.skip);
    prof_end(Lc, "hf_narrow_layer1", f1, 4.0 * a.B * (a.d[0] + a.d[1]));
    prof_begin(Lc, "hf_narrow_product4");
    hipExtLaunchKernelGGL(hf_narrow_product4, dim3((unsigned)((a.B + R4 - 1) / R4)), dim3(NT),
                          0, Lc.stream, prof_a(Lc), prof_b(Lc), 0, a);
    prof_end(Lc, "hf_narrow_product4", fr, 4.0 * a.B * 5.0 * a.d[1]);
  } else {
    prof_begin(Lc, "hf_narrow_product");
    hipExtLaunchKernelGGL(hf_narrow_product, dim3((unsigned)((a.B + RW - 1) / RW)), dim3(NT), 0,
                          Lc.stream, prof_a(Lc), prof_b(Lc), 0, a);
    prof_end(Lc, "hf_narrow_product", f1 + fr, 4.0 * a.B * (a.d[0] + 4.0 * a.d[1]));
  }
}

void narrow_forward(const Launch& Lc, const NarrowFwdArgs& a) {
  const dim3 g1((unsigned)((a.B + T1R - 1) / T1R), (unsigned)((a.d[1] + T1C - 1) / T1C));
  prof_begin(Lc, "hf_narrow_layer1");
  hipExtLaunchKernelGGL(hf_narrow_layer1, g1, dim3(NT1), 0, Lc.stream, prof_a(Lc), prof_b(Lc),
                        0, a.X, a.W, a.B, a.d[0], a.d[1], a.offW[1], a.offB[1], a.A[1],
                        a.ld[1], a.act, nullptr);
  prof_end(Lc, "hf_narrow_layer1", 2.0 * a.B * a.d[0] * a.d[1], 4.0 * a.B * (a.d[0] + a.d[1]));
  double fl = 0.0;
  for (int l = 2; l <= a.L; ++l)
    fl += 2.0 * a.B * a.d[l - 1] * a.d[l] * (a.hess || a.grad ? 2.0 : 1.0);
  prof_begin(Lc, "hf_narrow_forward4");
  hipExtLaunchKernelGGL(hf_narrow_forward4, dim3((unsigned)((a.B + R4 - 1) / R4)), dim3(NT), 0,
                        Lc.stream, prof_a(Lc), prof_b(Lc), 0, a);
  prof_end(Lc, "hf_narrow_forward4", fl, 4.0 * a.B * (a.d[0] + 4.0 * a.d[1]));
}

}  // namespace hfk
