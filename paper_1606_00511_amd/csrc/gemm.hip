// fp32 MFMA GEMMs for the dense layers of the forward, backward, R-forward
// and R-backward passes (the contractions behind the gradient and the
// curvature products of Sec. 2.1; Alg. 2 evaluates them on each node's
// minibatch).
//
// One workgroup of 256 threads (4 wave64) owns a 128 x 128 output tile;
// each wave owns a 64 x 64 quadrant computed as 2 x 2 blocks of
// v_mfma_f32_32x32x2_f32.  K advances in blocks of 16 through two LDS
// buffers: while the MFMAs consume one buffer, the next K block is fetched
// from global memory into registers and then written to the other buffer.
//
// Operand tiles are copied to LDS without transposition: a K-contiguous
// operand is kept as [row][k] (row stride 20 floats) and read back with two
// 128-bit LDS loads per lane; a row-contiguous operand is kept as [k][row]
// (row stride 132 floats) and read with 32-bit LDS loads.  Within a K block
// each half-wave works on its own 8 consecutive k values, which permutes the
// order of the K sum identically for both operands.
#include "hf_internal.h"

namespace hfk {
namespace {

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 16;
constexpr int NT = 256;
constexpr int LDK = BK + 4;     // [row][k] tile row stride
constexpr int LDM = BM + 4;     // [k][row] tile row stride
constexpr int TILE = (BM * LDK > BK * LDM) ? BM * LDK : BK * LDM;

static_assert(BM == BN, "one loader serves both operands");

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float act_f(int act, float z) {
  if (act == ACT_SIGMOID) return 1.0f / (1.0f + expf(-z));
  if (act == ACT_TANH) return tanhf(z);
  return fmaxf(z, 0.0f);
}
// phi'(z) written in terms of a = phi(z)
__device__ __forceinline__ float act_d1(int act, float a) {
  if (act == ACT_SIGMOID) return a * (1.0f - a);
  if (act == ACT_TANH) return 1.0f - a * a;
  return a > 0.0f ? 1.0f : 0.0f;
}
// phi''(z) written in terms of a = phi(z)
__device__ __forceinline__ float act_d2(int act, float a) {
  if (act == ACT_SIGMOID) return a * (1.0f - a) * (1.0f - 2.0f * a);
  if (act == ACT_TANH) return -2.0f * a * (1.0f - a * a);
  return 0.0f;
}

// ------------------------------------------------------------ tile loading
// MK: the operand is stored rows x K with K contiguous; otherwise K x rows
// with rows contiguous.  Each thread moves 8 floats of a 128 x 16 tile.
template <bool MK, int VEC>
struct Tile {
  __device__ static __forceinline__ void load(const float* __restrict__ base,
                                              int ld, int rows, int K, int r0,
                                              int k0, int tid, float (&g)[8]) {
    if (VEC == 4) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int idx = tid + NT * i;
        int r, k;
        if (MK) { r = r0 + (idx >> 2); k = k0 + (idx & 3) * 4; }
        else    { k = k0 + (idx >> 5); r = r0 + (idx & 31) * 4; }
        const bool full = MK ? (r < rows && k + 3 < K) : (k < K && r + 3 < rows);
        if (full) {
          const f32x4 v = MK ? *(const f32x4*)(base + (size_t)r * ld + k)
                             : *(const f32x4*)(base + (size_t)k * ld + r);
          g[4 * i + 0] = v[0]; g[4 * i + 1] = v[1];
          g[4 * i + 2] = v[2]; g[4 * i + 3] = v[3];
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int rr = MK ? r : r + j;
            const int kk = MK ? k + j : k;
            g[4 * i + j] = (rr < rows && kk < K)
                ? (MK ? base[(size_t)rr * ld + kk] : base[(size_t)kk * ld + rr])
                : 0.0f;
          }
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int idx = tid + NT * i;
        int r, k;
        if (MK) { r = r0 + (idx >> 4); k = k0 + (idx & 15); }
        else    { k = k0 + (idx >> 7); r = r0 + (idx & 127); }
        g[i] = (r < rows && k < K)
            ? (MK ? base[(size_t)r * ld + k] : base[(size_t)k * ld + r])
            : 0.0f;
      }
    }
  }

  __device__ static __forceinline__ void store(float* __restrict__ s, int tid,
                                               const float (&g)[8]) {
    if (VEC == 4) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int idx = tid + NT * i;
        float* d = MK ? s + (idx >> 2) * LDK + (idx & 3) * 4
                      : s + (idx >> 5) * LDM + (idx & 31) * 4;
        f32x4 v = {g[4 * i], g[4 * i + 1], g[4 * i + 2], g[4 * i + 3]};
        *(f32x4*)d = v;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int idx = tid + NT * i;
        if (MK) s[(idx >> 4) * LDK + (idx & 15)] = g[i];
        else    s[(idx >> 7) * LDM + (idx & 127)] = g[i];
      }
    }
  }

  // The 8 values lane (row, half h) feeds to MFMA steps 0..7 of a K block.
  __device__ static __forceinline__ void frag(const float* __restrict__ s,
                                              int row, int h, float (&f)[8]) {
    if (MK) {
      const f32x4 a = *(const f32x4*)(s + row * LDK + h * 8);
      const f32x4 b = *(const f32x4*)(s + row * LDK + h * 8 + 4);
      f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
      f[4] = b[0]; f[5] = b[1]; f[6] = b[2]; f[7] = b[3];
    } else {
#pragma unroll
      for (int s8 = 0; s8 < 8; ++s8) f[s8] = s[(h * 8 + s8) * LDM + row];
    }
  }
};

__device__ __forceinline__ f32x16 mfma(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// ----------------------------------------------------------------- epilogues
struct EFwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    const float z = v0 + e.bias[c];
    e.out0[(size_t)r * e.ldo + c] = e.hidden ? act_f(e.act, z) : z;
  }
};
struct EFwdRFwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float v1) {
    const size_t o = (size_t)r * e.ldo + c;
    const float z = v0 + e.bias[c];
    const float rz = v1 + e.rbias[c];
    if (e.hidden) {
      const float a = act_f(e.act, z);
      e.out0[o] = a;
      e.out1[o] = rz;
      e.out2[o] = act_d1(e.act, a) * rz;
    } else {
      e.out0[o] = z;
      e.out1[o] = rz;
    }
  }
};
struct ERFwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    const size_t o = (size_t)r * e.ldo + c;
    const float rz = v0 + e.rbias[c];
    e.out1[o] = rz;
    if (e.hidden) e.out2[o] = act_d1(e.act, e.aux0[(size_t)r * e.lda + c]) * rz;
  }
};
struct EBwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    const size_t o = (size_t)r * e.ldo + c;
    const float a = e.aux0[(size_t)r * e.lda + c];
    e.out0[o] = v0 * act_d1(e.act, a);
    if (e.out2) e.out2[o] = v0 * act_d2(e.act, a);
  }
};
struct EBwdRBwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float v1) {
    const size_t o = (size_t)r * e.ldo + c;
    const size_t ia = (size_t)r * e.lda + c;
    const float a = e.aux0[ia];
    const float d1 = act_d1(e.act, a);
    e.out0[o] = v0 * d1;
    e.out1[o] = v1 * d1 + v0 * act_d2(e.act, a) * e.aux1[ia];
  }
};
struct ERBwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    const size_t ia = (size_t)r * e.lda + c;
    e.out1[(size_t)r * e.ldo + c] =
        v0 * act_d1(e.act, e.aux0[ia]) + e.aux2[ia] * e.aux1[ia];
  }
};
struct EGNBwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    e.out1[(size_t)r * e.ldo + c] =
        v0 * act_d1(e.act, e.aux0[(size_t)r * e.lda + c]);
  }
};
struct EStore {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    e.out0[(size_t)blockIdx.z * e.split_stride + (size_t)r * e.ldo + c] = v0;
  }
};

// ------------------------------------------------------------------- body
// MODE 0: single (nseg K-segments, optional split-K over grid z)
// MODE 1: dual   acc0 = X0 Y0, acc1 = X1 Y0 + X0 Y1
// MODE 2: dual0  acc0 = X0 Y0, acc1 = X0 Y1
// BIAS (weight gradient): blocks of the first column tile also sum their X
// tiles of K-segment 0 over k, giving sum_k X(m, k) for their 128 rows.
template <int MODE, bool XK, bool YK, int VEC, class Epi, bool BIAS = false>
__device__ __forceinline__ void gemm_body(const GemmShape& s, const EpiArgs& e) {
  if (s.skip && *s.skip) return;
  constexpr int T = MODE == 0 ? 2 : (MODE == 1 ? 4 : 3);
  __shared__ __attribute__((aligned(16))) float lds[2][T][TILE];

  using TX = Tile<XK, VEC>;
  using TY = Tile<YK, VEC>;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;

  const int kbps = (s.K + BK - 1) / BK;
  const int nvb = (MODE == 0 ? s.nseg : 1) * kbps;
  int vb0 = 0, vb1 = nvb;
  if (MODE == 0 && s.splits > 1) {
    const int per = (nvb + s.splits - 1) / s.splits;
    vb0 = blockIdx.z * per;
    vb1 = min(nvb, vb0 + per);
  }

  f32x16 acc0[2][2], acc1[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) { acc0[a][b][r] = 0.0f; acc1[a][b][r] = 0.0f; }

  float g[T][8];
  auto gload = [&](int vb) {
    const int seg = (MODE == 0) ? vb / kbps : 0;
    const int k0 = (vb - seg * kbps) * BK;
    if (MODE == 0) {
      TX::load(s.X[seg], s.ldx, s.M, s.K, m0, k0, tid, g[0]);
      TY::load(s.Y[seg], s.ldy, s.N, s.K, n0, k0, tid, g[1]);
    } else if (MODE == 1) {
      TX::load(s.X[0], s.ldx, s.M, s.K, m0, k0, tid, g[0]);
      TX::load(s.X[1], s.ldx, s.M, s.K, m0, k0, tid, g[1]);
      TY::load(s.Y[0], s.ldy, s.N, s.K, n0, k0, tid, g[2]);
      TY::load(s.Y[1], s.ldy, s.N, s.K, n0, k0, tid, g[3]);
    } else {
      TX::load(s.X[0], s.ldx, s.M, s.K, m0, k0, tid, g[0]);
      TY::load(s.Y[0], s.ldy, s.N, s.K, n0, k0, tid, g[1]);
      TY::load(s.Y[1], s.ldy, s.N, s.K, n0, k0, tid, g[2]);
    }
  };
  auto sstore = [&](int buf) {
    if (MODE == 0) {
      TX::store(lds[buf][0], tid, g[0]);
      TY::store(lds[buf][1], tid, g[1]);
    } else if (MODE == 1) {
      TX::store(lds[buf][0], tid, g[0]);
      TX::store(lds[buf][1], tid, g[1]);
      TY::store(lds[buf][2], tid, g[2]);
      TY::store(lds[buf][3], tid, g[3]);
    } else {
      TX::store(lds[buf][0], tid, g[0]);
      TY::store(lds[buf][1], tid, g[1]);
      TY::store(lds[buf][2], tid, g[2]);
    }
  };
  auto compute = [&](int buf) {
    float x0[2][8], y0[2][8];
    if (MODE == 0) {
#pragma unroll
      for (int a = 0; a < 2; ++a) TX::frag(lds[buf][0], wm * 64 + a * 32 + li, h, x0[a]);
#pragma unroll
      for (int b = 0; b < 2; ++b) TY::frag(lds[buf][1], wn * 64 + b * 32 + li, h, y0[b]);
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b) acc0[a][b] = mfma(x0[a][k], y0[b][k], acc0[a][b]);
    } else if (MODE == 1) {
      float x1[2][8], y1[2][8];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        TX::frag(lds[buf][0], wm * 64 + a * 32 + li, h, x0[a]);
        TX::frag(lds[buf][1], wm * 64 + a * 32 + li, h, x1[a]);
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        TY::frag(lds[buf][2], wn * 64 + b * 32 + li, h, y0[b]);
        TY::frag(lds[buf][3], wn * 64 + b * 32 + li, h, y1[b]);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            acc0[a][b] = mfma(x0[a][k], y0[b][k], acc0[a][b]);
            acc1[a][b] = mfma(x1[a][k], y0[b][k], acc1[a][b]);
            acc1[a][b] = mfma(x0[a][k], y1[b][k], acc1[a][b]);
          }
    } else {
      float y1[2][8];
#pragma unroll
      for (int a = 0; a < 2; ++a) TX::frag(lds[buf][0], wm * 64 + a * 32 + li, h, x0[a]);
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        TY::frag(lds[buf][1], wn * 64 + b * 32 + li, h, y0[b]);
        TY::frag(lds[buf][2], wn * 64 + b * 32 + li, h, y1[b]);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            acc0[a][b] = mfma(x0[a][k], y0[b][k], acc0[a][b]);
            acc1[a][b] = mfma(x0[a][k], y1[b][k], acc1[a][b]);
          }
    }
  };

  const bool do_bias = BIAS && blockIdx.x == 0 && (e.bias_out || e.bias_part);
  double bsum = 0.0;
  if (vb0 < vb1) {
    gload(vb0);
    sstore(0);
    __syncthreads();
    int buf = 0;
    for (int vb = vb0; vb < vb1; ++vb) {
      const bool more = vb + 1 < vb1;
      if (more) gload(vb + 1);
      compute(buf);
      if (BIAS && do_bias && vb < kbps) {
        // X tile is [k][m] (XK = false): this thread sums 8 k for column m
        const float* xs = lds[buf][0] + (tid >> 7) * 8 * LDM + (tid & 127);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) bsum += (double)xs[kk * LDM];
      }
      if (more) sstore(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }
  }
  if (BIAS && do_bias) {
    __shared__ double bhalf[128];
    if (tid >= 128) bhalf[tid - 128] = bsum;
    __syncthreads();
    if (tid < 128 && m0 + tid < s.M) {
      const double t = bsum + bhalf[tid];
      if (s.splits > 1) e.bias_part[(size_t)blockIdx.z * s.M + m0 + tid] = t;
      else e.bias_out[m0 + tid] = (float)t;
    }
  }

  // 32x32 f32 accumulator layout: lane (li, h), register r holds
  // row 8 * (r / 4) + 4 * h + r % 4, column li of the 32 x 32 block.
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        const int col = n0 + wn * 64 + b * 32 + li;
        if (row < s.M && col < s.N)
          Epi::apply(e, row, col, acc0[a][b][r], MODE == 0 ? 0.0f : acc1[a][b][r]);
      }
}

}  // namespace

#define HF_GEMM_KERNEL(NAME, MODE, XK, YK, EPI, BIAS)                           \
  extern "C" __global__ __launch_bounds__(256, 1) void NAME##_v4(GemmShape s,   \
                                                                 EpiArgs e) {   \
    gemm_body<MODE, XK, YK, 4, EPI, BIAS>(s, e);                                \
  }                                                                             \
  extern "C" __global__ __launch_bounds__(256, 1) void NAME##_v1(GemmShape s,   \
                                                                 EpiArgs e) {   \
    gemm_body<MODE, XK, YK, 1, EPI, BIAS>(s, e);                                \
  }

HF_GEMM_KERNEL(hf_gemm_fwd, 0, true, true, EFwd, false)
HF_GEMM_KERNEL(hf_gemm_fwd_rfwd, 1, true, true, EFwdRFwd, false)
HF_GEMM_KERNEL(hf_gemm_fwd_rfwd0, 2, true, true, EFwdRFwd, false)
HF_GEMM_KERNEL(hf_gemm_rfwd, 0, true, true, ERFwd, false)
HF_GEMM_KERNEL(hf_gemm_bwd, 0, true, false, EBwd, false)
HF_GEMM_KERNEL(hf_gemm_bwd_rbwd, 1, true, false, EBwdRBwd, false)
HF_GEMM_KERNEL(hf_gemm_rbwd, 0, true, false, ERBwd, false)
HF_GEMM_KERNEL(hf_gemm_gnbwd, 0, true, false, EGNBwd, false)
HF_GEMM_KERNEL(hf_gemm_wgrad, 0, false, false, EStore, true)

namespace {

typedef void (*GemmKernel)(GemmShape, EpiArgs);

inline bool a16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int pick_vec(const GemmShape& s, int mode) {
  if ((s.ldx & 3) || (s.ldy & 3)) return 1;
  const int nx = (mode == 0) ? s.nseg : (mode == 1 ? 2 : 1);
  const int ny = (mode == 0) ? s.nseg : 2;
  for (int i = 0; i < nx; ++i) if (!a16(s.X[i])) return 1;
  for (int i = 0; i < ny; ++i) if (!a16(s.Y[i])) return 1;
  return 4;
}

void launch(const Launch& L, const char* name, GemmKernel k4, GemmKernel k1,
            int mode, const GemmShape& s, const EpiArgs& e, double flops,
            double bytes) {
  const int vec = pick_vec(s, mode);
  dim3 grid((s.N + BN - 1) / BN, (s.M + BM - 1) / BM,
            (mode == 0 && s.splits > 1) ? s.splits : 1);
  prof_begin(L, name);
  hipLaunchKernelGGL(vec == 4 ? k4 : k1, grid, dim3(NT), 0, L.stream, s, e);
  prof_end(L, name, flops, bytes);
}

inline double mnk(const GemmShape& s) { return 2.0 * s.M * s.N * (double)s.K; }
inline double io(const GemmShape& s, int nx, int ny, int nout) {
  return 4.0 * ((double)s.M * s.K * nx + (double)s.N * s.K * ny +
                (double)s.M * s.N * nout);
}

}  // namespace

void gemm_fwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_fwd", hf_gemm_fwd_v4, hf_gemm_fwd_v1, 0, s, e,
         mnk(s) * s.nseg, io(s, s.nseg, s.nseg, 1));
}
void gemm_fwd_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  if (s.X[1]) {
    launch(L, "hf_gemm_fwd_rfwd", hf_gemm_fwd_rfwd_v4, hf_gemm_fwd_rfwd_v1, 1,
           s, e, 3 * mnk(s), io(s, 2, 2, e.hidden ? 3 : 2));
  } else {
    launch(L, "hf_gemm_fwd_rfwd0", hf_gemm_fwd_rfwd0_v4, hf_gemm_fwd_rfwd0_v1,
           2, s, e, 2 * mnk(s), io(s, 1, 2, e.hidden ? 3 : 2));
  }
}
void gemm_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_rfwd", hf_gemm_rfwd_v4, hf_gemm_rfwd_v1, 0, s, e,
         mnk(s) * s.nseg, io(s, s.nseg, s.nseg, e.hidden ? 3 : 1));
}
void gemm_bwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_bwd", hf_gemm_bwd_v4, hf_gemm_bwd_v1, 0, s, e,
         mnk(s) * s.nseg, io(s, s.nseg, s.nseg, e.out2 ? 3 : 2));
}
void gemm_bwd_rbwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_bwd_rbwd", hf_gemm_bwd_rbwd_v4, hf_gemm_bwd_rbwd_v1, 1, s,
         e, 3 * mnk(s), io(s, 2, 2, 4));
}
void gemm_rbwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_rbwd", hf_gemm_rbwd_v4, hf_gemm_rbwd_v1, 0, s, e,
         mnk(s) * s.nseg, io(s, s.nseg, s.nseg, 4));
}
void gemm_gnbwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_gnbwd", hf_gemm_gnbwd_v4, hf_gemm_gnbwd_v1, 0, s, e,
         mnk(s) * s.nseg, io(s, s.nseg, s.nseg, 2));
}
void gemm_wgrad(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_wgrad", hf_gemm_wgrad_v4, hf_gemm_wgrad_v1, 0, s, e,
         mnk(s) * s.nseg, io(s, s.nseg, s.nseg, s.splits > 1 ? s.splits : 1));
}

}  // namespace hfk
