// bf16-input MFMA GEMMs: the same contractions as the fp32 kernels (the
// dense layers of the forward, backward, R-forward and R-backward passes of
// Sec. 2.1), with every operand rounded to bf16 and the products accumulated
// in fp32 by v_mfma_f32_32x32x16_bf16.  Epilogue arithmetic (bias, phi,
// phi', phi'', the R-operator combinations) stays in fp32.
//
// Every operand is K-contiguous: X(m, k) = X[m * ldx + k], Y(n, k) =
// Y[n * ldy + k].  The forward passes take W_l (d_l x d_{l-1}) as it is, the
// backward passes its transposed copy, and the weight gradient contracts
// over the batch using the transposed (batch-contiguous) copies of the
// activations and deltas that the producing epilogues write beside the
// row-major ones.  One LDS layout therefore serves every operand.
//
// One workgroup of 256 threads (4 wave64 in a 2 x 2 grid) owns a 128 x 128
// output tile; each wave owns a 64 x 64 quadrant as 2 x 2 blocks of 32 x 32.
// K advances in blocks of 32 through two LDS buffers; the next block's
// global loads are in flight while the MFMAs consume the current one.
// LDS tiles are [row][k] with 64 bytes per row; the four 16-byte chunks of a
// row are XOR-swizzled by (row >> 2) & 3, which keeps both the 128-bit
// stores and the 128-bit fragment loads free of bank conflicts.
// Lane (i, h) of an MFMA feeds the 8 consecutive k values 8h .. 8h + 7 of
// its row for both operands, so the sum over k is exact up to its order.
#include "act.h"
#include "hf_internal.h"

namespace hfk {
namespace {

constexpr int BK = 32;                  // k values per K block
constexpr int NT = 256;                 // threads per workgroup
constexpr int ROWS = 128;               // tile rows of each operand
constexpr int CH = BK / 8;              // 16-byte chunks per tile row
constexpr int CPT = ROWS * CH / NT;     // chunks per thread per tile
constexpr int TILE = ROWS * BK;         // bf16 elements per tile
constexpr int W = 2;                    // 2 x 2 MFMA blocks per wave

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int swz(int row) { return (row >> 2) & 3; }

__device__ __forceinline__ float bf2f(bf16_t h) {
  return __uint_as_float((uint32_t)h << 16);
}
// round to nearest even
__device__ __forceinline__ bf16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// ------------------------------------------------------------ tile loading
// The thread's CPT chunks of the ROWS x BK tile at (r0, k0) of an operand
// stored rows x K with leading dimension ld (a multiple of 8, rows 16-byte
// aligned).  Chunk i covers row (tid + NT i) / CH, k values 8 ((tid + NT i) %
// CH) .. + 7.
struct Tile {
  __device__ static __forceinline__ size_t offset(int ld, int tid) {
    return (size_t)(tid / CH) * ld + (tid % CH) * 8;
  }
  // tile fully inside the operand; p = operand + tile origin + offset()
  __device__ static __forceinline__ void load_fast(const bf16_t* __restrict__ p,
                                                   int ld, u32x4 (&g)[CPT]) {
    const size_t step = (size_t)(NT / CH) * ld;
#pragma unroll
    for (int i = 0; i < CPT; ++i) g[i] = *(const u32x4*)(p + i * step);
  }
  // guarded: elements outside rows x K read as zero
  __device__ static __forceinline__ void load(const bf16_t* __restrict__ base,
                                              int ld, int rows, int K, int r0,
                                              int k0, int tid, u32x4 (&g)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int idx = tid + NT * i;
      const int r = r0 + idx / CH, k = k0 + (idx % CH) * 8;
      const bf16_t* p = base + (size_t)r * ld + k;
      if (r < rows && k + 7 < K) {
        g[i] = *(const u32x4*)p;
      } else {
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        if (r < rows) {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (k + j < K) w[j >> 1] |= (uint32_t)p[j] << (16 * (j & 1));
        }
        g[i] = u32x4{w[0], w[1], w[2], w[3]};
      }
    }
  }
  __device__ static __forceinline__ void store(bf16_t* __restrict__ s, int tid,
                                               const u32x4 (&g)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int idx = tid + NT * i;
      const int row = idx / CH, c = idx % CH;
      *(u32x4*)(s + row * BK + ((c ^ swz(row)) * 8)) = g[i];
    }
  }
  // operand of MFMA step q (k = 16 q .. 16 q + 15) for lane (row, h)
  __device__ static __forceinline__ bf16x8 frag(const bf16_t* __restrict__ s,
                                                int row, int h, int q) {
    const int c = 2 * q + h;
    return *(const bf16x8*)(s + row * BK + ((c ^ swz(row)) * 8));
  }
};

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ----------------------------------------------------------------- epilogues
// Row-major bf16 outputs h* (leading dimension ldo), their transposed copies
// t* ([col][row], leading dimension ldt), fp32 outputs f* (ldf).  aux a0 is
// bf16 with ldo, a1 and a2 are fp32 with ldf.
__device__ __forceinline__ void put(const EpiH& e, bf16_t* h, bf16_t* t, int r,
                                    int c, float v) {
  const bf16_t b = f2bf(v);
  h[(size_t)r * e.ldo + c] = b;
  t[(size_t)c * e.ldt + r] = b;
}
__device__ __forceinline__ float aux0(const EpiH& e, int r, int c) {
  return bf2f(e.a0[(size_t)r * e.ldo + c]);
}

struct EFwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    const float z = v0 + e.bias[c];
    if (e.hidden) put(e, e.h0, e.t0, r, c, act_f(e.act, z));
    else e.f0[(size_t)r * e.ldf + c] = z;
  }
};
struct EFwdRFwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float v1) {
    const float z = v0 + e.bias[c];
    const float rz = v1 + e.rbias[c];
    e.f1[(size_t)r * e.ldf + c] = rz;
    if (e.hidden) {
      const float a = act_f(e.act, z);
      put(e, e.h0, e.t0, r, c, a);
      put(e, e.h2, e.t2, r, c, act_d1(e.act, a) * rz);
    } else {
      e.f0[(size_t)r * e.ldf + c] = z;
    }
  }
};
struct ERFwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    const float rz = v0 + e.rbias[c];
    e.f1[(size_t)r * e.ldf + c] = rz;
    if (e.hidden) put(e, e.h2, e.t2, r, c, act_d1(e.act, aux0(e, r, c)) * rz);
  }
};
struct EBwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    put(e, e.h0, e.t0, r, c, v0 * act_d1(e.act, aux0(e, r, c)));
  }
};
struct EBwdE2 {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    const float a = aux0(e, r, c);
    put(e, e.h0, e.t0, r, c, v0 * act_d1(e.act, a));
    e.f2[(size_t)r * e.ldf + c] = v0 * act_d2(e.act, a);
  }
};
struct EBwdRBwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float v1) {
    const float a = aux0(e, r, c);
    const float d1 = act_d1(e.act, a);
    put(e, e.h0, e.t0, r, c, v0 * d1);
    put(e, e.h1, e.t1, r, c,
        v1 * d1 + v0 * act_d2(e.act, a) * e.a1[(size_t)r * e.ldf + c]);
  }
};
struct ERBwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    const size_t o = (size_t)r * e.ldf + c;
    put(e, e.h1, e.t1, r, c, v0 * act_d1(e.act, aux0(e, r, c)) + e.a2[o] * e.a1[o]);
  }
};
struct EGNBwd {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    put(e, e.h1, e.t1, r, c, v0 * act_d1(e.act, aux0(e, r, c)));
  }
};
struct EStore {
  static __device__ __forceinline__ void apply(const EpiH& e, int r, int c,
                                               float v0, float) {
    e.f0[(size_t)blockIdx.z * e.split_stride + (size_t)r * e.ldf + c] = v0;
  }
};

// ------------------------------------------------------------------- body
// MODE 0: single (nseg K-segments, optional split-K over grid z)
// MODE 1: dual   acc0 = X0 Y0, acc1 = X1 Y0 + X0 Y1
// MODE 2: dual0  acc0 = X0 Y0, acc1 = X0 Y1
// BIAS (weight gradient): blocks of the first column tile also sum their X
// tiles of K-segment 0 over k, giving sum_k X(m, k) for their rows.
template <int MODE, class Epi, bool BIAS>
__device__ __forceinline__ void hgemm_body(const GemmShapeH& s, const EpiH& e) {
  if (s.skip && *s.skip) return;
  constexpr int T = MODE == 0 ? 2 : (MODE == 1 ? 4 : 3);
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][T][TILE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * ROWS;
  const int n0 = blockIdx.x * ROWS;

  const int kbps = (s.K + BK - 1) / BK;
  const int nvb = (MODE == 0 ? s.nseg : 1) * kbps;
  int vb0 = 0, vb1 = nvb;
  if (MODE == 0 && s.splits > 1) {
    const int per = (nvb + s.splits - 1) / s.splits;
    vb0 = blockIdx.z * per;
    vb1 = min(nvb, vb0 + per);
  }

  f32x16 acc0[W][W], acc1[W][W];
#pragma unroll
  for (int a = 0; a < W; ++a)
#pragma unroll
    for (int b = 0; b < W; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc0[a][b][r] = 0.0f;
        if (MODE != 0) acc1[a][b][r] = 0.0f;
      }

  u32x4 g[T][CPT];
  const bool in_x = m0 + ROWS <= s.M;
  const bool in_y = n0 + ROWS <= s.N;
  const size_t ox = Tile::offset(s.ldx, tid) + (size_t)m0 * s.ldx;
  const size_t oy = Tile::offset(s.ldy, tid) + (size_t)n0 * s.ldy;
  auto ldx = [&](const bf16_t* base, int k0, u32x4 (&r)[CPT]) {
    if (in_x && k0 + BK <= s.K) Tile::load_fast(base + ox + k0, s.ldx, r);
    else Tile::load(base, s.ldx, s.M, s.K, m0, k0, tid, r);
  };
  auto ldy = [&](const bf16_t* base, int k0, u32x4 (&r)[CPT]) {
    if (in_y && k0 + BK <= s.K) Tile::load_fast(base + oy + k0, s.ldy, r);
    else Tile::load(base, s.ldy, s.N, s.K, n0, k0, tid, r);
  };
  auto gload = [&](int vb) {
    const int seg = (MODE == 0) ? vb / kbps : 0;
    const int k0 = (vb - seg * kbps) * BK;
    if (MODE == 0) {
      ldx(s.X[seg], k0, g[0]);
      ldy(s.Y[seg], k0, g[1]);
    } else if (MODE == 1) {
      ldx(s.X[0], k0, g[0]);
      ldx(s.X[1], k0, g[1]);
      ldy(s.Y[0], k0, g[2]);
      ldy(s.Y[1], k0, g[3]);
    } else {
      ldx(s.X[0], k0, g[0]);
      ldy(s.Y[0], k0, g[1]);
      ldy(s.Y[1], k0, g[2]);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int t = 0; t < T; ++t) Tile::store(lds[buf][t], tid, g[t]);
  };
  const int xrow = wm * 32 * W + li;
  const int yrow = wn * 32 * W + li;
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < BK / 16; ++q) {
      bf16x8 x0[W], y0[W];
#pragma unroll
      for (int a = 0; a < W; ++a) x0[a] = Tile::frag(lds[buf][0], xrow + 32 * a, h, q);
      if (MODE == 0) {
#pragma unroll
        for (int b = 0; b < W; ++b) y0[b] = Tile::frag(lds[buf][1], yrow + 32 * b, h, q);
#pragma unroll
        for (int a = 0; a < W; ++a)
#pragma unroll
          for (int b = 0; b < W; ++b) acc0[a][b] = mfma(x0[a], y0[b], acc0[a][b]);
      } else if (MODE == 1) {
        bf16x8 x1[W], y1[W];
#pragma unroll
        for (int a = 0; a < W; ++a) x1[a] = Tile::frag(lds[buf][1], xrow + 32 * a, h, q);
#pragma unroll
        for (int b = 0; b < W; ++b) {
          y0[b] = Tile::frag(lds[buf][2], yrow + 32 * b, h, q);
          y1[b] = Tile::frag(lds[buf][3], yrow + 32 * b, h, q);
        }
#pragma unroll
        for (int a = 0; a < W; ++a)
#pragma unroll
          for (int b = 0; b < W; ++b) {
            acc0[a][b] = mfma(x0[a], y0[b], acc0[a][b]);
            acc1[a][b] = mfma(x1[a], y0[b], acc1[a][b]);
            acc1[a][b] = mfma(x0[a], y1[b], acc1[a][b]);
          }
      } else {
        bf16x8 y1[W];
#pragma unroll
        for (int b = 0; b < W; ++b) {
          y0[b] = Tile::frag(lds[buf][1], yrow + 32 * b, h, q);
          y1[b] = Tile::frag(lds[buf][2], yrow + 32 * b, h, q);
        }
#pragma unroll
        for (int a = 0; a < W; ++a)
#pragma unroll
          for (int b = 0; b < W; ++b) {
            acc0[a][b] = mfma(x0[a], y0[b], acc0[a][b]);
            acc1[a][b] = mfma(x0[a], y1[b], acc1[a][b]);
          }
      }
    }
  };

  // bias sums: thread t owns row t % ROWS of the X tile and the half
  // t / ROWS of its k values (two 16-byte chunks)
  static_assert(NT == 2 * ROWS && CH == 4, "bias sum layout");
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
        const int row = tid % ROWS, half = tid / ROWS;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
          const int c = 2 * half + cc;
          const u32x4 v = *(const u32x4*)(lds[buf][0] + row * BK + ((c ^ swz(row)) * 8));
          float part = 0.0f;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            part += __uint_as_float(v[j] << 16) + __uint_as_float(v[j] & 0xffff0000u);
          bsum += (double)part;
        }
      }
      if (more) sstore(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }
  }
  if (BIAS && do_bias) {
    __shared__ double bpart2[ROWS];
    if (tid >= ROWS) bpart2[tid - ROWS] = bsum;
    __syncthreads();
    if (tid < ROWS && m0 + tid < s.M) {
      const double t = bsum + bpart2[tid];
      if (s.splits > 1) e.bias_part[(size_t)blockIdx.z * s.M + m0 + tid] = t;
      else e.bias_out[m0 + tid] = (float)t;
    }
  }

  // 32 x 32 accumulator layout: lane (li, h), register r holds row
  // 8 (r / 4) + 4 h + r % 4, column li of the block.
#pragma unroll
  for (int a = 0; a < W; ++a)
#pragma unroll
    for (int b = 0; b < W; ++b) {
      const f32x16 v0 = acc0[a][b];
      const f32x16 v1 = MODE == 0 ? v0 : acc1[a][b];
      const int rbase = m0 + wm * 32 * W + a * 32 + 4 * h;
      const int col = n0 + wn * 32 * W + b * 32 + li;
      if (col < s.N) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = rbase + 8 * (r >> 2) + (r & 3);
          if (row < s.M) Epi::apply(e, row, col, v0[r], MODE == 0 ? 0.0f : v1[r]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
}

}  // namespace

#define HF_HGEMM_KERNEL(NAME, MODE, EPI, BIAS)                                 \
  extern "C" __global__ __launch_bounds__(256, 1) void NAME(GemmShapeH s,      \
                                                            EpiH e) {          \
    hgemm_body<MODE, EPI, BIAS>(s, e);                                         \
  }

HF_HGEMM_KERNEL(hf_hgemm_fwd, 0, EFwd, false)
HF_HGEMM_KERNEL(hf_hgemm_fwd_rfwd, 1, EFwdRFwd, false)
HF_HGEMM_KERNEL(hf_hgemm_fwd_rfwd0, 2, EFwdRFwd, false)
HF_HGEMM_KERNEL(hf_hgemm_rfwd, 0, ERFwd, false)
HF_HGEMM_KERNEL(hf_hgemm_bwd, 0, EBwd, false)
HF_HGEMM_KERNEL(hf_hgemm_bwd_e2, 0, EBwdE2, false)
HF_HGEMM_KERNEL(hf_hgemm_bwd_rbwd, 1, EBwdRBwd, false)
HF_HGEMM_KERNEL(hf_hgemm_rbwd, 0, ERBwd, false)
HF_HGEMM_KERNEL(hf_hgemm_gnbwd, 0, EGNBwd, false)
HF_HGEMM_KERNEL(hf_hgemm_wgrad, 0, EStore, true)

// out[r * ldo + c] = bf16(in[r * ldi + c]) and outT[c * ldt + r] = the same
// value, for r < R, c < C, through a padded 32 x 32 LDS tile so that the
// reads and both writes are coalesced.  Either output may be null.
extern "C" __global__ __launch_bounds__(256) void hf_cvt_bf16(
    const float* __restrict__ in, int R, int C, int ldi, bf16_t* __restrict__ out,
    int ldo, bf16_t* __restrict__ outT, int ldt, const int* __restrict__ skip) {
  if (skip && *skip) return;
  __shared__ bf16_t t[32][34];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = r0 + ty + 8 * j, c = c0 + tx;
    if (r < R && c < C) {
      const bf16_t b = f2bf(in[(size_t)r * ldi + c]);
      t[ty + 8 * j][tx] = b;
      if (out) out[(size_t)r * ldo + c] = b;
    }
  }
  if (!outT) return;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = c0 + ty + 8 * j, r = r0 + tx;
    if (r < R && c < C) outT[(size_t)c * ldt + r] = t[tx][ty + 8 * j];
  }
}

namespace {

typedef void (*HKernel)(GemmShapeH, EpiH);
inline int cdiv(int a, int b) { return (a + b - 1) / b; }

void launch(const Launch& L, const char* name, HKernel k, int mode,
            const GemmShapeH& s, const EpiH& e, double flops, double bytes) {
  dim3 grid(cdiv(s.N, ROWS), cdiv(s.M, ROWS),
            (mode == 0 && s.splits > 1) ? s.splits : 1);
  prof_begin(L, name);
  hipLaunchKernelGGL(k, grid, dim3(NT), 0, L.stream, s, e);
  prof_end(L, name, flops, bytes);
}

inline double mnk(const GemmShapeH& s) { return 2.0 * s.M * s.N * (double)s.K; }
// algorithmic bytes: bf16 operands read once, outputs of the given widths
inline double io(const GemmShapeH& s, int nx, int ny, double out_bytes) {
  return 2.0 * ((double)s.M * s.K * nx + (double)s.N * s.K * ny) +
         (double)s.M * s.N * out_bytes;
}

}  // namespace

void hgemm_fwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  launch(L, "hf_hgemm_fwd", hf_hgemm_fwd, 0, s, e, mnk(s) * s.nseg,
         io(s, s.nseg, s.nseg, 4.0));
}
void hgemm_fwd_rfwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  if (s.X[1])
    launch(L, "hf_hgemm_fwd_rfwd", hf_hgemm_fwd_rfwd, 1, s, e, 3 * mnk(s),
           io(s, 2, 2, e.hidden ? 12.0 : 8.0));
  else
    launch(L, "hf_hgemm_fwd_rfwd0", hf_hgemm_fwd_rfwd0, 2, s, e, 2 * mnk(s),
           io(s, 1, 2, e.hidden ? 12.0 : 8.0));
}
void hgemm_rfwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  launch(L, "hf_hgemm_rfwd", hf_hgemm_rfwd, 0, s, e, mnk(s) * s.nseg,
         io(s, s.nseg, s.nseg, e.hidden ? 10.0 : 4.0));
}
void hgemm_bwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  if (e.f2)
    launch(L, "hf_hgemm_bwd_e2", hf_hgemm_bwd_e2, 0, s, e, mnk(s) * s.nseg,
           io(s, s.nseg, s.nseg, 10.0));
  else
    launch(L, "hf_hgemm_bwd", hf_hgemm_bwd, 0, s, e, mnk(s) * s.nseg,
           io(s, s.nseg, s.nseg, 6.0));
}
void hgemm_bwd_rbwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  launch(L, "hf_hgemm_bwd_rbwd", hf_hgemm_bwd_rbwd, 1, s, e, 3 * mnk(s),
         io(s, 2, 2, 14.0));
}
void hgemm_rbwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  launch(L, "hf_hgemm_rbwd", hf_hgemm_rbwd, 0, s, e, mnk(s) * s.nseg,
         io(s, s.nseg, s.nseg, 14.0));
}
void hgemm_gnbwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  launch(L, "hf_hgemm_gnbwd", hf_hgemm_gnbwd, 0, s, e, mnk(s) * s.nseg,
         io(s, s.nseg, s.nseg, 6.0));
}
void hgemm_wgrad(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  launch(L, "hf_hgemm_wgrad", hf_hgemm_wgrad, 0, s, e, mnk(s) * s.nseg,
         io(s, s.nseg, s.nseg, 4.0 * (s.splits > 1 ? s.splits : 1)));
}
void cvt_bf16(const Launch& L, const float* in, int R, int C, int ldi,
              bf16_t* out, int ldo, bf16_t* outT, int ldt, const int* skip) {
  prof_begin(L, "hf_cvt_bf16");
  hipLaunchKernelGGL(hf_cvt_bf16, dim3(cdiv(C, 32), cdiv(R, 32)), dim3(256), 0,
                     L.stream, in, R, C, ldi, out, ldo, outT, ldt, skip);
  prof_end(L, "hf_cvt_bf16", 0.0,
           (double)R * C * (4.0 + (out ? 2.0 : 0.0) + (outT ? 2.0 : 0.0)));
}

}  // namespace hfk
