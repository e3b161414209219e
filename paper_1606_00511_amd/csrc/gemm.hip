// fp32 MFMA GEMMs for the dense layers of the forward, backward, R-forward
// and R-backward passes (the contractions behind the gradient and the
// curvature products of Sec. 2.1; Alg. 2 evaluates them on each node's
// minibatch).
//
// One workgroup of 256 threads (4 wave64 in a 2 x 2 grid) owns a 128 x 128
// output tile; each wave owns a 64 x 64 quadrant computed either as 2 x 2
// blocks of v_mfma_f32_32x32x2_f32 or as 4 x 4 blocks of
// v_mfma_f32_16x16x4_f32 (fp32 operands, fp32 accumulation).  The 16 x 16
// form runs 16 independent accumulation chains per wave instead of 4 (on
// MI355X, chains of dependent 32 x 32 fp32 MFMAs sustain about 90% of the
// issue rate with 4 accumulators and 98% with 8 or more); the 32 x 32 form
// writes 32-column row segments in the epilogue instead of 16.  Each kernel
// takes the form that measured faster for it.  (Measured on MI355X:
// 256 x 256 tiles with 4 x 4 blocks per wave ran 5-15% slower than this
// shape at one wave per SIMD.)
//
// K advances in blocks of 16 through two LDS stages filled by direct
// global-to-LDS loads (16 bytes per lane, no registers in between): after
// the barrier of a block, the next block's loads are issued into the other
// stage and land while this block's MFMAs run; each wave waits only for its
// own loads, then the workgroup meets at one barrier per block.  (Measured
// on MI355X: three stages, two blocks ahead, ran 2% slower at the same
// occupancy.)  Rows past an operand's edge are clamped to its last row (they feed
// only outputs that are never stored); the ragged last K block of a
// K-segment is loaded through registers with zeros past K.  Operands that
// are not 16-byte aligned or whose leading dimension is not a multiple of 4,
// and the squared-operand kernels, stage their loads through registers and
// two LDS buffers instead (element-wise guarded loads at the edges).
//
// LDS layouts (the gfx950 LDS has 64 four-byte banks):
//  - a row-contiguous operand is kept as [k][row], 128 floats per k row,
//    with the 16-byte row chunks XOR-swizzled by ((k >> 2) & 3) << 2 and
//    read with 32-bit LDS loads: the k rows read at once by the four
//    quarter-waves (16 x 16 form) or the two half-waves (32 x 32 form) fall
//    in distinct banks, and one direct load fills two whole k rows;
//  - a K-contiguous operand is kept as [row][k] with its four 16-byte k
//    chunks XOR-swizzled by (row >> 2) & 3: no bank conflicts on the 128-bit
//    stores and loads.
// A direct load writes lane i's 16 bytes at 16 i past the wave's LDS base,
// so both swizzles are applied by choosing which global chunk each lane
// fetches.
// Every single-product GEMM pairs a K-contiguous left operand with a
// row-contiguous right one (the forward passes take transposed weights),
// the pairing that measured fastest on MI355X.
// Within a K block each half-wave (32 x 32 form) or quarter-wave (16 x 16
// form) works on its own consecutive k values, which permutes the order of
// the K sum identically for both operands.
#include <type_traits>

#include "act.h"
#include "hf_internal.h"
#include "lds_dma.h"

namespace hfk {
namespace {

constexpr int BK = 16;
constexpr int HK = BK / 2;      // k values per half-wave per K block
constexpr int NT = 256;
constexpr int LDK = BK;         // [row][k] tile row stride (swizzled chunks)
__device__ __forceinline__ int swz(int row) { return (row >> 2) & 3; }

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------ tile loading
// A ROWS x BK operand tile.  MK: the operand is stored rows x K with K
// contiguous, kept in LDS as swizzled [row][k] (stride LDK); otherwise
// K x rows with rows contiguous, kept as swizzled [k][row] (stride LDM).
// Register-staged loads move V1 floats per thread and tile.
template <bool MK, int VEC, int ROWS>
struct Tile {
  static constexpr int LDM = ROWS;
  static constexpr int SIZE = (ROWS * LDK > BK * LDM) ? ROWS * LDK : BK * LDM;
  static constexpr int V4 = ROWS * BK / 4 / NT;
  static constexpr int V1 = ROWS * BK / NT;
  // 16-byte direct loads per wave that fill the tile (4 waves, 1 KB each)
  static constexpr int INSTR = ROWS * BK / 1024;

  // [k][row] element (kk, row): row chunk row / 4 sits at chunk position
  // (row / 4) ^ (((kk >> 2) & 3) << 2) of k row kk, which moves the 16-row
  // runs that lanes read from k rows 4 apart (or 8 apart) into distinct
  // groups of 16 (or 32) banks.
  __device__ static __forceinline__ int kr(int kk, int row) {
    return kk * LDM + (row ^ (((kk >> 2) & 3) << 4));
  }

  // Element offset, from the operand's K block 0, of the 16-byte chunk that
  // lane `lane` of wave `wave` loads with its direct load j (chunk position
  // P = 64 (wave INSTR + j) + lane of the tile).  Rows past the operand's
  // edge are clamped to its last row: they feed only outputs that are never
  // stored.
  __device__ static __forceinline__ size_t dma_src(int ld, int rows, int r0,
                                                   int wave, int lane, int j) {
    const int P = (wave * INSTR + j) * 64 + lane;
    if (MK) {
      const int row = P / (BK / 4), pos = P % (BK / 4);
      const int r = min(r0 + row, rows - 1);
      return (size_t)r * ld + 4 * (pos ^ swz(row));
    } else {
      const int kk = P / (ROWS / 4), pos = P % (ROWS / 4);
      const int c = pos ^ (((kk >> 2) & 3) << 2);
      const int r = min(r0 + 4 * c, (rows - 1) & ~3);
      return (size_t)kk * ld + r;
    }
  }

  // Guarded load of the tile at (r0, k0); elements outside are zero.
  __device__ static __forceinline__ void load(const float* __restrict__ base,
                                              int ld, int rows, int K, int r0,
                                              int k0, int tid, float (&g)[V1]) {
    if (VEC == 4) {
#pragma unroll
      for (int i = 0; i < V4; ++i) {
        const int idx = tid + NT * i;
        int r, k;
        if (MK) { r = r0 + idx / (BK / 4); k = k0 + (idx % (BK / 4)) * 4; }
        else    { k = k0 + idx / (ROWS / 4); r = r0 + (idx % (ROWS / 4)) * 4; }
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
      for (int i = 0; i < V1; ++i) {
        const int idx = tid + NT * i;
        int r, k;
        if (MK) { r = r0 + idx / BK; k = k0 + idx % BK; }
        else    { k = k0 + idx / ROWS; r = r0 + idx % ROWS; }
        g[i] = (r < rows && k < K)
            ? (MK ? base[(size_t)r * ld + k] : base[(size_t)k * ld + r])
            : 0.0f;
      }
    }
  }

  // Offset of the thread's first element from the tile origin.
  __device__ static __forceinline__ size_t offset(int ld, int tid) {
    if (VEC == 4)
      return MK ? (size_t)(tid / (BK / 4)) * ld + (tid % (BK / 4)) * 4
                : (size_t)(tid / (ROWS / 4)) * ld + (tid % (ROWS / 4)) * 4;
    return MK ? (size_t)(tid / BK) * ld + tid % BK
              : (size_t)(tid / ROWS) * ld + tid % ROWS;
  }

  // Unguarded load of a tile that lies fully inside the operand; p points at
  // the thread's first element (operand + tile origin + offset()).
  __device__ static __forceinline__ void load_fast(const float* __restrict__ p,
                                                   int ld, float (&g)[V1]) {
    if (VEC == 4) {
      const size_t step = MK ? (size_t)(NT / (BK / 4)) * ld
                             : (size_t)(NT / (ROWS / 4)) * ld;
#pragma unroll
      for (int i = 0; i < V4; ++i) {
        const f32x4 v = *(const f32x4*)(p + i * step);
        g[4 * i + 0] = v[0]; g[4 * i + 1] = v[1];
        g[4 * i + 2] = v[2]; g[4 * i + 3] = v[3];
      }
    } else {
      const size_t step = MK ? (size_t)(NT / BK) * ld : (size_t)(NT / ROWS) * ld;
#pragma unroll
      for (int i = 0; i < V1; ++i) g[i] = p[i * step];
    }
  }

  __device__ static __forceinline__ void store(float* __restrict__ s, int tid,
                                               const float (&g)[V1]) {
    if (VEC == 4) {
#pragma unroll
      for (int i = 0; i < V4; ++i) {
        const int idx = tid + NT * i;
        float* d;
        if (MK) {
          const int row = idx / (BK / 4), c = idx % (BK / 4);
          d = s + row * LDK + ((c ^ swz(row)) * 4);
        } else {
          d = s + kr(idx / (ROWS / 4), (idx % (ROWS / 4)) * 4);
        }
        f32x4 v = {g[4 * i], g[4 * i + 1], g[4 * i + 2], g[4 * i + 3]};
        *(f32x4*)d = v;
      }
    } else {
#pragma unroll
      for (int i = 0; i < V1; ++i) {
        const int idx = tid + NT * i;
        if (MK) {
          const int row = idx / BK, k = idx % BK;
          s[row * LDK + (((k >> 2) ^ swz(row)) * 4) + (k & 3)] = g[i];
        } else {
          s[kr(idx / ROWS, idx % ROWS)] = g[i];
        }
      }
    }
  }

  // 16 x 16 x 4 operands: lane group g (lanes 16 g .. 16 g + 15) feeds
  // k = 4 g + step at MFMA step 0..3 of a K block, so a lane reads one
  // 16-byte chunk of a K-contiguous row (16 lanes, 16 rows, 16 distinct
  // bank groups under the swizzle) or, from a [k][row] tile, 16 consecutive
  // rows of k row 4 g + step.
  __device__ static __forceinline__ void frag16(const float* __restrict__ s,
                                                int row, int g, float (&f)[4]) {
    if (MK) {
      const f32x4 a = *(const f32x4*)(s + row * LDK + ((g ^ swz(row)) * 4));
      f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) f[q] = s[kr(4 * g + q, row)];
    }
  }

  // The HK values lane (row, half h) feeds to MFMA steps 0..HK-1 of a K
  // block: k = h * HK + step.  Both operands use the same k order, so the
  // sum over k is unchanged.
  __device__ static __forceinline__ void frag(const float* __restrict__ s,
                                              int row, int h, float (&f)[HK]) {
    if (MK) {
#pragma unroll
      for (int q = 0; q < HK / 4; ++q) {
        const int c = (h * HK) / 4 + q;
        const f32x4 a = *(const f32x4*)(s + row * LDK + ((c ^ swz(row)) * 4));
        f[4 * q + 0] = a[0]; f[4 * q + 1] = a[1];
        f[4 * q + 2] = a[2]; f[4 * q + 3] = a[3];
      }
    } else {
#pragma unroll
      for (int q = 0; q < HK; ++q) f[q] = s[kr(h * HK + q, row)];
    }
  }
};

__device__ __forceinline__ f32x4 mfma16(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
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
    if (e.out1) e.out1[o] = rz;      // null: RZ not needed downstream
    if (e.hidden) e.out2[o] = act_d1(e.act, e.aux0[(size_t)r * e.lda + c]) * rz;
  }
};
struct EBwd {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    e.out0[(size_t)r * e.ldo + c] =
        v0 * act_d1(e.act, e.aux0[(size_t)r * e.lda + c]);
  }
};
// backward data that also caches E * phi''(A) for the Hessian product
struct EBwdE2 {
  static __device__ __forceinline__ void apply(const EpiArgs& e, int r, int c,
                                               float v0, float) {
    const size_t o = (size_t)r * e.ldo + c;
    const float a = e.aux0[(size_t)r * e.lda + c];
    e.out0[o] = v0 * act_d1(e.act, a);
    e.out2[o] = v0 * act_d2(e.act, a);
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
// tiles of K-segment 0 over k, giving sum_k X(m, k) for their rows.
// M16: 4 x 4 blocks of 16 x 16 x 4 MFMAs per wave instead of 2 x 2 blocks
// of 32 x 32 x 2.
// TS: output tile rows and columns, 128 or 64 (64: single-product M16
// kernels only; each wave then holds 2 x 2 blocks of 16 x 16).
// SQ: every operand element is squared on its way into LDS (so the product
// is sum_k X(m, k)^2 Y(n, k)^2, and the bias sums are sums of squares).
// The output tile (tn, tm) of this workgroup within its split.  Linear
// dispatch index L goes to XCD L % 8 (each XCD has its own L2).  When a
// split's grid is a multiple of 8 tiles, XCD x gets the x-th contiguous
// eighth of the logical order, which walks groups of 8 tile rows column by
// column: the workgroups resident on one XCD then share their row panels of
// X and column panels of Y in its L2, instead of every XCD fetching every
// panel.  Otherwise the order is the dispatch order.
__device__ __forceinline__ void tile_of(int& tn, int& tm) {
  const int gx = gridDim.x, gy = gridDim.y, T = gx * gy;
  if (T % 8) {
    tn = blockIdx.x;
    tm = blockIdx.y;
    return;
  }
  const int L = blockIdx.x + gx * blockIdx.y;
  const int Lg = (L % 8) * (T / 8) + L / 8;
  constexpr int G = 8;
  const int g = Lg / (G * gx);
  const int first = g * G;
  const int rows = min(G, gy - first);
  const int w = Lg - g * G * gx;
  tm = first + w % rows;
  tn = w / rows;
}

template <int MODE, bool XK, bool YK, int VEC, class Epi, bool BIAS, bool M16,
          bool SQ = false, int TS = 128>
__device__ __forceinline__ void gemm_body(const GemmShape& s, const EpiArgs& e) {
  if (s.skip && *s.skip) return;
  static_assert(TS == 128 || (TS == 64 && M16 && MODE == 0), "tile size");
  constexpr int ROWS = TS;
  constexpr int W = ROWS / 64;  // 32 x 32 blocks per wave and dimension
  constexpr int HALF = ROWS / 2;  // rows (and columns) of a wave's quadrant
  using TX = Tile<XK, VEC, ROWS>;
  using TY = Tile<YK, VEC, ROWS>;
  constexpr int T = MODE == 0 ? 2 : (MODE == 1 ? 4 : 3);
  constexpr int SZ = TX::SIZE > TY::SIZE ? TX::SIZE : TY::SIZE;
  constexpr int V1 = TX::V1;
  constexpr bool DMA = VEC == 4 && !SQ;
  // LDS stages: 64 x 64 tiles have short K chains (split K, small grids)
  // and a quarter of the LDS per stage, so they keep three blocks in flight
  constexpr int S = TS == 64 ? 4 : 2;
  __shared__ __attribute__((aligned(16))) float lds[S][T][SZ];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, h = lane >> 5;
  int tn, tm;
  tile_of(tn, tm);
  const int m0 = tm * ROWS;
  const int n0 = tn * ROWS;

  const int kbps = (s.K + BK - 1) / BK;
  const int nvb = (MODE == 0 ? s.nseg : 1) * kbps;
  int vb0 = 0, vb1 = nvb;
  if (MODE == 0 && s.splits > 1) {
    const int per = (nvb + s.splits - 1) / s.splits;
    vb0 = blockIdx.z * per;
    vb1 = min(nvb, vb0 + per);
  }

  // MFMA blocks per wave and dimension, and accumulator registers per block
  constexpr int NB = M16 ? HALF / 16 : W;
  constexpr int AR = M16 ? 4 : 16;
  using Acc = typename std::conditional<M16, f32x4, f32x16>::type;
  const int r16 = lane & 15, g16 = lane >> 4;   // 16 x 16 lane coordinates
  Acc acc0[NB][NB], acc1[NB][NB];
#pragma unroll
  for (int a = 0; a < NB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < AR; ++r) {
        acc0[a][b][r] = 0.0f;
        if (MODE != 0) acc1[a][b][r] = 0.0f;
      }

  float g[T][V1];
  // Whether this tile's rows lie inside each operand: full K blocks of such
  // an operand take unguarded loads, the rest (a ragged last K block, or an
  // operand whose tile runs past its edge) take guarded ones.
  const bool in_x = m0 + ROWS <= s.M;
  const bool in_y = n0 + ROWS <= s.N;
  const size_t ox = TX::offset(s.ldx, tid) + (XK ? (size_t)m0 * s.ldx : (size_t)m0);
  const size_t oy = TY::offset(s.ldy, tid) + (YK ? (size_t)n0 * s.ldy : (size_t)n0);
  auto ldx = [&](const float* base, int k0, float (&r)[V1]) {
    if (in_x && k0 + BK <= s.K)
      TX::load_fast(base + ox + (XK ? (size_t)k0 : (size_t)k0 * s.ldx), s.ldx, r);
    else
      TX::load(base, s.ldx, s.M, s.K, m0, k0, tid, r);
  };
  auto ldy = [&](const float* base, int k0, float (&r)[V1]) {
    if (in_y && k0 + BK <= s.K)
      TY::load_fast(base + oy + (YK ? (size_t)k0 : (size_t)k0 * s.ldy), s.ldy, r);
    else
      TY::load(base, s.ldy, s.N, s.K, n0, k0, tid, r);
  };
  // Operand pointers are read once: indexing the kernel-argument arrays
  // with the loop's segment number would reload them with scalar loads on
  // every K block, and waiting for those also waits for every LDS access
  // in flight (one counter covers both).
  const float* const X0 = s.X[0];
  const float* const X1 = s.X[1];
  const float* const Y0 = s.Y[0];
  const float* const Y1 = s.Y[1];
  auto gload = [&](int vb) {
    const int seg = (MODE == 0) ? vb / kbps : 0;
    const int k0 = (vb - seg * kbps) * BK;
    if (MODE == 0) {
      ldx(seg ? X1 : X0, k0, g[0]);
      ldy(seg ? Y1 : Y0, k0, g[1]);
    } else if (MODE == 1) {
      ldx(X0, k0, g[0]);
      ldx(X1, k0, g[1]);
      ldy(Y0, k0, g[2]);
      ldy(Y1, k0, g[3]);
    } else {
      ldx(X0, k0, g[0]);
      ldy(Y0, k0, g[1]);
      ldy(Y1, k0, g[2]);
    }
  };
  auto sstore = [&](int buf) {
    if (SQ) {
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int i = 0; i < V1; ++i) g[t][i] *= g[t][i];
    }
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
  // Operand fragments of one K block (KF k values per lane and block), and
  // the MFMAs that consume them.
  constexpr int KF = M16 ? 4 : HK;
  constexpr int NXT = MODE == 1 ? 2 : 1;     // X tiles per K block
  struct Frags {
    float x0[NB][KF], x1[NB][KF], y0[NB][KF], y1[NB][KF];
  };
  auto fetch = [&](Frags& f, int buf) {
    const float* lx0 = lds[buf][0];
    const float* lx1 = lds[buf][NXT - 1];
    const float* ly0 = lds[buf][NXT];
    const float* ly1 = lds[buf][T - 1];
    if constexpr (M16) {
      const int rx = wm * HALF + r16, ry = wn * HALF + r16;
#pragma unroll
      for (int a = 0; a < NB; ++a) {
        TX::frag16(lx0, rx + 16 * a, g16, f.x0[a]);
        if (MODE == 1) TX::frag16(lx1, rx + 16 * a, g16, f.x1[a]);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        TY::frag16(ly0, ry + 16 * b, g16, f.y0[b]);
        if (MODE != 0) TY::frag16(ly1, ry + 16 * b, g16, f.y1[b]);
      }
    } else {
#pragma unroll
      for (int a = 0; a < NB; ++a) {
        TX::frag(lx0, wm * 32 * W + a * 32 + li, h, f.x0[a]);
        if (MODE == 1) TX::frag(lx1, wm * 32 * W + a * 32 + li, h, f.x1[a]);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        TY::frag(ly0, wn * 32 * W + b * 32 + li, h, f.y0[b]);
        if (MODE != 0) TY::frag(ly1, wn * 32 * W + b * 32 + li, h, f.y1[b]);
      }
    }
  };
  auto mma = [&](const Frags& f) {
#pragma unroll
    for (int k = 0; k < KF; ++k)
#pragma unroll
      for (int a = 0; a < NB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          if constexpr (M16) {
            acc0[a][b] = mfma16(f.x0[a][k], f.y0[b][k], acc0[a][b]);
            if (MODE == 1) {
              acc1[a][b] = mfma16(f.x1[a][k], f.y0[b][k], acc1[a][b]);
              acc1[a][b] = mfma16(f.x0[a][k], f.y1[b][k], acc1[a][b]);
            } else if (MODE == 2) {
              acc1[a][b] = mfma16(f.x0[a][k], f.y1[b][k], acc1[a][b]);
            }
          } else {
            acc0[a][b] = mfma(f.x0[a][k], f.y0[b][k], acc0[a][b]);
            if (MODE == 1) {
              acc1[a][b] = mfma(f.x1[a][k], f.y0[b][k], acc1[a][b]);
              acc1[a][b] = mfma(f.x0[a][k], f.y1[b][k], acc1[a][b]);
            } else if (MODE == 2) {
              acc1[a][b] = mfma(f.x0[a][k], f.y1[b][k], acc1[a][b]);
            }
          }
        }
  };
  auto compute = [&](int buf) {
    Frags f;
    fetch(f, buf);
    mma(f);
  };

  // bias sums: thread t owns column t % ROWS and KPT consecutive k of a block
  constexpr int KPT = BK * ROWS / NT;
  const bool do_bias = BIAS && tn == 0 && (e.bias_out || e.bias_part);
  double bsum = 0.0;
  if constexpr (DMA) {
    constexpr int NYT = T - NXT;               // Y tiles per K block
    constexpr int LPB = NXT * TX::INSTR + NYT * TY::INSTR;
    static_assert(S >= 2 && S <= 4 && (S - 2) * LPB < 64, "pipeline depth");
    size_t offx[TX::INSTR], offy[TY::INSTR];
#pragma unroll
    for (int j = 0; j < TX::INSTR; ++j) offx[j] = TX::dma_src(s.ldx, s.M, m0, wave, lane, j);
#pragma unroll
    for (int j = 0; j < TY::INSTR; ++j) offy[j] = TY::dma_src(s.ldy, s.N, n0, wave, lane, j);
    const int nblk = vb1 > vb0 ? vb1 - vb0 : 0;
    // K block vb into stage st: direct loads for a full block; a ragged last
    // block takes guarded register loads (zeros past K), whose wait also
    // drains every direct load issued before them
    auto issue = [&](int vb, int st) {
      const int seg = (MODE == 0) ? vb / kbps : 0;
      const int k0 = (vb - seg * kbps) * BK;
      if (k0 + BK <= s.K) {
        const size_t kx = XK ? (size_t)k0 : (size_t)k0 * s.ldx;
        const size_t ky = YK ? (size_t)k0 : (size_t)k0 * s.ldy;
#pragma unroll
        for (int t = 0; t < NXT; ++t) {
          const float* x = ((MODE == 0 ? seg : t) ? X1 : X0) + kx;
#pragma unroll
          for (int j = 0; j < TX::INSTR; ++j)
            dma16(x + offx[j], lds[st][t] + (wave * TX::INSTR + j) * 256);
        }
#pragma unroll
        for (int t = 0; t < NYT; ++t) {
          const float* y = ((MODE == 0 ? seg : t) ? Y1 : Y0) + ky;
#pragma unroll
          for (int j = 0; j < TY::INSTR; ++j)
            dma16(y + offy[j], lds[st][NXT + t] + (wave * TY::INSTR + j) * 256);
        }
      } else {
        gload(vb);
        sstore(st);
      }
    };
#pragma unroll
    for (int i = 0; i < S - 1; ++i)
      if (i < nblk) issue(vb0 + i, i);
    for (int it = 0; it < nblk; ++it) {
      // this wave's loads of block it have landed once at most
      // min(S - 2, nblk - 1 - it) later blocks are still pending
      const int ahead = min(S - 2, nblk - 1 - it);
      wait_vm<(S - 2) * LPB>();
      if (S > 3 && ahead == 1) wait_vm<(S > 3 ? LPB : 0)>();
      if (ahead == 0) wait_vm<0>();
      stage_barrier();     // every wave's loads landed; stage it - 1 is free
      if (it + S - 1 < nblk) issue(vb0 + it + S - 1, (it + S - 1) % S);
      const int st = it % S;
      compute(st);
      if (BIAS && do_bias && vb0 + it < kbps) {
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk)
          bsum += (double)lds[st][0][TX::kr((tid / ROWS) * KPT + kk, tid % ROWS)];
      }
    }
  } else
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
        // X tile is [k][m] (XK = false)
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk)
          bsum += (double)lds[buf][0][TX::kr((tid / ROWS) * KPT + kk, tid % ROWS)];
      }
      if (more) sstore(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }
  }
  if (BIAS && do_bias) {
    // NT / ROWS threads hold partial sums of one row, over consecutive k;
    // they are added in k order
    constexpr int PARTS = NT / ROWS;
    __shared__ double bparts[NT];
    if (PARTS > 1 && tid >= ROWS) bparts[tid - ROWS] = bsum;
    __syncthreads();
    if (tid < ROWS && m0 + tid < s.M) {
      double t = bsum;
#pragma unroll
      for (int q = 1; q < PARTS; ++q) t += bparts[(q - 1) * ROWS + tid];
      if (s.splits > 1) e.bias_part[(size_t)blockIdx.z * s.M + m0 + tid] = t;
      else e.bias_out[m0 + tid] = (float)t;
    }
  }

  if constexpr (M16) {
    // 16x16 f32 accumulator layout: lane (r16, g16), register r holds row
    // 4 * g16 + r, column r16 of the 16 x 16 block.
#pragma unroll
    for (int a = 0; a < NB; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const Acc v0 = acc0[a][b];
        const Acc v1 = MODE == 0 ? v0 : acc1[a][b];
        const int rbase = m0 + wm * HALF + a * 16 + 4 * g16;
        const int col = n0 + wn * HALF + b * 16 + r16;
        if (col < s.N) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = rbase + r;
            if (row < s.M) Epi::apply(e, row, col, v0[r], MODE == 0 ? 0.0f : v1[r]);
          }
        }
        // 128 x 128 tiles: keep the scheduler from hoisting every block's
        // epilogue loads to the top (registers); a 64 x 64 tile's four
        // blocks may issue theirs together
        if constexpr (TS == 128) __builtin_amdgcn_sched_barrier(0);
      }
  } else {
    // 32x32 f32 accumulator layout: lane (li, h), register r holds
    // row 8 * (r / 4) + 4 * h + r % 4, column li of the 32 x 32 block.
#pragma unroll
    for (int a = 0; a < W; ++a)
#pragma unroll
      for (int b = 0; b < W; ++b) {
        const Acc v0 = acc0[a][b];
        const Acc v1 = MODE == 0 ? v0 : acc1[a][b];
        const int rbase = m0 + wm * 32 * W + a * 32 + 4 * h;
        const int col = n0 + wn * 32 * W + b * 32 + li;
        if (col < s.N) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = rbase + 8 * (r >> 2) + (r & 3);
            if (row < s.M) Epi::apply(e, row, col, v0[r], MODE == 0 ? 0.0f : v1[r]);
          }
        }
        // keep the scheduler from hoisting every block's loads to the top
        __builtin_amdgcn_sched_barrier(0);
      }
  }
}

}  // namespace

#define HF_GEMM_KERNEL(NAME, MODE, XK, YK, EPI, BIAS, M16, WAVES)               \
  extern "C" __global__ __launch_bounds__(256, WAVES) void NAME##_v4(GemmShape s,   \
                                                                 EpiArgs e) {   \
    gemm_body<MODE, XK, YK, 4, EPI, BIAS, M16>(s, e);                           \
  }                                                                             \
  extern "C" __global__ __launch_bounds__(256, 1) void NAME##_v1(GemmShape s,   \
                                                                 EpiArgs e) {   \
    gemm_body<MODE, XK, YK, 1, EPI, BIAS, M16>(s, e);                           \
  }

// M16 selects the 16 x 16 form (measured on the speech-frame net: bwd_rbwd
// +22%, bwd and gnbwd +3%, wgrad +1.5%, fwd +1%; with direct loads, rfwd
// +2.6%; the fused forward + R-forward kernels, which write three row-major
// outputs, ran 2.6% slower in it).  WAVES is the occupancy the register
// allocation is held to: four waves per SIMD (128 registers) made the
// batch-row kernels 1-3% faster than three; the weight gradient spills at
// four and keeps three; the dual kernels at two waves (202-228 registers,
// no spills) ran 6-20% faster than at one.
HF_GEMM_KERNEL(hf_gemm_fwd, 0, true, false, EFwd, false, true, 4)
HF_GEMM_KERNEL(hf_gemm_fwd_rfwd, 1, true, true, EFwdRFwd, false, false, 2)
HF_GEMM_KERNEL(hf_gemm_fwd_rfwd0, 2, true, true, EFwdRFwd, false, false, 2)
HF_GEMM_KERNEL(hf_gemm_rfwd, 0, true, false, ERFwd, false, true, 4)
HF_GEMM_KERNEL(hf_gemm_bwd, 0, true, false, EBwd, false, true, 4)
HF_GEMM_KERNEL(hf_gemm_bwd_e2, 0, true, false, EBwdE2, false, true, 4)
HF_GEMM_KERNEL(hf_gemm_bwd_rbwd, 1, true, false, EBwdRBwd, false, true, 2)
HF_GEMM_KERNEL(hf_gemm_rbwd, 0, true, false, ERBwd, false, true, 4)
HF_GEMM_KERNEL(hf_gemm_gnbwd, 0, true, false, EGNBwd, false, true, 4)
HF_GEMM_KERNEL(hf_gemm_wgrad, 0, false, false, EStore, true, true, 3)
// split-K partials of the batch-row single-product GEMMs (X K-contiguous,
// Y row-contiguous): out0[z * split_stride + m * ldo + n]
HF_GEMM_KERNEL(hf_gemm_part, 0, true, false, EStore, false, true, 4)

// 64 x 64 output tiles for small outputs (gemm_tile): four times the
// workgroups of the 128 x 128 form, a quarter of the MFMA chain per
// workgroup and K block, and a quarter of the padding for a narrow output.
#define HF_GEMM_KERNEL64(NAME, XK, YK, EPI, BIAS, SQ)                            \
  extern "C" __global__ __launch_bounds__(256, 4) void NAME##_t64_v4(          \
      GemmShape s, EpiArgs e) {                                                \
    gemm_body<0, XK, YK, 4, EPI, BIAS, true, SQ, 64>(s, e);                     \
  }                                                                             \
  extern "C" __global__ __launch_bounds__(256, 4) void NAME##_t64_v1(          \
      GemmShape s, EpiArgs e) {                                                \
    gemm_body<0, XK, YK, 1, EPI, BIAS, true, SQ, 64>(s, e);                     \
  }
HF_GEMM_KERNEL64(hf_gemm_fwd, true, false, EFwd, false, false)
HF_GEMM_KERNEL64(hf_gemm_rfwd, true, false, ERFwd, false, false)
HF_GEMM_KERNEL64(hf_gemm_bwd, true, false, EBwd, false, false)
HF_GEMM_KERNEL64(hf_gemm_bwd_e2, true, false, EBwdE2, false, false)
HF_GEMM_KERNEL64(hf_gemm_rbwd, true, false, ERBwd, false, false)
HF_GEMM_KERNEL64(hf_gemm_gnbwd, true, false, EGNBwd, false, false)
HF_GEMM_KERNEL64(hf_gemm_wgrad, false, false, EStore, true, false)
HF_GEMM_KERNEL64(hf_gemm_part, true, false, EStore, false, false)
HF_GEMM_KERNEL64(hf_gemm_wgrad_sq, false, false, EStore, true, true)

// weight gradient of squared operands: sum over the rows of delta^2 a^2 (the
// per-example squared gradients of a weight layer, up to the batch scale),
// bias sums of delta^2
extern "C" __global__ __launch_bounds__(256, 1) void hf_gemm_wgrad_sq_v4(
    GemmShape s, EpiArgs e) {
  gemm_body<0, false, false, 4, EStore, true, true, true>(s, e);
}
extern "C" __global__ __launch_bounds__(256, 1) void hf_gemm_wgrad_sq_v1(
    GemmShape s, EpiArgs e) {
  gemm_body<0, false, false, 1, EStore, true, true, true>(s, e);
}

namespace {

// Sum of the split-K partials in split order (fp64), then the kernel's own
// epilogue on the sum: the result is that of the unsplit kernel up to the
// rounding of the partial sums.  One thread per output element: its SP
// partial loads and the epilogue's own loads are independent, so they are
// all in flight at once.
template <class Epi, int SP>
__global__ __launch_bounds__(256) void splitk_epi(EpiArgs e, const float* part,
                                                  int M, int N, const int* skip) {
  if (skip && *skip) return;
  const size_t mn = (size_t)M * N;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= mn) return;
  float p[SP];
#pragma unroll
  for (int z = 0; z < SP; ++z) p[z] = part[z * mn + i];
  double v = 0.0;
#pragma unroll
  for (int z = 0; z < SP; ++z) v += (double)p[z];
  int r, c;
  if (mn <= 0xffffffffu) {
    r = (int)((uint32_t)i / (uint32_t)N);
    c = (int)((uint32_t)i - (uint32_t)r * (uint32_t)N);
  } else {
    r = (int)(i / (size_t)N);
    c = (int)(i - (size_t)r * N);
  }
  Epi::apply(e, r, c, (float)v, 0.0f);
}

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

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

void launch(const Launch& L, const char* name, GemmKernel k4, GemmKernel k1,
            int rows, int mode, const GemmShape& s, const EpiArgs& e,
            double flops, double bytes) {
  const int vec = pick_vec(s, mode);
  dim3 grid(cdiv(s.N, rows), cdiv(s.M, rows),
            (mode == 0 && s.splits > 1) ? s.splits : 1);
  prof_begin(L, name);
  hipExtLaunchKernelGGL(vec == 4 ? k4 : k1, grid, dim3(NT), 0, L.stream, prof_a(L), prof_b(L), 0, s, e);
  prof_end(L, name, flops, bytes);
}

// The four kernels of a single-product GEMM: 128 and 64 tiles, 16-byte and
// element loads
struct Kernels {
  GemmKernel k4, k1, t4, t1;
};
#define HF_KERNELS(NAME) Kernels{NAME##_v4, NAME##_v1, NAME##_t64_v4, NAME##_t64_v1}

void launch_single(const Launch& L, const char* name, const Kernels& k,
                   const GemmShape& s, const EpiArgs& e, double flops,
                   double bytes) {
  if (gemm_tile(s.M, s.N, s.K * s.nseg) == 64)
    launch(L, name, k.t4, k.t1, 64, 0, s, e, flops, bytes);
  else
    launch(L, name, k.k4, k.k1, 128, 0, s, e, flops, bytes);
}

#define HF_LAUNCH_SINGLE(NAME, L, s, e, fl, by) \
  launch_single(L, #NAME, HF_KERNELS(NAME), s, e, fl, by)

// Split-K factor for a batch-row single-product GEMM: enough workgroups for
// two per compute unit while every split keeps at least 64 of K (4 K
// blocks), within the scratch.  1 = no split (always so at the speech net's
// full batch).
int row_splits(const GemmShape& s, const EpiArgs& e) {
  if (!e.split_buf) return 1;
  const int ts = gemm_tile(s.M, s.N, s.K * s.nseg);
  const long long tiles = (long long)cdiv(s.M, ts) * cdiv(s.N, ts);
  const int ktot = s.K * s.nseg;
  int sp = 1;
  while (sp < 16 && tiles * sp < 512 && ktot / (2 * sp) >= 64) sp *= 2;
  while (sp > 1 && (long long)sp * s.M * s.N > e.split_cap) sp /= 2;
  return sp;
}

// A batch-row single-product GEMM: one kernel with its epilogue, or, when
// the output has too few tiles, split-K partials into the scratch (timed
// under the kernel's name) and the reduce that applies the epilogue.
template <class Epi>
void launch_rows(const Launch& L, const char* name, const Kernels& k,
                 const GemmShape& s, const EpiArgs& e, double flops, double bytes) {
  const int sp = row_splits(s, e);
  if (sp == 1) {
    launch_single(L, name, k, s, e, flops, bytes);
    return;
  }
  GemmShape ps = s;
  ps.splits = sp;
  EpiArgs pe = e;
  pe.out0 = e.split_buf;
  pe.ldo = s.N;
  pe.split_stride = (long long)s.M * s.N;
  launch_single(L, name, HF_KERNELS(hf_gemm_part), ps, pe, flops,
                bytes + 4.0 * sp * s.M * (double)s.N);
  const long long mn = (long long)s.M * s.N;
  const dim3 grid((unsigned)((mn + 255) / 256));
  // sp is a power of two from 2 to 16 (row_splits doubles from 1)
  void (*kr)(EpiArgs, const float*, int, int, const int*) =
      sp == 2 ? splitk_epi<Epi, 2> : sp == 4 ? splitk_epi<Epi, 4>
      : sp == 8 ? splitk_epi<Epi, 8> : splitk_epi<Epi, 16>;
  prof_begin(L, "hf_splitk_epi");
  hipExtLaunchKernelGGL(kr, grid, dim3(256), 0, L.stream, prof_a(L), prof_b(L), 0, e,
                        (const float*)e.split_buf, s.M, s.N, s.skip);
  prof_end(L, "hf_splitk_epi", 0.0, 4.0 * (sp + 1) * (double)mn);
}

#define HF_LAUNCH_ROWS(NAME, EPI, L, s, e, fl, by) \
  launch_rows<EPI>(L, #NAME, HF_KERNELS(NAME), s, e, fl, by)

inline double mnk(const GemmShape& s) { return 2.0 * s.M * s.N * (double)s.K; }
inline double io(const GemmShape& s, int nx, int ny, int nout) {
  return 4.0 * ((double)s.M * s.K * nx + (double)s.N * s.K * ny +
                (double)s.M * s.N * nout);
}

}  // namespace

int gemm_tile(int M, int N, int K) {
  if (M <= 64 || N <= 64) return 64;
  const long long t128 = (long long)cdiv(M, 128) * cdiv(N, 128);
  const long long splits = std::max(1, std::min(32, K / 128));
  return t128 * splits < 256 ? 64 : 128;
}

void gemm_fwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  HF_LAUNCH_ROWS(hf_gemm_fwd, EFwd, L, s, e, mnk(s) * s.nseg, io(s, s.nseg, s.nseg, 1));
}
void gemm_fwd_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  if (s.X[1]) {
    launch(L, "hf_gemm_fwd_rfwd", hf_gemm_fwd_rfwd_v4, hf_gemm_fwd_rfwd_v1,
           128, 1, s, e, 3 * mnk(s), io(s, 2, 2, e.hidden ? 3 : 2));
  } else {
    launch(L, "hf_gemm_fwd_rfwd0", hf_gemm_fwd_rfwd0_v4, hf_gemm_fwd_rfwd0_v1,
           128, 2, s, e, 2 * mnk(s), io(s, 1, 2, e.hidden ? 3 : 2));
  }
}
void gemm_rfwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  HF_LAUNCH_ROWS(hf_gemm_rfwd, ERFwd, L, s, e, mnk(s) * s.nseg,
                   io(s, s.nseg, s.nseg, e.hidden ? (e.out1 ? 3 : 2) : 1));
}
void gemm_bwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  if (e.out2)
    HF_LAUNCH_ROWS(hf_gemm_bwd_e2, EBwdE2, L, s, e, mnk(s) * s.nseg,
                     io(s, s.nseg, s.nseg, 3));
  else
    HF_LAUNCH_ROWS(hf_gemm_bwd, EBwd, L, s, e, mnk(s) * s.nseg,
                     io(s, s.nseg, s.nseg, 2));
}
void gemm_bwd_rbwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  launch(L, "hf_gemm_bwd_rbwd", hf_gemm_bwd_rbwd_v4, hf_gemm_bwd_rbwd_v1, 128,
         1, s, e, 3 * mnk(s), io(s, 2, 2, 4));
}
void gemm_rbwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  HF_LAUNCH_ROWS(hf_gemm_rbwd, ERBwd, L, s, e, mnk(s) * s.nseg, io(s, s.nseg, s.nseg, 4));
}
void gemm_gnbwd(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  HF_LAUNCH_ROWS(hf_gemm_gnbwd, EGNBwd, L, s, e, mnk(s) * s.nseg, io(s, s.nseg, s.nseg, 2));
}
void gemm_wgrad(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  HF_LAUNCH_SINGLE(hf_gemm_wgrad, L, s, e, mnk(s) * s.nseg,
                   io(s, s.nseg, s.nseg, s.splits > 1 ? s.splits : 1));
}
void gemm_wgrad_sq(const Launch& L, const GemmShape& s, const EpiArgs& e) {
  HF_LAUNCH_SINGLE(hf_gemm_wgrad_sq, L, s, e, mnk(s) * s.nseg,
                   io(s, s.nseg, s.nseg, s.splits > 1 ? s.splits : 1));
}

}  // namespace hfk
