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
// Operand buffers are laid out so that no load needs a bounds check: every
// leading dimension is a multiple of 64 with zeros between K and the next
// multiple of 64, and every operand has rows up to the next multiple of 256
// (rows past M or N only feed outputs that are not stored).  The epilogues
// keep the zeros: a transposed copy gets zeros in its rows M .. (M rounded
// up to 64), which the next weight-gradient GEMM reads as K padding.
//
// A workgroup of GM x GN wave64s owns a (32 WM GM) x (32 WN GN) output
// tile; each wave owns WM x WN blocks of 32 x 32.  Tiles are handed out in
// an order that keeps neighbouring tiles on one XCD (the hardware deals
// consecutive workgroups to the 8 XCDs in turn, each with its own L2) and,
// within an XCD, walks groups of 8 tile rows column by column, so that the
// workgroups resident at one time share their operand panels in L2.
// K advances BK at a time through S stages of LDS, filled by direct
// global-to-LDS loads (global_load_lds_dwordx4) issued S - 1 blocks ahead of
// the block the MFMAs consume: no registers stage the operands, and each
// wave waits only for the loads of the block it is about to read.
// LDS tiles are [row][k]; the 16-byte chunks of a row are XOR-swizzled so
// that the 128-bit fragment loads are free of bank conflicts.  A direct
// load writes lane i's 16 bytes at 16 i past the wave's LDS base, so the
// swizzle is applied by choosing which global chunk each lane fetches.
// Lane (i, h) of an MFMA feeds the 8 consecutive k values 8h .. 8h + 7 of
// its row for both operands, so the sum over k is exact up to its order.
#include "act.h"
#include "hf_internal.h"
#include "lds_dma.h"

namespace hfk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16_t h) {
  return __uint_as_float((uint32_t)h << 16);
}
// round to nearest even
__device__ __forceinline__ bf16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// ------------------------------------------------------------ tile loading
// A ROWS x BK tile kept in LDS as [row][k]; the CH 16-byte chunks of a row
// are XOR-swizzled by (row / RPB) % CH, RPB being the number of rows that
// span the 64 banks.  Chunk position P of the tile (P = row * CH + pos, 64
// chunks per direct-load instruction) holds global chunk pos ^ swz(row).
template <int ROWS, int BK, int NW>
struct Tile {
  static constexpr int CH = BK / 8;
  static constexpr int RPB = 128 / BK;
  static constexpr int SIZE = ROWS * BK;             // bf16 elements
  static constexpr int INSTR = ROWS * CH / 64 / NW;  // direct loads per wave
  static_assert(INSTR >= 1 && ROWS * CH % (64 * NW) == 0, "tile does not split over the waves");

  __device__ static __forceinline__ int swz(int row) { return (row / RPB) % CH; }
  // element offset, within an operand of leading dimension ld, of the chunk
  // that lane `lane` of wave `wave` fetches with its instruction j
  __device__ static __forceinline__ uint32_t src(int ld, int wave, int lane, int j) {
    const int P = (wave * INSTR + j) * 64 + lane;
    const int row = P / CH, pos = P % CH;
    return (uint32_t)row * (uint32_t)ld + 8u * (uint32_t)(pos ^ swz(row));
  }
  // LDS element offset of the 64 chunks written by instruction j of a wave
  __device__ static __forceinline__ int dst(int wave, int j) {
    return (wave * INSTR + j) * 512;
  }
  // operand of MFMA step q (k = 16 q .. 16 q + 15) for lane (row, h)
  __device__ static __forceinline__ bf16x8 frag(const bf16_t* __restrict__ s,
                                                int row, int h, int q) {
    const int c = 2 * q + h;
    return *(const bf16x8*)(s + row * BK + ((c ^ swz(row)) * 8));
  }
  // sum of the 8 k values of chunk c of a row
  __device__ static __forceinline__ float chunk_sum(const bf16_t* __restrict__ s,
                                                    int row, int c) {
    const u32x4 v = *(const u32x4*)(s + row * BK + ((c ^ swz(row)) * 8));
    float t = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      t += __uint_as_float(v[j] << 16) + __uint_as_float(v[j] & 0xffff0000u);
    return t;
  }
};

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ----------------------------------------------------------------- epilogues
// An epilogue handles 4 consecutive rows r0 .. r0 + 3 (r0 a multiple of 4)
// of one column c < N, with r0 below M rounded up to 64.  Row-major bf16
// outputs h* (leading dimension ldo) and fp32 outputs f* (ldf) are stored
// for rows below M; the transposed copy t* gets the 4 rows as one 8-byte
// store, with zeros for rows at or past M.  aux a0 is bf16 with ldo, a1 and
// a2 are fp32 with ldf; their rows exist up to the next multiple of 256, so
// they are read without checks and only masked.
struct Q {                          // 4 consecutive rows of one column
  float v[4];
};

__device__ __forceinline__ void st_h(const EpiH& e, bf16_t* h, int r0, int c,
                                     const Q& q, int M) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (r0 + j < M) h[(size_t)(r0 + j) * e.ldo + c] = f2bf(q.v[j]);
}
__device__ __forceinline__ void st_t(const EpiH& e, bf16_t* t, int r0, int c,
                                     const Q& q, int M) {
  uint32_t w[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const uint32_t lo = r0 + 2 * j < M ? f2bf(q.v[2 * j]) : 0u;
    const uint32_t hi = r0 + 2 * j + 1 < M ? f2bf(q.v[2 * j + 1]) : 0u;
    w[j] = lo | (hi << 16);
  }
  *(u32x2*)(t + (size_t)c * e.ldt + r0) = u32x2{w[0], w[1]};
}
__device__ __forceinline__ void st_ht(const EpiH& e, bf16_t* h, bf16_t* t,
                                      int r0, int c, const Q& q, int M) {
  st_h(e, h, r0, c, q, M);
  if (t) st_t(e, t, r0, c, q, M);
}
__device__ __forceinline__ void st_f(const EpiH& e, float* f, int r0, int c,
                                     const Q& q, int M) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (r0 + j < M) f[(size_t)(r0 + j) * e.ldf + c] = q.v[j];
}
__device__ __forceinline__ Q ld_a0(const EpiH& e, int r0, int c) {
  Q a;
#pragma unroll
  for (int j = 0; j < 4; ++j) a.v[j] = bf2f(e.a0[(size_t)(r0 + j) * e.ldo + c]);
  return a;
}
__device__ __forceinline__ Q ld_f(const EpiH& e, const float* f, int r0, int c) {
  Q a;
#pragma unroll
  for (int j = 0; j < 4; ++j) a.v[j] = f[(size_t)(r0 + j) * e.ldf + c];
  return a;
}

// Epilogues with bf16 outputs also have a staged form (see stage_epilogue):
//   NB        bf16 outputs (row-major h + transposed t pairs) when staged
//   A0        whether it reads a0
//   staged(e) whether this launch writes bf16 outputs
//   stage()   fp32 outputs stored directly, bf16 output values returned in o[]
//             (a = the a0 values of the 4 rows, when A0)
//   hout/tout the row-major and transposed destinations of bf16 output i
struct EFwd {
  static constexpr int NB = 1;
  static constexpr bool A0 = false;
  static __device__ __forceinline__ bool staged(const EpiH& e) { return e.hidden; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int) { return e.h0; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int) { return e.t0; }
  static __device__ __forceinline__ void stage(const EpiH& e, int r0, int c, int M,
                                               const Q& v0, const Q&, const Q&, Q* o) {
#pragma unroll
    for (int j = 0; j < 4; ++j) o[0].v[j] = act_f(e.act, v0.v[j] + e.bias[c]);
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
    Q z;
#pragma unroll
    for (int j = 0; j < 4; ++j) z.v[j] = v0.v[j] + e.bias[c];
    if (e.hidden) {
      Q a;
#pragma unroll
      for (int j = 0; j < 4; ++j) a.v[j] = act_f(e.act, z.v[j]);
      st_ht(e, e.h0, e.t0, r0, c, a, M);
    } else {
      st_f(e, e.f0, r0, c, z, M);
    }
  }
};
struct EFwdRFwd {
  static constexpr int NB = 2;
  static constexpr bool A0 = false;
  static __device__ __forceinline__ bool staged(const EpiH& e) { return e.hidden; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int i) { return i ? e.h2 : e.h0; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int i) { return i ? e.t2 : e.t0; }
  static __device__ __forceinline__ void stage(const EpiH& e, int r0, int c, int M,
                                               const Q& v0, const Q& v1, const Q&, Q* o) {
    Q rz;
#pragma unroll
    for (int j = 0; j < 4; ++j) rz.v[j] = v1.v[j] + e.rbias[c];
    if (e.f1) st_f(e, e.f1, r0, c, rz, M);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a = act_f(e.act, v0.v[j] + e.bias[c]);
      o[0].v[j] = a;
      o[1].v[j] = act_d1(e.act, a) * rz.v[j];
    }
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q& v1) {
    Q z, rz;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      z.v[j] = v0.v[j] + e.bias[c];
      rz.v[j] = v1.v[j] + e.rbias[c];
    }
    if (e.f1) st_f(e, e.f1, r0, c, rz, M);
    if (e.hidden) {
      Q a, ra;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a.v[j] = act_f(e.act, z.v[j]);
        ra.v[j] = act_d1(e.act, a.v[j]) * rz.v[j];
      }
      st_ht(e, e.h0, e.t0, r0, c, a, M);
      st_ht(e, e.h2, e.t2, r0, c, ra, M);
    } else {
      st_f(e, e.f0, r0, c, z, M);
    }
  }
};
struct ERFwd {
  static constexpr int NB = 1;
  static constexpr bool A0 = true;
  static __device__ __forceinline__ bool staged(const EpiH& e) { return e.hidden; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int) { return e.h2; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int) { return e.t2; }
  static __device__ __forceinline__ void stage(const EpiH& e, int r0, int c, int M,
                                               const Q& v0, const Q&, const Q& a, Q* o) {
    Q rz;
#pragma unroll
    for (int j = 0; j < 4; ++j) rz.v[j] = v0.v[j] + e.rbias[c];
    if (e.f1) st_f(e, e.f1, r0, c, rz, M);
#pragma unroll
    for (int j = 0; j < 4; ++j) o[0].v[j] = act_d1(e.act, a.v[j]) * rz.v[j];
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
    Q rz;
#pragma unroll
    for (int j = 0; j < 4; ++j) rz.v[j] = v0.v[j] + e.rbias[c];
    if (e.f1) st_f(e, e.f1, r0, c, rz, M);
    if (e.hidden) {
      const Q a = ld_a0(e, r0, c);
      Q ra;
#pragma unroll
      for (int j = 0; j < 4; ++j) ra.v[j] = act_d1(e.act, a.v[j]) * rz.v[j];
      st_ht(e, e.h2, e.t2, r0, c, ra, M);
    }
  }
};
struct EBwd {
  static constexpr int NB = 1;
  static constexpr bool A0 = true;
  static __device__ __forceinline__ bool staged(const EpiH&) { return true; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int) { return e.h0; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int) { return e.t0; }
  static __device__ __forceinline__ void stage(const EpiH& e, int, int, int,
                                               const Q& v0, const Q&, const Q& a, Q* o) {
#pragma unroll
    for (int j = 0; j < 4; ++j) o[0].v[j] = v0.v[j] * act_d1(e.act, a.v[j]);
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
    const Q a = ld_a0(e, r0, c);
    Q d;
#pragma unroll
    for (int j = 0; j < 4; ++j) d.v[j] = v0.v[j] * act_d1(e.act, a.v[j]);
    st_ht(e, e.h0, e.t0, r0, c, d, M);
  }
};
// backward data that also caches E * phi''(A) for the Hessian product
struct EBwdE2 {
  static constexpr int NB = 1;
  static constexpr bool A0 = true;
  static __device__ __forceinline__ bool staged(const EpiH&) { return true; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int) { return e.h0; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int) { return e.t0; }
  static __device__ __forceinline__ void stage(const EpiH& e, int r0, int c, int M,
                                               const Q& v0, const Q&, const Q& a, Q* o) {
    Q e2;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[0].v[j] = v0.v[j] * act_d1(e.act, a.v[j]);
      e2.v[j] = v0.v[j] * act_d2(e.act, a.v[j]);
    }
    st_f(e, e.f2, r0, c, e2, M);
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
    const Q a = ld_a0(e, r0, c);
    Q d, e2;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      d.v[j] = v0.v[j] * act_d1(e.act, a.v[j]);
      e2.v[j] = v0.v[j] * act_d2(e.act, a.v[j]);
    }
    st_ht(e, e.h0, e.t0, r0, c, d, M);
    st_f(e, e.f2, r0, c, e2, M);
  }
};
struct EBwdRBwd {
  static constexpr int NB = 2;
  static constexpr bool A0 = true;
  static __device__ __forceinline__ bool staged(const EpiH&) { return true; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int i) { return i ? e.h1 : e.h0; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int i) { return i ? e.t1 : e.t0; }
  static __device__ __forceinline__ void stage(const EpiH& e, int r0, int c, int,
                                               const Q& v0, const Q& v1, const Q& a, Q* o) {
    const Q rz = ld_f(e, e.a1, r0, c);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float d1 = act_d1(e.act, a.v[j]);
      o[0].v[j] = v0.v[j] * d1;
      o[1].v[j] = v1.v[j] * d1 + v0.v[j] * act_d2(e.act, a.v[j]) * rz.v[j];
    }
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q& v1) {
    const Q a = ld_a0(e, r0, c);
    const Q rz = ld_f(e, e.a1, r0, c);
    Q d, rd;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float d1 = act_d1(e.act, a.v[j]);
      d.v[j] = v0.v[j] * d1;
      rd.v[j] = v1.v[j] * d1 + v0.v[j] * act_d2(e.act, a.v[j]) * rz.v[j];
    }
    st_ht(e, e.h0, e.t0, r0, c, d, M);
    st_ht(e, e.h1, e.t1, r0, c, rd, M);
  }
};
struct ERBwd {
  static constexpr int NB = 1;
  static constexpr bool A0 = true;
  static __device__ __forceinline__ bool staged(const EpiH&) { return true; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int) { return e.h1; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int) { return e.t1; }
  static __device__ __forceinline__ void stage(const EpiH& e, int r0, int c, int,
                                               const Q& v0, const Q&, const Q& a, Q* o) {
    const Q rz = ld_f(e, e.a1, r0, c);
    const Q e2 = ld_f(e, e.a2, r0, c);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[0].v[j] = v0.v[j] * act_d1(e.act, a.v[j]) + e2.v[j] * rz.v[j];
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
    const Q a = ld_a0(e, r0, c);
    const Q rz = ld_f(e, e.a1, r0, c);
    const Q e2 = ld_f(e, e.a2, r0, c);
    Q rd;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      rd.v[j] = v0.v[j] * act_d1(e.act, a.v[j]) + e2.v[j] * rz.v[j];
    st_ht(e, e.h1, e.t1, r0, c, rd, M);
  }
};
struct EGNBwd {
  static constexpr int NB = 1;
  static constexpr bool A0 = true;
  static __device__ __forceinline__ bool staged(const EpiH&) { return true; }
  static __device__ __forceinline__ bf16_t* hout(const EpiH& e, int) { return e.h1; }
  static __device__ __forceinline__ bf16_t* tout(const EpiH& e, int) { return e.t1; }
  static __device__ __forceinline__ void stage(const EpiH& e, int, int, int,
                                               const Q& v0, const Q&, const Q& a, Q* o) {
#pragma unroll
    for (int j = 0; j < 4; ++j) o[0].v[j] = v0.v[j] * act_d1(e.act, a.v[j]);
  }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
    const Q a = ld_a0(e, r0, c);
    Q rd;
#pragma unroll
    for (int j = 0; j < 4; ++j) rd.v[j] = v0.v[j] * act_d1(e.act, a.v[j]);
    st_ht(e, e.h1, e.t1, r0, c, rd, M);
  }
};
struct EStore {                      // fp32 only: never staged
  static constexpr int NB = 0;
  static constexpr bool A0 = false;
  static __device__ __forceinline__ bool staged(const EpiH&) { return false; }
  static __device__ __forceinline__ void apply(const EpiH& e, int r0, int c, int M, int zs,
                                               const Q& v0, const Q&) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (r0 + j < M)
        e.f0[(size_t)zs * e.split_stride + (size_t)(r0 + j) * e.ldf + c] = v0.v[j];
  }
};

// ------------------------------------------------------------- tile order
// The tile (tn, tm) and split tz this workgroup computes.  Linear dispatch
// index L goes to XCD L % 8; when the grid is a multiple of 8, XCD x gets
// the x-th contiguous eighth of the logical order.  Within a split, the
// logical order walks groups of 8 tile rows, column by column.
__device__ __forceinline__ void tile_of(int& tn, int& tm, int& tz) {
  const int gx = gridDim.x, gy = gridDim.y;
  const int T = gx * gy * gridDim.z;
  const int L = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int Lg = (T % 8 == 0) ? (L % 8) * (T / 8) + L / 8 : L;
  tz = Lg / (gx * gy);
  const int r = Lg % (gx * gy);
  constexpr int G = 8;
  const int g = r / (G * gx);
  const int first = g * G;
  const int rows = min(G, gy - first);
  const int w = r - g * G * gx;
  tm = first + w % rows;
  tn = w / rows;
}

// ------------------------------------------------------------------- body
#ifndef HF_H_STAGE
#define HF_H_STAGE 1
#endif

// MODE 0: single (nseg K-segments, optional split-K over grid z)
// MODE 1: dual   acc0 = X0 Y0, acc1 = X1 Y0 + X0 Y1
// MODE 2: dual0  acc0 = X0 Y0, acc1 = X0 Y1
// BIAS (weight gradient): blocks of the first column tile also sum their X
// tiles of K-segment 0 over k, giving sum_k X(m, k) for their rows.
template <int MODE, class Epi, bool BIAS, int WM, int WN, int GM, int GN, int BK, int S>
__device__ __forceinline__ void hgemm_body(const GemmShapeH& s, const EpiH& e) {
  if (s.skip && *s.skip) return;
  constexpr int NW = GM * GN, NT = 64 * NW;
  constexpr int RM = 32 * WM * GM, RN = 32 * WN * GN;
  using TX = Tile<RM, BK, NW>;
  using TY = Tile<RN, BK, NW>;
  constexpr int NX = MODE == 1 ? 2 : 1;      // X tiles per K block
  constexpr int NY = MODE == 0 ? 1 : 2;      // Y tiles per K block
  constexpr int STAGE = NX * TX::SIZE + NY * TY::SIZE;
  constexpr int LPB = NX * TX::INSTR + NY * TY::INSTR;   // loads per block per wave
  static_assert(S >= 2 && (S - 2) * LPB < 64, "pipeline depth");
  __shared__ __attribute__((aligned(16))) bf16_t lds[S * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / GN, wn = wave % GN;
  const int li = lane & 31, h = lane >> 5;
  int tn, tm, tz;
  tile_of(tn, tm, tz);
  const int m0 = tm * RM;
  const int n0 = tn * RN;

  const int kbps = (s.K + BK - 1) / BK;
  const int nvb = (MODE == 0 ? s.nseg : 1) * kbps;
  int vb0 = 0, vb1 = nvb;
  if (MODE == 0 && s.splits > 1) {
    const int per = (nvb + s.splits - 1) / s.splits;
    vb0 = tz * per;
    vb1 = min(nvb, vb0 + per);
  }
  const int nblk = vb1 > vb0 ? vb1 - vb0 : 0;

  f32x16 acc0[WM][WN], acc1[WM][WN];
#pragma unroll
  for (int a = 0; a < WM; ++a)
#pragma unroll
    for (int b = 0; b < WN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc0[a][b][r] = 0.0f;
        if (MODE != 0) acc1[a][b][r] = 0.0f;
      }

  // per-lane source offsets of the direct loads, relative to the tile origin
  uint32_t offx[TX::INSTR], offy[TY::INSTR];
#pragma unroll
  for (int j = 0; j < TX::INSTR; ++j) offx[j] = TX::src(s.ldx, wave, lane, j);
#pragma unroll
  for (int j = 0; j < TY::INSTR; ++j) offy[j] = TY::src(s.ldy, wave, lane, j);
  const size_t bx = (size_t)m0 * s.ldx, by = (size_t)n0 * s.ldy;

  // operand pointers in registers: an indexed read of the argument array
  // inside the loop would be a scalar memory load, which shares the LDS
  // wait counter and forces every fragment wait to drain it completely
  const bf16_t* const X0 = s.X[0];
  const bf16_t* const X1 = s.X[1];
  const bf16_t* const Y0 = s.Y[0];
  const bf16_t* const Y1 = s.Y[1];
  // the direct loads of K block vb into stage st (X tiles, then Y tiles)
  auto issue = [&](int vb, int st) {
    const int seg = (MODE == 0) ? vb / kbps : 0;
    const int k0 = (vb - seg * kbps) * BK;
    bf16_t* base = lds + st * STAGE;
#pragma unroll
    for (int t = 0; t < NX; ++t) {
      const bf16_t* x = ((MODE == 0 ? seg : t) ? X1 : X0) + bx + k0;
#pragma unroll
      for (int j = 0; j < TX::INSTR; ++j)
        dma16(x + offx[j], base + t * TX::SIZE + TX::dst(wave, j));
    }
#pragma unroll
    for (int t = 0; t < NY; ++t) {
      const bf16_t* y = ((MODE == 0 ? seg : t) ? Y1 : Y0) + by + k0;
#pragma unroll
      for (int j = 0; j < TY::INSTR; ++j)
        dma16(y + offy[j], base + NX * TX::SIZE + t * TY::SIZE + TY::dst(wave, j));
    }
  };
  const int xrow = wm * 32 * WM + li;
  const int yrow = wn * 32 * WN + li;
  // Fragments of one MFMA step; two sets alternate so that the LDS reads of
  // step q + 1 are in flight while the MFMAs of step q run.
  struct Frags {
    bf16x8 x0[WM], x1[WM], y0[WN], y1[WN];
  };
  auto fetch = [&](Frags& f, int st, int q) {
    const bf16_t* lx0 = lds + st * STAGE;
    const bf16_t* lx1 = lx0 + (NX - 1) * TX::SIZE;
    const bf16_t* ly0 = lds + st * STAGE + NX * TX::SIZE;
    const bf16_t* ly1 = ly0 + (NY - 1) * TY::SIZE;
#pragma unroll
    for (int a = 0; a < WM; ++a) {
      f.x0[a] = TX::frag(lx0, xrow + 32 * a, h, q);
      if (MODE == 1) f.x1[a] = TX::frag(lx1, xrow + 32 * a, h, q);
    }
#pragma unroll
    for (int b = 0; b < WN; ++b) {
      f.y0[b] = TY::frag(ly0, yrow + 32 * b, h, q);
      if (MODE != 0) f.y1[b] = TY::frag(ly1, yrow + 32 * b, h, q);
    }
  };
  auto mma = [&](const Frags& f) {
#pragma unroll
    for (int a = 0; a < WM; ++a)
#pragma unroll
      for (int b = 0; b < WN; ++b) {
        acc0[a][b] = mfma(f.x0[a], f.y0[b], acc0[a][b]);
        if (MODE == 1) {
          acc1[a][b] = mfma(f.x1[a], f.y0[b], acc1[a][b]);
          acc1[a][b] = mfma(f.x0[a], f.y1[b], acc1[a][b]);
        } else if (MODE == 2) {
          acc1[a][b] = mfma(f.x0[a], f.y1[b], acc1[a][b]);
        }
      }
  };
  auto compute = [&](int st) {
    constexpr int NQ = BK / 16;
    Frags fa, fb;
    fetch(fa, st, 0);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if (q + 1 < NQ) fetch((q & 1) ? fa : fb, st, q + 1);
      __builtin_amdgcn_sched_barrier(0);
      mma((q & 1) ? fb : fa);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // bias sums: thread t owns row t % RM of the X tile and part t / RM of
  // its chunks
  constexpr int PARTS = NT / RM > 0 ? NT / RM : 1;
  static_assert(!BIAS || (NT % RM == 0 && TX::CH % PARTS == 0 && PARTS <= 2),
                "bias sum layout");
  const bool do_bias = BIAS && tn == 0 && (e.bias_out || e.bias_part);
  double bsum = 0.0;

  // The staged epilogue's a0 tile ([RM][RN] bf16, 16-byte chunks swizzled
  // as in the staged output tile, so that each output overwrites its own a0
  // in place) arrives by direct loads as well: with two stages, the half of
  // it that covers the stage the last K block leaves free is fetched while
  // that block's MFMAs run, the other half right after them.  Chunks past
  // ldo (only in a last column tile, feeding columns that are not stored)
  // fetch the row's last chunk instead, so that every load stays in the row.
  constexpr int TA = RM * RN;
  constexpr bool A0PF = Epi::NB > 0 && Epi::A0 && S == 2 && TA == S * STAGE;
  const bool a0pf = A0PF && HF_H_STAGE && Epi::staged(e);
  auto a0_half = [&](int half) {
    constexpr int CPR = RN / 8;                      // chunks per tile row
    constexpr int ROWS = RM / 2 / NW;                // rows per wave
    static_assert(!A0PF || (CPR == 32 && ROWS % 2 == 0), "a0 direct-load layout");
    const int kmax = (e.ldo - n0) / 8 - 1;
#pragma unroll
    for (int j = 0; j < ROWS / 2; ++j) {
      const int r = half * (RM / 2) + wave * ROWS + 2 * j + (lane >> 5);
      const int k = min((lane & 31) ^ ((r >> 3) % CPR), kmax);
      dma16(e.a0 + (size_t)(m0 + r) * e.ldo + n0 + 8 * k,
            lds + (half * (RM / 2) + wave * ROWS + 2 * j) * RN);
    }
  };

  // prologue: the first S - 1 blocks in flight
#pragma unroll
  for (int i = 0; i < S - 1; ++i)
    if (i < nblk) issue(vb0 + i, i);
  for (int it = 0; it < nblk; ++it) {
    // this wave's loads of block it have landed once at most
    // min(S - 2, nblk - 1 - it) later blocks are still pending
    // (one unconditional wait, so that the compiler sees every earlier
    // scalar and LDS operation complete on every path)
    const int ahead = min(S - 2, nblk - 1 - it);
    wait_vm<(S - 2) * LPB>();
    if (S > 3 && ahead == 1) wait_vm<(S > 3 ? LPB : 0)>();
    if (ahead == 0) wait_vm<0>();
    stage_barrier();     // every wave's loads landed; stage it - 1 is free
    if (it + S - 1 < nblk) issue(vb0 + it + S - 1, (it + S - 1) % S);
    const int st = it % S;
    if (A0PF && a0pf && it == nblk - 1) a0_half(1 - st);
    compute(st);
    if (BIAS && do_bias && vb0 + it < kbps) {
      const int row = tid % RM, part = tid / RM;
      constexpr int CPP = TX::CH / PARTS;
      const bf16_t* lx0 = lds + st * STAGE;
      float t = 0.0f;
#pragma unroll
      for (int cc = 0; cc < CPP; ++cc) t += TX::chunk_sum(lx0, row, part * CPP + cc);
      bsum += (double)t;
    }
  }
  if (BIAS && do_bias) {
    __shared__ double bpart2[RM];
    if (PARTS == 2 && tid >= RM) bpart2[tid - RM] = bsum;
    __syncthreads();
    if (tid < RM && m0 + tid < s.M) {
      const double t = PARTS == 2 ? bsum + bpart2[tid] : bsum;
      if (s.splits > 1) e.bias_part[(size_t)tz * s.M + m0 + tid] = t;
      else e.bias_out[m0 + tid] = (float)t;
    }
  }

  // 32 x 32 accumulator layout: lane (li, h), register r holds row
  // 8 (r / 4) + 4 h + r % 4, column li of the block; registers 4g .. 4g + 3
  // are 4 consecutive rows.
  const int Mpad = (s.M + 63) & ~63;
  if constexpr (Epi::NB > 0) {
    if (HF_H_STAGE && Epi::staged(e)) {
      // Staged epilogue.  The bf16 outputs pass through LDS (the operand
      // stages are free by now), so that global memory sees 16-byte
      // coalesced loads of a0 and 16-byte coalesced stores of both the
      // row-major and the transposed copy, instead of 2-byte row accesses
      // and scattered 8-byte column stores.  One [RM][RN] bf16 tile per
      // output; the 16-byte chunks of tile row r are XOR-swizzled by
      // (r / 8) % (RN / 8), so that the transposed pass (eight rows of one
      // column per thread) reads without bank conflicts.  a0 is loaded into
      // the first tile and each thread overwrites its own elements with the
      // first output.
      constexpr int T = RM * RN;
      constexpr int CPR = RN / 8;
      static_assert(Epi::NB * T <= S * STAGE, "staged tiles exceed the operand stages");
      static_assert(RM % 64 == 0 && RN % 128 == 0, "staged tile shape");
      static_assert(T / 8 % NT == 0, "staged passes: whole 16-byte chunks per thread");
      constexpr int PASS = T / 8 / NT;               // chunks per thread and pass
      auto lidx = [&](int r, int c) {
        return r * RN + (((c >> 3) ^ ((r >> 3) % CPR)) << 3) + (c & 7);
      };
      __syncthreads();     // every wave is done with the operand stages
      if (A0PF) {
        // the half the last block's stage covered (all of it if the loop
        // had no blocks), then every wave's direct loads landed
        if (nblk > 0) {
          a0_half((nblk - 1) % S);
        } else {
          a0_half(0);
          a0_half(1);
        }
        wait_vm<0>();
        stage_barrier();
      } else if (Epi::A0) {
        // a0 rows exist up to M rounded up to 256; columns past ldo read 0
        u32x4 v[PASS];
#pragma unroll
        for (int p = 0; p < PASS; ++p) {
          const int i = tid + p * NT;
          const int r = i / CPR, k = i % CPR;
          v[p] = u32x4{0u, 0u, 0u, 0u};
          if (n0 + 8 * k + 8 <= e.ldo)
            v[p] = *(const u32x4*)(e.a0 + (size_t)(m0 + r) * e.ldo + n0 + 8 * k);
        }
#pragma unroll
        for (int p = 0; p < PASS; ++p) {
          const int i = tid + p * NT;
          const int r = i / CPR, k = i % CPR;
          *(u32x4*)(lds + r * RN + ((k ^ ((r >> 3) % CPR)) << 3)) = v[p];
        }
        __syncthreads();
      }
#pragma unroll
      for (int a = 0; a < WM; ++a)
#pragma unroll
        for (int b = 0; b < WN; ++b) {
          const int lc = wn * 32 * WN + b * 32 + li;
          const int col = n0 + lc;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int lr0 = wm * 32 * WM + a * 32 + 4 * h + 8 * g;
            const int r0 = m0 + lr0;
            if (col < s.N && r0 < Mpad) {
              Q v0, v1, av, o[Epi::NB];
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                v0.v[j] = acc0[a][b][4 * g + j];
                v1.v[j] = MODE == 0 ? 0.0f : acc1[a][b][4 * g + j];
                av.v[j] = Epi::A0 ? bf2f(lds[lidx(lr0 + j, lc)]) : 0.0f;
              }
              Epi::stage(e, r0, col, s.M, v0, v1, av, o);
#pragma unroll
              for (int i = 0; i < Epi::NB; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) lds[i * T + lidx(lr0 + j, lc)] = f2bf(o[i].v[j]);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < Epi::NB; ++i) {
        bf16_t* hp = Epi::hout(e, i);
        bf16_t* tp = Epi::tout(e, i);
        const bf16_t* tile = lds + i * T;
        // row-major copy: one 16-byte chunk per thread, rows below M,
        // columns below N (a partial last chunk element by element)
#pragma unroll
        for (int p = 0; p < PASS; ++p) {
          const int it = tid + p * NT;
          const int r = it / CPR, k = it % CPR;
          const int grow = m0 + r, gcol = n0 + 8 * k;
          if (grow < s.M && gcol < s.N) {
            const u32x4 v = *(const u32x4*)(tile + r * RN + ((k ^ ((r >> 3) % CPR)) << 3));
            bf16_t* dst = hp + (size_t)grow * e.ldo + gcol;
            if (gcol + 8 <= s.N) {
              *(u32x4*)dst = v;
            } else {
#pragma unroll
              for (int j = 0; j < 8; ++j)
                if (gcol + j < s.N) dst[j] = (bf16_t)(v[j >> 1] >> (16 * (j & 1)));
            }
          }
        }
        // transposed copy (where one is wanted): eight consecutive rows of
        // one column per thread, zeros for rows from M to Mpad; a wave
        // covers 8 columns x 64 rows, 128 contiguous bytes per column
        if (!tp) continue;
#pragma unroll
        for (int p = 0; p < PASS; ++p) {
          const int it = tid + p * NT;
          const int cc = it & 7, r8 = (it >> 3) & 7, grp = it >> 6;
          const int lc = (grp % CPR) * 8 + cc, lr = (grp / CPR) * 64 + r8 * 8;
          const int gcol = n0 + lc, grow = m0 + lr;
          if (gcol < s.N && grow < Mpad) {
            uint32_t w[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const uint32_t lo = grow + 2 * j < s.M ? (uint32_t)tile[lidx(lr + 2 * j, lc)] : 0u;
              const uint32_t hi =
                  grow + 2 * j + 1 < s.M ? (uint32_t)tile[lidx(lr + 2 * j + 1, lc)] : 0u;
              w[j] = lo | (hi << 16);
            }
            *(u32x4*)(tp + (size_t)gcol * e.ldt + grow) = u32x4{w[0], w[1], w[2], w[3]};
          }
        }
      }
      return;
    }
  }
#pragma unroll
  for (int a = 0; a < WM; ++a)
#pragma unroll
    for (int b = 0; b < WN; ++b) {
      const int rbase = m0 + wm * 32 * WM + a * 32 + 4 * h;
      const int col = n0 + wn * 32 * WN + b * 32 + li;
      if (col < s.N) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r0 = rbase + 8 * g;
          if (r0 < Mpad) {
            Q v0, v1;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              v0.v[j] = acc0[a][b][4 * g + j];
              v1.v[j] = MODE == 0 ? 0.0f : acc1[a][b][4 * g + j];
            }
            Epi::apply(e, r0, col, s.M, tz, v0, v1);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
}

// Tile shapes (WM, WN, GM, GN, BK, stages) of the single-product kernels
// and of the dual ones (which hold two accumulator sets and up to four
// tiles).
#ifndef HF_HS_WM
#define HF_HS_WM 4
#endif
#ifndef HF_HS_WN
#define HF_HS_WN 2
#endif
#ifndef HF_HS_GM
#define HF_HS_GM 2
#endif
#ifndef HF_HS_GN
#define HF_HS_GN 4
#endif
#ifndef HF_HS_BK
#define HF_HS_BK 64
#endif
#ifndef HF_HS_S
#define HF_HS_S 2
#endif
#ifndef HF_HD_WM
#define HF_HD_WM 2
#endif
#ifndef HF_HD_WN
#define HF_HD_WN 2
#endif
#ifndef HF_HD_GM
#define HF_HD_GM 2
#endif
#ifndef HF_HD_GN
#define HF_HD_GN 2
#endif
#ifndef HF_HD_BK
#define HF_HD_BK 32
#endif
#ifndef HF_HD_S
#define HF_HD_S 3
#endif
// minimum waves per SIMD the register allocation must allow (workgroups
// resident per CU = OCC * 4 / waves per workgroup)
#ifndef HF_HS_OCC
#define HF_HS_OCC 1
#endif
#ifndef HF_HD_OCC
#define HF_HD_OCC 1
#endif
constexpr int SWM = HF_HS_WM, SWN = HF_HS_WN, SGM = HF_HS_GM, SGN = HF_HS_GN;
constexpr int SBK = HF_HS_BK, SS = HF_HS_S;
constexpr int DWM = HF_HD_WM, DWN = HF_HD_WN, DGM = HF_HD_GM, DGN = HF_HD_GN;
constexpr int DBK = HF_HD_BK, DS = HF_HD_S;
constexpr int SOCC = HF_HS_OCC, DOCC = HF_HD_OCC;
constexpr int SNT = 64 * SGM * SGN, DNT = 64 * DGM * DGN;

}  // namespace

#define HF_HGEMM_KERNEL(NAME, MODE, EPI, BIAS, P)                              \
  extern "C" __global__ __launch_bounds__(P##NT, P##OCC) void NAME(GemmShapeH s, \
                                                              EpiH e) {        \
    hgemm_body<MODE, EPI, BIAS, P##WM, P##WN, P##GM, P##GN, P##BK, P##S>(s, e);  \
  }

HF_HGEMM_KERNEL(hf_hgemm_fwd, 0, EFwd, false, S)
HF_HGEMM_KERNEL(hf_hgemm_fwd_rfwd, 1, EFwdRFwd, false, D)
HF_HGEMM_KERNEL(hf_hgemm_fwd_rfwd0, 2, EFwdRFwd, false, D)
HF_HGEMM_KERNEL(hf_hgemm_rfwd, 0, ERFwd, false, S)
HF_HGEMM_KERNEL(hf_hgemm_bwd, 0, EBwd, false, S)
HF_HGEMM_KERNEL(hf_hgemm_bwd_e2, 0, EBwdE2, false, S)
HF_HGEMM_KERNEL(hf_hgemm_bwd_rbwd, 1, EBwdRBwd, false, D)
HF_HGEMM_KERNEL(hf_hgemm_rbwd, 0, ERBwd, false, S)
HF_HGEMM_KERNEL(hf_hgemm_gnbwd, 0, EGNBwd, false, S)
HF_HGEMM_KERNEL(hf_hgemm_wgrad, 0, EStore, true, S)

// out[r * ldo + c] = bf16(in[r * ldi + c]) for r < R, and outT[c * ldt + r]
// = the same value for r < R, zero for R <= r < Rpad (the K padding a later
// GEMM reads), for c < C; through a padded 32 x 32 LDS tile so that the
// reads and both writes are coalesced.  Either output may be null.
namespace {
__device__ __forceinline__ bf16_t to_bf16(float v) { return f2bf(v); }
__device__ __forceinline__ bf16_t to_bf16(bf16_t v) { return v; }

template <class IN>
__device__ __forceinline__ void cvt_body(
    const IN* __restrict__ in, int R, int C, int ldi, bf16_t* __restrict__ out,
    int ldo, bf16_t* __restrict__ outT, int ldt, int Rpad) {
  __shared__ bf16_t t[32][34];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = r0 + ty + 8 * j, c = c0 + tx;
    bf16_t b = 0;
    if (r < R && c < C) {
      b = to_bf16(in[(size_t)r * ldi + c]);
      if (out) out[(size_t)r * ldo + c] = b;
    }
    t[ty + 8 * j][tx] = b;
  }
  if (!outT) return;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = c0 + ty + 8 * j, r = r0 + tx;
    if (r < Rpad && c < C) outT[(size_t)c * ldt + r] = t[tx][ty + 8 * j];
  }
}

}  // namespace

extern "C" __global__ __launch_bounds__(256) void hf_cvt_bf16(
    const float* __restrict__ in, int R, int C, int ldi, bf16_t* __restrict__ out,
    int ldo, bf16_t* __restrict__ outT, int ldt, int Rpad,
    const int* __restrict__ skip) {
  if (skip && *skip) return;
  cvt_body(in, R, C, ldi, out, ldo, outT, ldt, Rpad);
}

// Row-major copy only, 8 elements per thread and step (two 16-byte loads,
// one 16-byte store); C a multiple of 8, in and out 16-byte aligned, ldi a
// multiple of 4 and ldo of 8.
extern "C" __global__ __launch_bounds__(256) void hf_cvt_bf16_rows(
    const float* __restrict__ in, int R, int C, int ldi, bf16_t* __restrict__ out,
    int ldo, const int* __restrict__ skip) {
  if (skip && *skip) return;
  const int cpr = C >> 3;
  const long long n = (long long)R * cpr;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (long long)gridDim.x * 256) {
    const int r = (int)(i / cpr), c = 8 * (int)(i - (long long)r * cpr);
    const float4 a = *(const float4*)(in + (size_t)r * ldi + c);
    const float4 b = *(const float4*)(in + (size_t)r * ldi + c + 4);
    const uint32_t w0 = (uint32_t)f2bf(a.x) | ((uint32_t)f2bf(a.y) << 16);
    const uint32_t w1 = (uint32_t)f2bf(a.z) | ((uint32_t)f2bf(a.w) << 16);
    const uint32_t w2 = (uint32_t)f2bf(b.x) | ((uint32_t)f2bf(b.y) << 16);
    const uint32_t w3 = (uint32_t)f2bf(b.z) | ((uint32_t)f2bf(b.w) << 16);
    *(uint4*)(out + (size_t)r * ldo + c) = make_uint4(w0, w1, w2, w3);
  }
}

// The transposed copy of a bf16 matrix (zeros in the padding rows) in
// 64 x 64 tiles with 16-byte loads and stores: in and outT 16-byte aligned,
// ldi and ldt multiples of 8, Rpad a multiple of 8.  A thread loads 8
// consecutive columns of a row (element by element past C) and stores 8
// consecutive rows of a column.
extern "C" __global__ __launch_bounds__(256) void hf_transpose_bf16_v(
    const bf16_t* __restrict__ in, int R, int C, int ldi, bf16_t* __restrict__ outT,
    int ldt, int Rpad, const int* __restrict__ skip) {
  if (skip && *skip) return;
  __shared__ __attribute__((aligned(16))) bf16_t t[64][72];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int q = threadIdx.x + 256 * h;
    const int rr = q >> 3, cc = (q & 7) * 8;
    const int r = r0 + rr, c = c0 + cc;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < R) {
      const bf16_t* src = in + (size_t)r * ldi + c;
      if (c + 8 <= C) {
        v = *(const u32x4*)src;
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (c + j < C) v[j >> 1] |= (uint32_t)src[j] << (16 * (j & 1));
      }
    }
    *(u32x4*)&t[rr][cc] = v;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int q = threadIdx.x + 256 * h;
    const int cc = q >> 3, rr = (q & 7) * 8;
    const int c = c0 + cc, r = r0 + rr;
    if (c < C && r < Rpad) {
      u32x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = (uint32_t)t[rr + 2 * j][cc] | ((uint32_t)t[rr + 2 * j + 1][cc] << 16);
      *(u32x4*)(outT + (size_t)c * ldt + r) = w;
    }
  }
}

// the transposed copy of a bf16 matrix (with zeros in the padding rows)
extern "C" __global__ __launch_bounds__(256) void hf_transpose_bf16(
    const bf16_t* __restrict__ in, int R, int C, int ldi, bf16_t* __restrict__ outT,
    int ldt, int Rpad, const int* __restrict__ skip) {
  if (skip && *skip) return;
  cvt_body(in, R, C, ldi, (bf16_t*)nullptr, 0, outT, ldt, Rpad);
}

// p[i] = bf16(p[i]^2) for i < n: squares a bf16 operand in place (the
// Fisher diagonal's squared weight-gradient operands)
extern "C" __global__ __launch_bounds__(256) void hf_square_bf16(
    bf16_t* __restrict__ p, long long n) {
  const long long n8 = n >> 3;
  const long long stride = (long long)gridDim.x * 256;
  const long long t0 = (long long)blockIdx.x * 256 + threadIdx.x;
  for (long long i = t0; i < n8; i += stride) {
    uint4 v = ((const uint4*)p)[i];
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float lo = bf2f((bf16_t)(w[k] & 0xffffu));
      const float hi = bf2f((bf16_t)(w[k] >> 16));
      w[k] = (uint32_t)f2bf(lo * lo) | ((uint32_t)f2bf(hi * hi) << 16);
    }
    ((uint4*)p)[i] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  for (long long e = n8 * 8 + t0; e < n; e += stride) {
    const float f = bf2f(p[e]);
    p[e] = f2bf(f * f);
  }
}

namespace {

typedef void (*HKernel)(GemmShapeH, EpiH);
inline int cdiv(int a, int b) { return (a + b - 1) / b; }

void launch(const Launch& L, const char* name, HKernel k, int mode,
            const GemmShapeH& s, const EpiH& e, double flops, double bytes) {
  const bool sg = mode == 0;
  const int rm = 32 * (sg ? SWM * SGM : DWM * DGM);
  const int rn = 32 * (sg ? SWN * SGN : DWN * DGN);
  dim3 grid(cdiv(s.N, rn), cdiv(s.M, rm), (sg && s.splits > 1) ? s.splits : 1);
  prof_begin(L, name);
  hipExtLaunchKernelGGL(k, grid, dim3(sg ? SNT : DNT), 0, L.stream, prof_a(L), prof_b(L), 0, s, e);
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
  // hidden layer: A row-major and transposed, RA row-major, RZ and the
  // transposed RA where wanted; output layer: logits and RZ
  const double out = e.hidden ? 6.0 + (e.f1 ? 4.0 : 0.0) + (e.t2 ? 2.0 : 0.0) : 8.0;
  if (s.X[1])
    launch(L, "hf_hgemm_fwd_rfwd", hf_hgemm_fwd_rfwd, 1, s, e, 3 * mnk(s), io(s, 2, 2, out));
  else
    launch(L, "hf_hgemm_fwd_rfwd0", hf_hgemm_fwd_rfwd0, 2, s, e, 2 * mnk(s), io(s, 1, 2, out));
}
void hgemm_rfwd(const Launch& L, const GemmShapeH& s, const EpiH& e) {
  // hidden layer: a0 read, RA stored row-major, RZ and the transposed RA
  // where wanted; output layer: RZ
  const double out = e.hidden ? 4.0 + (e.f1 ? 4.0 : 0.0) + (e.t2 ? 2.0 : 0.0) : 4.0;
  launch(L, "hf_hgemm_rfwd", hf_hgemm_rfwd, 0, s, e, mnk(s) * s.nseg,
         io(s, s.nseg, s.nseg, out));
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
void square_bf16(const Launch& L, bf16_t* p, long long n) {
  if (n <= 0) return;
  const long long nb = std::min<long long>((n + 8 * 256 - 1) / (8 * 256), 2048);
  prof_begin(L, "hf_square_bf16");
  hipExtLaunchKernelGGL(hf_square_bf16, dim3((unsigned)nb), dim3(256), 0, L.stream,
                        prof_a(L), prof_b(L), 0, p, n);
  prof_end(L, "hf_square_bf16", 0.0, 4.0 * n);
}
void transpose_bf16(const Launch& L, const bf16_t* in, int R, int C, int ldi,
                    bf16_t* outT, int ldt, int Rpad, const int* skip) {
  if (Rpad < R) Rpad = R;
  if (ldi % 8 == 0 && ldt % 8 == 0 && Rpad % 8 == 0 && ((uintptr_t)in & 15u) == 0 &&
      ((uintptr_t)outT & 15u) == 0) {
    prof_begin(L, "hf_transpose_bf16");
    hipExtLaunchKernelGGL(hf_transpose_bf16_v, dim3(cdiv(C, 64), cdiv(Rpad, 64)), dim3(256), 0,
                          L.stream, prof_a(L), prof_b(L), 0, in, R, C, ldi, outT, ldt, Rpad,
                          skip);
    prof_end(L, "hf_transpose_bf16", 0.0, 4.0 * (double)R * C);
    return;
  }
  prof_begin(L, "hf_transpose_bf16");
  hipExtLaunchKernelGGL(hf_transpose_bf16, dim3(cdiv(C, 32), cdiv(Rpad, 32)), dim3(256), 0,
                        L.stream, prof_a(L), prof_b(L), 0, in, R, C, ldi, outT, ldt, Rpad, skip);
  prof_end(L, "hf_transpose_bf16", 0.0, 4.0 * (double)R * C);
}
void cvt_bf16(const Launch& L, const float* in, int R, int C, int ldi,
              bf16_t* out, int ldo, bf16_t* outT, int ldt, int Rpad,
              const int* skip) {
  if (out && !outT && C % 8 == 0 && ldi % 4 == 0 && ldo % 8 == 0 &&
      ((uintptr_t)in & 15u) == 0 && ((uintptr_t)out & 15u) == 0) {
    const long long n = (long long)R * (C / 8);
    const long long nb = std::min<long long>((n + 255) / 256, 2048);
    if (nb < 1) return;
    prof_begin(L, "hf_cvt_bf16");
    hipExtLaunchKernelGGL(hf_cvt_bf16_rows, dim3((unsigned)nb), dim3(256), 0, L.stream,
                          prof_a(L), prof_b(L), 0, in, R, C, ldi, out, ldo, skip);
    prof_end(L, "hf_cvt_bf16", 0.0, 6.0 * (double)R * C);
    return;
  }
  if (Rpad < R) Rpad = R;
  prof_begin(L, "hf_cvt_bf16");
  hipExtLaunchKernelGGL(hf_cvt_bf16, dim3(cdiv(C, 32), cdiv(Rpad, 32)), dim3(256), 0,
                     L.stream, prof_a(L), prof_b(L), 0, in, R, C, ldi, out, ldo, outT, ldt, Rpad, skip);
  prof_end(L, "hf_cvt_bf16", 0.0,
           (double)R * C * (4.0 + (out ? 2.0 : 0.0) + (outT ? 2.0 : 0.0)));
}

}  // namespace hfk
