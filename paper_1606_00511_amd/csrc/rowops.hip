// Output-layer and reduction kernels that sit between the GEMMs.
//
// softmax_xent: the softmax cross-entropy objective averaged over the batch
//   (the f whose gradient Alg. 1 takes), its output-layer error
//   delta_L = (p - e_y) / B and the probabilities p kept for the curvature
//   products.
// softmax_rop:  the output-layer factor of both curvature products, the
//   Hessian of the batch-mean cross-entropy with respect to the logits applied
//   to R{z}: (diag p - p p^T) R{z} / B per row (Sec. 2.1, after Alg. 1).
// splitk_reduce: deterministic fixed-order reduction of split-K partials of
//   the weight gradients and of their bias sums (one kernel per split count).
//
// One wave64 per row, held in registers (the values of columns lane, lane +
// 64, ...); row reductions use wave shuffles.  Every sum runs in a fixed order, so repeated calls give
// bit-identical results.
#include <algorithm>
#include <type_traits>

#include "hf_internal.h"


namespace hfk {
namespace {

constexpr int ROWS_PER_BLOCK = 4;   // 4 waves, one row each

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
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


// softmax_xent keeps its row of logits in registers (KMAX per lane,
// C <= 64 KMAX), as softmax_rop does; the sums run in the same order as a
// column-order pass per lane followed by the wave reduction.
template <int KMAX>
__device__ __forceinline__ void softmax_xent_body(
    const float* __restrict__ Z, const int32_t* __restrict__ y, int B, int C,
    int ld, float invB, float* __restrict__ P, float* __restrict__ D,
    double* __restrict__ loss_part, int* __restrict__ err) {
  __shared__ float wl[ROWS_PER_BLOCK];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * ROWS_PER_BLOCK + wave;
  float li = 0.0f;
  if (row < B) {
    const float* z = Z + (size_t)row * ld;
    float v[KMAX];
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const int c = lane + 64 * k;
      v[k] = c < C ? z[c] : -INFINITY;
      m = fmaxf(m, v[k]);
    }
    m = wave_max(m);
    float sum = 0.0f;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      if (lane + 64 * k < C) {
        v[k] = expf(v[k] - m);
        sum += v[k];
      }
    }
    sum = wave_sum(sum);
    const float inv = 1.0f / sum;
    int yi = -1;
    if (y) {
      yi = y[row];
      if (yi < 0 || yi >= C) {
        if (lane == 0) *err = 1;
        yi = -1;
      }
    }
    float* prow = P + (size_t)row * ld;
    float* drow = D ? D + (size_t)row * ld : nullptr;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const int c = lane + 64 * k;
      if (c < C) {
        const float p = v[k] * inv;
        prow[c] = p;
        if (drow) drow[c] = (c == yi ? p - 1.0f : p) * invB;
      }
    }
    if (yi >= 0) li = (m + logf(sum)) - z[yi];
  }
  if (lane == 0) wl[wave] = li;
  __syncthreads();
  if (threadIdx.x == 0 && loss_part)
    loss_part[blockIdx.x] = ((double)wl[0] + (double)wl[1]) +
                            ((double)wl[2] + (double)wl[3]);
}

#define HF_SOFTMAX_XENT(K)                                                      \
  extern "C" __global__ __launch_bounds__(256) void hf_softmax_xent_k##K(       \
      const float* __restrict__ Z, const int32_t* __restrict__ y, int B, int C, \
      int ld, float invB, float* __restrict__ P, float* __restrict__ D,         \
      double* __restrict__ loss_part, int* __restrict__ err) {                  \
    softmax_xent_body<K>(Z, y, B, C, ld, invB, P, D, loss_part, err);           \
  }
HF_SOFTMAX_XENT(4)
HF_SOFTMAX_XENT(8)
HF_SOFTMAX_XENT(16)
HF_SOFTMAX_XENT(32)
HF_SOFTMAX_XENT(64)

extern "C" __global__ __launch_bounds__(256) void hf_loss_finalize(
    const double* __restrict__ part, int nparts, double invB,
    float* __restrict__ loss, double* __restrict__ loss64) {
  __shared__ double ws[4];
  double s = 0.0;
  for (int i = threadIdx.x; i < nparts; i += 256) s += part[i];
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double f = ((ws[0] + ws[1]) + (ws[2] + ws[3])) * invB;
    if (loss) *loss = (float)f;
    if (loss64) *loss64 = f;
  }
}

// softmax_rop keeps its row in registers, KMAX values of P and of RZ per
// lane (C <= 64 KMAX), instead of staging it in LDS: the LDS rows of four
// waves (2 x 4 x C floats) allowed only two blocks per compute unit, too few
// waves in flight to cover the memory latency of this HBM-bound pass.  The
// row sum runs in the same order as before (each lane's values in column
// order, then the wave reduction).
// OUT: float, or bf16_t (the bf16-operand products' row-major copy, rounded
// to nearest even once from the same fp32 value)
template <int KMAX, class OUT>
__device__ __forceinline__ void softmax_rop_body(
    const float* __restrict__ P, const float* __restrict__ RZ, int B, int C,
    int ld, float invB, OUT* __restrict__ RD, int ldo) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * ROWS_PER_BLOCK + wave;
  if (row >= B) return;
  const float* prow = P + (size_t)row * ld;
  const float* rrow = RZ + (size_t)row * ld;
  float p[KMAX], r[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int c = lane + 64 * k;
    p[k] = c < C ? prow[c] : 0.0f;
    r[k] = c < C ? rrow[c] : 0.0f;
  }
  float dot = 0.0f;
#pragma unroll
  for (int k = 0; k < KMAX; ++k)
    if (lane + 64 * k < C) dot += p[k] * r[k];
  dot = wave_sum(dot);
  OUT* out = RD + (size_t)row * ldo;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int c = lane + 64 * k;
    if (c < C) {
      const float v = p[k] * (r[k] - dot) * invB;
      if constexpr (std::is_same<OUT, float>::value) out[c] = v;
      else out[c] = __builtin_bit_cast(uint16_t, (__bf16)v);
    }
  }
}

#define HF_SOFTMAX_ROP(K)                                                       \
  extern "C" __global__ __launch_bounds__(256) void hf_softmax_rop_k##K(        \
      const float* __restrict__ P, const float* __restrict__ RZ, int B, int C,  \
      int ld, float invB, float* __restrict__ RD, const int* __restrict__ skip) { \
    if (skip && *skip) return;                                                  \
    softmax_rop_body<K, float>(P, RZ, B, C, ld, invB, RD, ld);                  \
  }                                                                             \
  extern "C" __global__ __launch_bounds__(256) void hf_softmax_rop_h_k##K(      \
      const float* __restrict__ P, const float* __restrict__ RZ, int B, int C,  \
      int ld, float invB, bf16_t* __restrict__ RD, int ldo,                     \
      const int* __restrict__ skip) {                                           \
    if (skip && *skip) return;                                                  \
    softmax_rop_body<K, bf16_t>(P, RZ, B, C, ld, invB, RD, ldo);                \
  }
HF_SOFTMAX_ROP(4)
HF_SOFTMAX_ROP(8)
HF_SOFTMAX_ROP(16)
HF_SOFTMAX_ROP(32)
HF_SOFTMAX_ROP(64)

// Split-K partials of a weight gradient summed in split order (fp64), and
// the bias partials likewise.  SP is a template constant so that every
// partial load of an element is issued before the first add.
template <int SP>
__device__ __forceinline__ void splitk_reduce_body(
    const float* __restrict__ part, const double* __restrict__ bpart, int M,
    int N, float* __restrict__ out, int ldo, float* __restrict__ bout, int vec4,
    const int* __restrict__ skip) {
  if (skip && *skip) return;
  const size_t mn = (size_t)M * N;
  if (bpart) {
    for (int m = blockIdx.x * 256 + threadIdx.x; m < M; m += gridDim.x * 256) {
      double b[SP];
#pragma unroll
      for (int z = 0; z < SP; ++z) b[z] = bpart[(size_t)z * M + m];
      double t = 0.0;
#pragma unroll
      for (int z = 0; z < SP; ++z) t += b[z];
      bout[m] = (float)t;
    }
  }
  if (vec4) {
    // four consecutive elements of one row per thread: 16-byte loads of
    // every partial and one 16-byte store (N, ldo multiples of 4, out
    // 16-byte aligned)
    typedef float f4 __attribute__((ext_vector_type(4)));
    const size_t mn4 = mn / 4;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < mn4;
         i += (size_t)gridDim.x * 256) {
      f4 v[SP];
#pragma unroll
      for (int z = 0; z < SP; ++z) v[z] = ((const f4*)part)[(size_t)z * mn4 + i];
      double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
#pragma unroll
      for (int z = 0; z < SP; ++z) {
        s0 += v[z][0]; s1 += v[z][1]; s2 += v[z][2]; s3 += v[z][3];
      }
      const size_t m = 4 * i / N, n = 4 * i - m * N;
      *(f4*)(out + m * ldo + n) = f4{(float)s0, (float)s1, (float)s2, (float)s3};
    }
    return;
  }
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < mn;
       i += (size_t)gridDim.x * 256) {
    float v[SP];
#pragma unroll
    for (int z = 0; z < SP; ++z) v[z] = part[(size_t)z * mn + i];
    double s = 0.0;
#pragma unroll
    for (int z = 0; z < SP; ++z) s += v[z];
    const size_t m = i / N, n = i - m * N;
    out[m * ldo + n] = (float)s;
  }
}

#define HF_SPLITK_REDUCE(SP)                                                  \
  extern "C" __global__ __launch_bounds__(256) void hf_splitk_reduce_##SP(    \
      const float* __restrict__ part, const double* __restrict__ bpart,      \
      int M, int N, float* __restrict__ out, int ldo,                        \
      float* __restrict__ bout, int vec4, const int* __restrict__ skip) {    \
    splitk_reduce_body<SP>(part, bpart, M, N, out, ldo, bout, vec4, skip);   \
  }
HF_SPLITK_REDUCE(2)
HF_SPLITK_REDUCE(4)
HF_SPLITK_REDUCE(8)
HF_SPLITK_REDUCE(16)
HF_SPLITK_REDUCE(32)

// Block z of the batch: out[c * ldo + r] = in[r * ldi + c] for r < R,
// c < C, through a padded 32 x 32 LDS tile so both the reads and the writes
// are coalesced.  The grid covers the largest block; workgroups past a
// smaller block's edge return at once.
extern "C" __global__ __launch_bounds__(256) void hf_transpose(
    TransposeBatch b, const int* __restrict__ skip) {
  if (skip && *skip) return;
  const int z = blockIdx.z;
  const int R = b.R[z], C = b.C[z];
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  if (r0 >= R || c0 >= C) return;
  const float* __restrict__ in = b.in[z];
  float* __restrict__ out = b.out[z];
  const int ldi = b.ldi[z], ldo = b.ldo[z];
  __shared__ float t[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = r0 + ty + 8 * j, c = c0 + tx;
    if (r < R && c < C) t[ty + 8 * j][tx] = in[(size_t)r * ldi + c];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = c0 + ty + 8 * j, r = r0 + tx;
    if (r < R && c < C) out[(size_t)c * ldo + r] = t[tx][ty + 8 * j];
  }
}

// ------------------------------------------------------------- launchers
void softmax_xent(const Launch& L, const float* Z, const int32_t* y, int B,
                  int C, int ld, float* P, float* D, double* loss_part,
                  int* err_flag) {
  const int blocks = (B + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK;
  typedef void (*K)(const float*, const int32_t*, int, int, int, float, float*,
                    float*, double*, int*);
  // C <= HF_MAX_CLASSES = 64 x 64 (checked by hf_create)
  const K k = C <= 256 ? hf_softmax_xent_k4 : C <= 512 ? hf_softmax_xent_k8
            : C <= 1024 ? hf_softmax_xent_k16 : C <= 2048 ? hf_softmax_xent_k32
            : hf_softmax_xent_k64;
  prof_begin(L, "hf_softmax_xent");
  hipExtLaunchKernelGGL(k, dim3(blocks), dim3(256), 0, L.stream, prof_a(L), prof_b(L), 0,
                     Z, y, B, C, ld, 1.0f / (float)B, P, D, loss_part, err_flag);
  prof_end(L, "hf_softmax_xent", 0.0,
           4.0 * B * C * (D ? 3.0 : 2.0) + (y ? 4.0 * B : 0.0));
}

void loss_finalize(const Launch& L, const double* loss_part, int nparts,
                   int B, float* loss, double* loss64) {
  prof_begin(L, "hf_loss_finalize");
  hipExtLaunchKernelGGL(hf_loss_finalize, dim3(1), dim3(256), 0, L.stream, prof_a(L), prof_b(L), 0,
                     loss_part, nparts, 1.0 / (double)B, loss, loss64);
  prof_end(L, "hf_loss_finalize", 0.0, 8.0 * nparts);
}

void softmax_rop(const Launch& L, const float* P, const float* RZ, int B,
                 int C, int ld, float* RD, const int* skip) {
  const int blocks = (B + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK;
  typedef void (*K)(const float*, const float*, int, int, int, float, float*,
                    const int*);
  // C <= HF_MAX_CLASSES = 64 x 64 (checked by hf_create)
  const K k = C <= 256 ? hf_softmax_rop_k4 : C <= 512 ? hf_softmax_rop_k8
            : C <= 1024 ? hf_softmax_rop_k16 : C <= 2048 ? hf_softmax_rop_k32
            : hf_softmax_rop_k64;
  prof_begin(L, "hf_softmax_rop");
  hipExtLaunchKernelGGL(k, dim3(blocks), dim3(256), 0, L.stream, prof_a(L), prof_b(L), 0, P, RZ, B, C, ld,
                     1.0f / (float)B, RD, skip);
  prof_end(L, "hf_softmax_rop", 0.0, 12.0 * B * C);
}

void softmax_rop_h(const Launch& L, const float* P, const float* RZ, int B,
                   int C, int ld, bf16_t* RD, int ldo, const int* skip) {
  const int blocks = (B + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK;
  typedef void (*K)(const float*, const float*, int, int, int, float, bf16_t*, int,
                    const int*);
  const K k = C <= 256 ? hf_softmax_rop_h_k4 : C <= 512 ? hf_softmax_rop_h_k8
            : C <= 1024 ? hf_softmax_rop_h_k16 : C <= 2048 ? hf_softmax_rop_h_k32
            : hf_softmax_rop_h_k64;
  prof_begin(L, "hf_softmax_rop");
  hipExtLaunchKernelGGL(k, dim3(blocks), dim3(256), 0, L.stream, prof_a(L), prof_b(L), 0, P, RZ, B, C, ld,
                     1.0f / (float)B, RD, ldo, skip);
  prof_end(L, "hf_softmax_rop", 0.0, 10.0 * B * C);
}

void transpose_batch(const Launch& L, const TransposeBatch& b, const int* skip) {
  int gx = 0, gy = 0;
  double bytes = 0.0;
  for (int i = 0; i < b.n; ++i) {
    gx = std::max(gx, (b.C[i] + 31) / 32);
    gy = std::max(gy, (b.R[i] + 31) / 32);
    bytes += 8.0 * b.R[i] * (double)b.C[i];
  }
  if (b.n < 1 || gx < 1 || gy < 1) return;
  prof_begin(L, "hf_transpose");
  hipExtLaunchKernelGGL(hf_transpose, dim3(gx, gy, b.n), dim3(256), 0, L.stream,
                        prof_a(L), prof_b(L), 0, b, skip);
  prof_end(L, "hf_transpose", 0.0, bytes);
}

void splitk_reduce(const Launch& L, const float* part, const double* bpart,
                   int splits, int M, int N, float* out, int ldo, float* bout,
                   const int* skip) {
  const long long mn = (long long)M * N;
  // the split scratch is 256-byte aligned, so every partial starts 16-byte
  // aligned when N is a multiple of 4
  const int vec4 = (N % 4 == 0) && (ldo % 4 == 0) && (((uintptr_t)out & 15) == 0) &&
                   (((uintptr_t)part & 15) == 0);
  long long blocks = ((vec4 ? mn / 4 : mn) + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  // splits is a power of two from 2 to 32 (the split rules double from 1)
  void (*k)(const float*, const double*, int, int, float*, int, float*, int, const int*) =
      splits == 2 ? hf_splitk_reduce_2 : splits == 4 ? hf_splitk_reduce_4
      : splits == 8 ? hf_splitk_reduce_8 : splits == 16 ? hf_splitk_reduce_16
      : hf_splitk_reduce_32;
  prof_begin(L, "hf_splitk_reduce");
  hipExtLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(256), 0,
                        L.stream, prof_a(L), prof_b(L), 0, part, bpart, M, N, out, ldo, bout, vec4, skip);
  prof_end(L, "hf_splitk_reduce", 0.0, 4.0 * mn * (splits + 1));
}

}  // namespace hfk
