// Hidden-unit activations phi and their derivatives, the latter written in
// terms of the stored activation a = phi(z) (so a backward pass needs only
// A_l): sigmoid phi' = a(1 - a), phi'' = a(1 - a)(1 - 2a); tanh phi' = 1 - a^2,
// phi'' = -2a(1 - a^2); ReLU phi' = 1[a > 0], phi'' = 0.  Shared by the fp32
// and the bf16-input GEMM epilogues.
#pragma once

#include "hf_internal.h"

namespace hfk {

__device__ __forceinline__ float act_f(int act, float z) {
  if (act == ACT_SIGMOID) return 1.0f / (1.0f + expf(-z));
  if (act == ACT_TANH) return tanhf(z);
  return fmaxf(z, 0.0f);
}
// selects rather than branches keep the epilogue loops straight-line so the
// accumulators stay in registers
__device__ __forceinline__ float act_d1(int act, float a) {
  const float sg = a * (1.0f - a);
  const float th = 1.0f - a * a;
  const float rl = a > 0.0f ? 1.0f : 0.0f;
  return act == ACT_SIGMOID ? sg : (act == ACT_TANH ? th : rl);
}
__device__ __forceinline__ float act_d2(int act, float a) {
  const float sg = a * (1.0f - a) * (1.0f - 2.0f * a);
  const float th = -2.0f * a * (1.0f - a * a);
  return act == ACT_SIGMOID ? sg : (act == ACT_TANH ? th : 0.0f);
}

}  // namespace hfk
