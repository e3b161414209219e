// Device scratch of the entry point that allocates nothing (hf_hvp_noalloc).
//
// The array below is the workspace of that entry point: one per GPU, held
// for the life of the process, shared by every call on that GPU.  In host
// code its name is only a host-side stand-in; the device address is looked
// up once per device with hipGetSymbolAddress (with that device current)
// and every host use goes through that address.
#include "hf.h"
#include "hf_internal.h"

#include <mutex>

static __device__ __align__(256) unsigned char scratch[HF_NOALLOC_SCRATCH_BYTES];

namespace hfk {

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void* g_ptr[MAX_DEVICES] = {};

__global__ __launch_bounds__(256) void hf_fill_zero(uint32_t* __restrict__ p,
                                                    long long words) {
  const long long stride = (long long)gridDim.x * 256;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < words; i += stride)
    p[i] = 0u;
}

}  // namespace

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

// Zero `bytes` (a multiple of 4) at p with a kernel (no memset node, so the
// call can be captured into a graph).
void fill_zero(const Launch& L, void* p, size_t bytes) {
  const long long words = (long long)(bytes / 4);
  if (words <= 0) return;
  long long blocks = (words + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(hf_fill_zero, dim3((unsigned)blocks), dim3(256), 0, L.stream,
                     reinterpret_cast<uint32_t*>(p), words);
}

}  // namespace hfk
