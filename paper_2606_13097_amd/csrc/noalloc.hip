// Static device scratch of fcg_decode_noalloc, the decode entry point that
// allocates nothing: the split partials and arrival counters of its launches
// live in one file-scope device array instead of memory the cache allocates.
//
// In host code the array's name is a host-side stand-in, not a device address;
// its device address is taken once per device with hipGetSymbolAddress (with
// that device current) and kept, and only that address is handed to kernels.
// Every call on a device shares the device's copy, so calls that overlap on
// one GPU race; each launch leaves the counters at zero.
#include <mutex>

#include "kernels.hpp"

namespace fcg {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, null until set up
std::mutex g_mu;

__global__ void __launch_bounds__(256) zero_words_kernel(int32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

int noalloc_scratch(hipStream_t s, void** base) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    // the arrival counters must start at zero (a fill kernel, not a memset, so
    // that a caller may capture this first call in a graph)
    const int n = (int)(kNoAllocCountBytes / sizeof(int32_t));
    hipLaunchKernelGGL(zero_words_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (int32_t*)p, n);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    g_scratch[dev] = p;
  }
  *base = g_scratch[dev];
  return 0;
}

}  // namespace fcg
