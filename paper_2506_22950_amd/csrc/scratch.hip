// Static device scratch for the allocation-free decode entry point
// (infs_decode_step_static): the split-K workspace and the arrival counters of
// a decode launch live in one file-scope device array instead of memory that
// infs_create allocates.
//
// Each GPU holds its own copy of `scratch` at its own address, for the life of
// the process.  Host code never uses the array's name as an address (on the
// host it is only a stand-in symbol): the device address is looked up once per
// device with hipGetSymbolAddress, with that device current, and kept in a
// per-device table; kernels receive that address as an argument.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace infs {
namespace {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Zero n 32-bit words (grid-stride).  A kernel rather than hipMemsetAsync, so
// that the clear is an ordinary kernel node when a caller captures the stream.
__global__ __launch_bounds__(256) void zero_words_kernel(uint32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

hipError_t static_scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_zero_words(uint32_t* p, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

}  // namespace infs
