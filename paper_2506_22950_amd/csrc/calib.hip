// Measurement helper, not part of the decode path: the read-bandwidth ceiling
// of a single launch on this GPU, for comparison with the decode kernel's
// achieved bytes per launch.
//
// Each work-group streams one contiguous span of the buffer with 16-byte
// loads, kUnroll of them in flight per lane, and folds every loaded word into
// one value so that no load can be dropped.  Nothing is written unless the
// fold equals a sentinel, so the launch moves only the bytes it reads.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

__global__ __launch_bounds__(kThreads) void stream_read(const u32x4* __restrict__ buf, int64_t vec_per_block,
                                                        uint32_t* sink) {
  const u32x4* p = buf + blockIdx.x * vec_per_block;
  uint32_t acc = 0;
  for (int64_t i = threadIdx.x; i < vec_per_block; i += (int64_t)kThreads * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t j = i + (int64_t)u * kThreads;
      v[u] = j < vec_per_block ? p[j] : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

}  // namespace

// Read `bytes` from `buf` (device memory, 16-byte aligned) in one launch of
// `blocks` work-groups on `stream` (a hipStream_t; null: the default stream).
// bytes must be a positive multiple of 16 * blocks; `sink` (device, >= blocks
// uint32) is written only in the unlikely case described above.  Returns the
// hipError_t of the launch (hipErrorInvalidValue for bad arguments).
extern "C" int infs_calib_stream_read(const void* buf, int64_t bytes, int32_t blocks, void* stream, uint32_t* sink) {
  if (!buf || !sink || blocks <= 0 || bytes <= 0 || bytes % (16 * (int64_t)blocks) != 0 ||
      ((uintptr_t)buf & 15) != 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(stream_read, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream, (const u32x4*)buf,
                     bytes / 16 / blocks, sink);
  return (int)hipGetLastError();
}
