// Streaming-read probe (measurement helper, not part of the method): the rate
// at which the device streams a large buffer it reads once, the yardstick of
// the bandwidth-bound decode kernels.  Each lane keeps eight 16-byte
// non-temporal loads in flight (a grid-strided walk), folds the words it read
// into one, and stores it only if it equals a magic value, so no load can be
// dropped and almost nothing is written.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace tactic {

constexpr uint32_t kProbeMagic = 0x9e3779b9u;

__global__ __launch_bounds__(256) void stream_read_kernel(const uint4* buf, int64_t n16, uint32_t* sink) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t x = 0;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  constexpr int kU = 8;
  for (; i + (kU - 1) * stride < n16; i += kU * stride) {
    u32x4 v[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) v[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(buf + i + k * stride));
#pragma unroll
    for (int k = 0; k < kU; ++k) x ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(buf + i));
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (x == kProbeMagic) sink[0] = x;
}

hipError_t launch_stream_read(const void* buf, int64_t n16, int workgroups, uint32_t* sink, hipStream_t st) {
  int64_t blocks = workgroups;
  if (blocks <= 0) {  // the device's resident capacity
    int dev = 0, cus = 0, per = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, stream_read_kernel, 256, 0);
    if (e != hipSuccess) return e;
    blocks = (int64_t)std::max(per, 1) * std::max(cus, 1);
  }
  blocks = std::min<int64_t>(blocks, (n16 + 255) / 256);
  hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(256), 0, st,
                     reinterpret_cast<const uint4*>(buf), n16, sink);
  return hipGetLastError();
}

}  // namespace tactic
