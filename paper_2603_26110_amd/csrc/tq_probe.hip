// Streaming read of a device buffer: a measurement of the HBM read rate a
// transfer of a given size reaches on this GPU, for comparison with the
// kernels of the method (which read the same number of bytes). Not part of
// the method.
//
// Each thread keeps four 16-byte loads in flight per grid-stride step and
// folds them into a register; a block stores its word only if it equals a
// constant that stands for "never", which keeps the loads.
#include "tq_internal.hpp"

namespace tq {

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 4;

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const uint4* p, int64_t n16, uint32_t* sink) {
  uint32_t acc = 0;
  const int64_t step = (int64_t)gridDim.x * kProbeThreads * kProbeUnroll;
  for (int64_t i = (int64_t)blockIdx.x * kProbeThreads * kProbeUnroll + threadIdx.x; i < n16; i += step) {
    uint4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t k = i + (int64_t)u * kProbeThreads;
      v[u] = k < n16 ? p[k] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
}

}  // namespace

hipError_t launch_read_probe(const void* data, int64_t bytes, int blocks, uint32_t* sink, hipStream_t st) {
  hipLaunchKernelGGL(read_probe_kernel, dim3((unsigned)blocks), dim3(kProbeThreads), 0, st,
                     reinterpret_cast<const uint4*>(data), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace tq
