// Streaming-read probe (instrumentation, not part of the attention path): reads a device buffer
// once with 16-byte non-temporal loads -- the load the decode and pack kernels use for data they
// read exactly once -- so a benchmark can log what HBM reading reaches on the part it runs on,
// beside the 8 TB/s specification the roofline fractions are quoted against.
#include "device_common.hpp"
#include "kernels.hpp"

namespace cs {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;

// Thread t of the grid reads 16-byte chunks t, t + T, t + 2T, ... (T = grid threads), eight
// independent loads in flight per iteration, and folds them with XOR; the fold is stored only if
// it equals a fixed value, so the loads stay live while (almost) nothing is written.
__global__ __launch_bounds__(kProbeThreads) void stream_read_probe_kernel(const uint4* __restrict__ src,
                                                                          size_t n16, uint32_t* sink) {
  const size_t T = static_cast<size_t>(gridDim.x) * kProbeThreads;
  size_t i = static_cast<size_t>(blockIdx.x) * kProbeThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kProbeUnroll - 1) * T < n16; i += kProbeUnroll * T) {
    uint4 x[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) x[u] = ld16_nt(src + i + u * T);
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= x[u].x ^ x[u].y ^ x[u].z ^ x[u].w;
  }
  for (; i < n16; i += T) {
    const uint4 x = ld16_nt(src + i);
    acc ^= x.x ^ x.y ^ x.z ^ x.w;
  }
  if (acc == 0x9E3779B9u) sink[0] = acc;
}

hipError_t launch_stream_read_probe(const void* src, size_t bytes, uint32_t* sink, int n_cus,
                                    hipStream_t stream) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  const int blocks = 8 * n_cus;     // 8 workgroups of 4 waves per CU
  stream_read_probe_kernel<<<blocks, kProbeThreads, 0, stream>>>(static_cast<const uint4*>(src), n16, sink);
  return hipGetLastError();
}

}  // namespace cs
