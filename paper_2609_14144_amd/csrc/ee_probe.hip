// Streaming-read probe: the HBM read bandwidth a plain kernel reaches on this
// device, the ceiling the decode path's achieved bandwidth is compared with.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ee {

// Workgroup b reads the contiguous range [b n / G, (b+1) n / G) of 16-byte
// words (G workgroups): its threads stride through the range with U loads in
// flight each and fold the words into one. The word is stored only when it
// equals `key`, so the loads cannot be dropped and nothing is written in
// practice. (Contiguous ranges per workgroup, as the decode phases stream
// their rows; a grid-stride loop, which scatters every wave's loads over the
// whole buffer, reads about 15% slower.)
template <int U>
__global__ __launch_bounds__(256) void k_stream_read(const uint4* __restrict__ p, int64_t n, uint32_t key,
                                                     uint32_t* sink) {
  const int64_t b0 = n * blockIdx.x / gridDim.x, b1 = n * (blockIdx.x + 1) / gridDim.x;
  const int64_t stride = blockDim.x;
  int64_t i = b0 + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + (U - 1) * stride < b1; i += U * stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = p[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < b1; i += stride) {
    const uint4 a = p[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == key) sink[0] = acc;
}

// n 16-byte words at p; eight 256-thread workgroups per compute unit, eight
// loads in flight per thread (the fastest of 1-8 workgroups per unit and 4, 8
// or 16 loads: about 6.3e12 B/s over 2 GiB)
hipError_t launch_stream_read(const void* p, int64_t n, int n_cu, uint32_t* sink, hipStream_t s) {
  hipLaunchKernelGGL(k_stream_read<8>, dim3(8 * n_cu), dim3(256), 0, s, static_cast<const uint4*>(p), n,
                     0x9e3779b9u, sink);
  return hipGetLastError();
}

}  // namespace ee
