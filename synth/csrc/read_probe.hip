// Streaming-read probe for the benchmark: reads a device buffer once with
// 16-byte loads (grid-stride, UNROLL loads in flight per thread) and folds
// the words into one value per workgroup, so that the achievable HBM read
// rate of the part can be measured next to the kernels.  It holds no
// arithmetic of the quantization method.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

template <int UNROLL>
__global__ __launch_bounds__(256) void read_probe_kernel(const uint4* __restrict__ p, int64_t n16,
                                                         uint32_t* __restrict__ sink) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  uint32_t acc = 0;
  int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  for (; i + (UNROLL - 1) * stride < n16; i += UNROLL * stride) {
    uint4 v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) v[u] = p[i + u * stride];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const uint4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  // one word per workgroup (lane 0's fold of its own loads is enough to keep them)
  if (threadIdx.x == 0) sink[blockIdx.x] = acc;
}

}  // namespace

// Reads n16 16-byte words at p_dev with `blocks` workgroups of 256 threads and
// `unroll` (1, 2, 4 or 8) loads in flight per thread; sink_dev holds `blocks`
// words.  Returns 0, -1 for bad arguments, -7 for a launch error.
extern "C" int synth_read_probe(const void* p_dev, int64_t n16, int blocks, int unroll, void* sink_dev,
                                void* stream) {
  if (!p_dev || !sink_dev || n16 <= 0 || blocks <= 0) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint4* p = static_cast<const uint4*>(p_dev);
  uint32_t* sink = static_cast<uint32_t*>(sink_dev);
  switch (unroll) {
    case 1: read_probe_kernel<1><<<blocks, 256, 0, s>>>(p, n16, sink); break;
    case 2: read_probe_kernel<2><<<blocks, 256, 0, s>>>(p, n16, sink); break;
    case 4: read_probe_kernel<4><<<blocks, 256, 0, s>>>(p, n16, sink); break;
    case 8: read_probe_kernel<8><<<blocks, 256, 0, s>>>(p, n16, sink); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -7;
}
