// Device twin of the synthetic input generator (synth/__init__.py): the same
// counter-based definition, written independently for the GPU so that
// weights of any size can be produced in place.  It holds no arithmetic of
// the quantization method.
//
//   hash(i)  = SplitMix64 output function of base + (i + 1) * GAMMA
//              (Steele, Lea and Flood, OOPSLA 2014);
//   normal   = Irwin-Hall sum S of the eight 16-bit halves of hash(3e) and
//              hash(3e + 1), value = fp32(fp64(2S - 8*65535) * factor);
//   outlier  = hash(3e + 2) < threshold multiplies the value by 10 in fp32.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kMix1 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kMix2 = 0x94D049BB133111EBull;

__device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * kMix1;
  z = (z ^ (z >> 27)) * kMix2;
  return z ^ (z >> 31);
}

__device__ inline uint64_t hash_at(uint64_t base, uint64_t i) { return mix64(base + (i + 1) * kGamma); }

__device__ inline int64_t halves(uint64_t h) {
  return static_cast<int64_t>((h & 0xFFFFull) + ((h >> 16) & 0xFFFFull) + ((h >> 32) & 0xFFFFull) + (h >> 48));
}

__global__ void normal_kernel(float* __restrict__ out, int64_t rows, int64_t cols, int64_t row0,
                              uint64_t base, double factor, int outliers, uint64_t threshold) {
  const int64_t total = rows * cols;
  for (int64_t idx = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const uint64_t e = static_cast<uint64_t>((row0 + idx / cols) * cols + idx % cols);
    const int64_t s = halves(hash_at(base, 3 * e)) + halves(hash_at(base, 3 * e + 1));
    float v = static_cast<float>(static_cast<double>(2 * s - 8 * 65535) * factor);
    if (outliers && hash_at(base, 3 * e + 2) < threshold) v = v * 10.0f;
    out[idx] = v;
  }
}

}  // namespace

extern "C" int synth_normal_f32(float* out_dev, int64_t rows, int64_t cols, int64_t row0,
                                uint64_t base, double factor, int outliers, uint64_t threshold,
                                void* stream) {
  if (rows < 0 || cols <= 0 || row0 < 0 || (rows > 0 && !out_dev)) return -1;
  if (rows == 0) return 0;
  const int64_t total = rows * cols;
  const int64_t want = (total + 255) / 256;
  const unsigned grid = static_cast<unsigned>(want < 65536 ? want : 65536);
  normal_kernel<<<dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream)>>>(
      out_dev, rows, cols, row0, base, factor, outliers, threshold);
  return hipGetLastError() == hipSuccess ? 0 : -7;
}
