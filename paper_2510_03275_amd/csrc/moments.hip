// Mean and population variance of a weight matrix (the variance input of
// MultiOSR, Section 3.4): two passes, fp64 accumulation, fixed reduction order
// (grid-stride partial sums per workgroup, then one workgroup folds the
// partials), so the result is deterministic.
#include <hip/hip_runtime.h>

#include "sdq_internal.h"

namespace sdq {
namespace {

constexpr int kMomBlocks = 1024;
constexpr int kMomThreads = 256;

__device__ inline double block_sum(double v, double* sh) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int s = kMomThreads / 2; s > 0; s >>= 1) {
    if (tid < s) sh[tid] += sh[tid + s];
    __syncthreads();
  }
  return sh[0];
}

// pass 0: partial sums of w; pass 1: partial sums of (w - mean)^2.
__global__ __launch_bounds__(kMomThreads) void moments_partial_kernel(
    const float* __restrict__ w, int64_t count, const double* __restrict__ out, int pass,
    double* __restrict__ partial) {
  __shared__ double sh[kMomThreads];
  const double mean = pass ? out[0] : 0.0;
  double acc = 0.0;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kMomThreads) + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * kMomThreads) {
    const double v = static_cast<double>(w[i]);
    acc += pass ? (v - mean) * (v - mean) : v;
  }
  const double tot = block_sum(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kMomThreads) void moments_final_kernel(
    const double* __restrict__ partial, int nparts, int64_t count, int pass, double* __restrict__ out) {
  __shared__ double sh[kMomThreads];
  double acc = 0.0;
  for (int i = threadIdx.x; i < nparts; i += kMomThreads) acc += partial[i];
  const double tot = block_sum(acc, sh);
  if (threadIdx.x == 0) out[pass] = tot / static_cast<double>(count);
}

}  // namespace

size_t moments_ws_bytes(int64_t count) {
  (void)count;
  return kMomBlocks * sizeof(double);
}

sdq_status launch_moments(const float* w, int64_t count, double* out, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
  (void)ws_bytes;
  double* partial = static_cast<double*>(ws);
  const int64_t want = (count + kMomThreads - 1) / kMomThreads;
  const int blocks = static_cast<int>(want < kMomBlocks ? want : kMomBlocks);
  for (int pass = 0; pass < 2; ++pass) {
    moments_partial_kernel<<<dim3(blocks), dim3(kMomThreads), 0, stream>>>(w, count, out, pass, partial);
    moments_final_kernel<<<dim3(1), dim3(kMomThreads), 0, stream>>>(partial, blocks, count, pass, out);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "moments launch");
  return SDQ_OK;
}

}  // namespace sdq
