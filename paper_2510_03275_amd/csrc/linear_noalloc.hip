// sdq_linear_noalloc: sdq_linear for callers that cannot allocate device
// memory (code under HIP graph capture, serving loops, harnesses that forbid
// hipMalloc).  The workspace is a file-scope device array of fixed size, one
// copy per GPU, alive until the process ends; the coefficient tables must
// already be on the device (sdq_prepare_layout), since building them allocates.
//
// In host code the array's name is only a host-side stand-in, not a device
// address.  Its address on each device is looked up once, with that device
// current, on the first call there (hipGetSymbolAddress); after that the
// looked-up pointer is the only handle host code uses.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "sdq_internal.h"

namespace sdq {
namespace {

constexpr size_t kScratchBytes = SDQ_NOALLOC_SCRATCH_BYTES;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mutex;
std::map<int, void*> g_scratch_ptr;   // device -> device address of its copy of scratch

sdq_status scratch_for_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return SDQ_OK;
  }
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return hip_error(e, "hipGetSymbolAddress(scratch)");
  if (!ptr) return set_error(SDQ_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
  g_scratch_ptr.emplace(dev, ptr);
  *out = ptr;
  return SDQ_OK;
}

}  // namespace
}  // namespace sdq

using namespace sdq;

extern "C" {

sdq_status sdq_linear_noalloc(const void* x, sdq_dtype xt, int64_t m, const void* codes,
                              const float* scales, const sdq_layout* layout, float* y,
                              int32_t accumulate, void* stream) {
  if (m > 0 && layout && layout->n > 0) {
    const size_t need = linear_ws_need(layout, m);
    if (need > kScratchBytes)
      return set_error(SDQ_ERR_WORKSPACE,
                       "this call needs %zu bytes of workspace; sdq_linear_noalloc has %zu "
                       "(use sdq_linear with a workspace)", need, kScratchBytes);
  }
  void* ws = nullptr;
  sdq_status st = scratch_for_current_device(&ws);
  if (st != SDQ_OK) return st;
  return linear_impl(x, xt, m, codes, scales, layout, y, accumulate, ws, kScratchBytes, stream, false);
}

}  // extern "C"
