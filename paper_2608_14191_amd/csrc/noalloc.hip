// The workspace of aatc_append_decode_attention_noalloc: a file-scope device array, one per
// GPU that the library runs on, held until the process ends.  It serves callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops).
//
// Layout: the arrival counters of up to kScratchRows (sequence, KV head) rows at the start
// (fixed, whatever the shape of a call), then the split partials and the fused append's
// coefficients of the call.  The counters must start at zero: the array is zero when the
// code object loads, a fill kernel clears that region once more at the first call on each
// device, and every decode launch leaves the counters it used at zero.  Everything else is
// written before it is read.  Calls that overlap on one GPU share the array and race.
#include <mutex>

#include <hip/hip_runtime.h>

#include "launch.h"
#include "params.h"

static __device__ __align__(256) unsigned char scratch[aatc::kScratchBytes];

namespace aatc {
namespace {

constexpr int kMaxDevices = 64;

__global__ void zero_words(unsigned* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

struct DeviceScratch {
  std::once_flag once;
  void* ptr = nullptr;
  aatc_status status = AATC_E_DEVICE;
};
DeviceScratch g_scratch[kMaxDevices];

}  // namespace

aatc_status noalloc_scratch(void** ptr, void* stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return AATC_E_DEVICE;
  DeviceScratch& s = g_scratch[dev];
  std::call_once(s.once, [&] {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return;
    // The counters region (its size in the layout that reserves kScratchRows rows).
    const size_t words = decode_workspace_bytes(1, 1, 1, kTile, kScratchRows) / 4;
    hipLaunchKernelGGL(zero_words, dim3(16), dim3(256), 0, (hipStream_t)stream,
                       static_cast<unsigned*>(p), words);
    if (hipGetLastError() != hipSuccess) return;
    s.ptr = p;
    s.status = AATC_OK;
  });
  if (s.status != AATC_OK) return s.status;
  *ptr = s.ptr;
  return AATC_OK;
}

}  // namespace aatc
