// Scratch of the decode entry point that allocates nothing: one fixed device array
// per GPU, holding the decode's completion counters and split partials.
#include <mutex>
#include <vector>

#include "common.h"

namespace sonic {

// In host code this name stands for the array, not for its device address: that
// address comes from hipGetSymbolAddress, once per device (see decode_scratch).
static __device__ __align__(256) char scratch[kScratchBytes];

__global__ void clear_counters_kernel(int32_t *p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

namespace {
std::mutex g_scratch_mutex;
std::vector<char *> g_scratch;   // per device: the device address of `scratch` (null until set up)
}  // namespace

// The device address of the current device's scratch.  The first call on a device
// looks it up and enqueues on `stream` a kernel that zeroes the counter region (every
// decode call leaves its counters at zero again, so this is needed once).
hipError_t decode_scratch(hipStream_t stream, char **base) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (static_cast<int>(g_scratch.size()) <= dev) g_scratch.resize(dev + 1, nullptr);
  if (g_scratch[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    const int n = static_cast<int>(kScratchCounterBytes / sizeof(int32_t));
    clear_counters_kernel<<<dim3(16), dim3(256), 0, stream>>>(static_cast<int32_t *>(p), n);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<char *>(p);
  }
  *base = g_scratch[dev];
  return hipSuccess;
}

}  // namespace sonic
