// The fixed device scratch of fold_decode_fused_noalloc: the one-launch
// decode's slots and arrival counts for callers that cannot allocate device
// memory (code under HIP graph capture, serving loops, harnesses that forbid
// allocation).  The array lives in the library's code object, one copy per
// GPU, from the first load of the library until the process ends.
#include <mutex>

#include "fold_internal.h"

namespace fold {

namespace {

constexpr size_t kScratchBytes = size_t{8} << 20;  // 8 MiB per GPU
constexpr int kMaxDevices = 64;

// Host code must never pass `scratch` itself to a kernel: in host code the
// name is a host-side stand-in, not a device address.  scratch_device_ptr()
// returns the device address.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

__global__ void clear_i32_kernel(int32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

size_t scratch_capacity() { return kScratchBytes; }

// The address of `scratch` on the current device: looked up with
// hipGetSymbolAddress the first time the current device asks (with that
// device current) and kept per device.
hipError_t scratch_device_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

// Zeroes n int32 values at p (a fill kernel, not a memset node, so that a
// captured graph replays it faithfully).
hipError_t launch_clear_i32(int32_t* p, int n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int threads = 256;
  hipLaunchKernelGGL(clear_i32_kernel, dim3((n + threads - 1) / threads), dim3(threads), 0, stream,
                     p, n);
  return hipGetLastError();
}

}  // namespace fold
