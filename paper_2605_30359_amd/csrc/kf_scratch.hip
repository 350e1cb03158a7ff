// The static device scratch of kf_fused_op_noalloc: one file-scope device
// array per GPU that the library runs on, held until the process ends, for
// callers that cannot allocate device memory.  The array's name is a host
// stand-in in host code, so its device address is looked up once per device
// (with that device current) and only that address is passed to kernels.
#include <hip/hip_runtime.h>

#include <atomic>

#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr size_t kScratchBytes = size_t(4) << 20;  // 4 MiB per device
constexpr int kMaxScratchDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::atomic<void*> g_scratch_ptr[kMaxScratchDevices];

}  // namespace

hipError_t scratch_address(int device, void** out) {
  if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[device].load(std::memory_order_acquire);
  if (!p) {
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device].store(p, std::memory_order_release);
  }
  *out = p;
  return hipSuccess;
}

size_t scratch_bytes() { return kScratchBytes; }

}  // namespace kf
