// Device memory of ipk_relpos_attn_run_noalloc: the workspace of such runs lives in one
// file-scope device array, which the module loader places in device memory once per
// GPU (it stays there until the process ends), so those runs allocate nothing.
//
// On the host the array's name is only a stand-in for the device symbol, not a device
// address: host code uses the address hipGetSymbolAddress returns for the current
// device, looked up once per device and kept.
#include <mutex>

#include "../../include/ipk.h"
#include "ipk_internal.h"

static __device__ __align__(256) uint8_t scratch[IPK_NOALLOC_SCRATCH_BYTES];

namespace ipk {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // per device: the array's address, once looked up
}  // namespace

hipError_t noalloc_scratch(uint8_t** base, size_t* bytes) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *base = (uint8_t*)g_scratch_ptr[dev];
  *bytes = IPK_NOALLOC_SCRATCH_BYTES;
  return hipSuccess;
}

}  // namespace ipk
