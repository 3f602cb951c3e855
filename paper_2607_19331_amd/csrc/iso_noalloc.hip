// iso_update_noalloc: iso_update for callers that cannot allocate device memory.  Its workspace
// is one static block of device memory per GPU (`scratch`, ISO_NOALLOC_SCRATCH_BYTES), held
// until the process ends.  In host code the name `scratch` only stands in for the device
// symbol: its device address comes from hipGetSymbolAddress, taken once per device on the
// first call there (with that device current) and kept; only that address is passed on.
#include <hip/hip_runtime.h>

#include <mutex>

#include "iso.h"
#include "iso_update_call.h"

namespace {

constexpr size_t kScratchBytes = ISO_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of the current device's block (looked up once per device).
iso_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return ISO_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return ISO_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return ISO_ERR_HIP;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return ISO_OK;
}

iso_status acquire_scratch(size_t need, void** ws, size_t* bytes) {
  if (need > kScratchBytes) return ISO_ERR_UNSUPPORTED;
  const iso_status st = scratch_address(ws);
  if (st == ISO_OK) *bytes = kScratchBytes;
  return st;
}

}  // namespace

extern "C" iso_status iso_update_noalloc(const iso_tensor* t, int n_t, int K, int dt,
                                         const iso_update_args* a, void** scratch_out, void* stream) {
  if (scratch_out != nullptr) {
    *scratch_out = nullptr;
    const iso_status st = scratch_address(scratch_out);
    if (st != ISO_OK) return st;
  }
  iso::WsSource src;
  src.acquire = acquire_scratch;
  return iso::update_call(t, n_t, K, dt, a, src, stream);
}
