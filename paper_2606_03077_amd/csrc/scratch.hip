// The library's static device scratch, used by libra_decode_attn_noalloc in place of a
// caller-provided workspace (plan tables and float32 split partials).  Each GPU the
// library runs on holds its own copy of the array, at its own address, until the process
// ends.  In host code the array's name is only a host-side stand-in: host code uses the
// device address that hipGetSymbolAddress returns for the current device, never the name.
#include <mutex>

#include "internal.h"

namespace {
constexpr size_t kScratchBytes = size_t(8) << 20;  // 8 MiB per device
}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace libra {

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};
}  // namespace

size_t scratch_capacity() { return kScratchBytes; }

// Device address of `scratch` on device `dev`, which must be the calling thread's current
// device.  Looked up once per device (the first call on it) and cached.
libra_status scratch_buffer(int dev, void** out) {
  if (dev < 0 || dev >= kMaxScratchDevices)
    return set_error(LIBRA_E_UNSUPPORTED, "device ordinal outside the scratch table (64 devices)");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_error(e, "hipGetSymbolAddress(scratch)");
    if (!p) return set_error(LIBRA_E_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LIBRA_OK;
}

}  // namespace libra
