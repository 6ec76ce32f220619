// Kernel-launcher stand-ins for the host-only builds, which compile no device code.  By
// default every launch fails (the sanitizer driver calls only host entry points); built
// with LIBRA_STUB_LAUNCH_OK (beside the HIP stand-in of fake_hip.cpp), every launch
// succeeds and is counted, so that decode / append calls run their host path to the end.
#include "internal.h"

#ifdef LIBRA_STUB_LAUNCH_OK
#include "fake_hip.h"
#define LAUNCH_RESULT (++g_fake_hip.launches, hipSuccess)
#else
#define LAUNCH_RESULT hipErrorUnknown
#endif

namespace libra {
hipError_t launch_pack(const KvLayout&, const void*, const void*, int64_t, int64_t, hipStream_t) { return LAUNCH_RESULT; }
hipError_t launch_unpack(const KvLayout&, void*, void*, int64_t, int64_t, hipStream_t) { return LAUNCH_RESULT; }
hipError_t launch_gather(const KvLayout&, const int32_t*, int32_t, const int32_t*, int32_t, int32_t, void*, void*, hipStream_t) { return LAUNCH_RESULT; }
hipError_t launch_cache_write(const KvLayout&, const Plan&, const void*, const void*, const void*, const int32_t*, int32_t, hipStream_t) { return LAUNCH_RESULT; }
hipError_t launch_decode(const KvLayout&, const Plan&, void*, const void*, const int32_t*, int32_t, float, void*, float*, hipStream_t) { return LAUNCH_RESULT; }
hipError_t launch_merge(const Plan&, void*, void*, float*, hipStream_t) { return LAUNCH_RESULT; }
bool merge_launches(const Plan&) { return false; }
hipError_t launch_chunk(const KvLayout&, const Plan&, void*, const void*, const int32_t*, int32_t, float, void*, float*, hipStream_t) { return LAUNCH_RESULT; }
libra_status measure_xcd_weights(const void*, size_t, int, int32_t*, hipStream_t) { return LIBRA_E_HIP; }
libra_status measure_hbm_read_rate(const void*, size_t, int, double*, double*, hipStream_t) { return LIBRA_E_HIP; }
hipError_t launch_page_copy(const KvLayout&, const int32_t*, int64_t, void*, void*, bool, hipStream_t) { return LAUNCH_RESULT; }
// The static device scratch lives in device code; here it is a host array.
size_t scratch_capacity() { return size_t(8) << 20; }
libra_status scratch_buffer(int, void** out) {
  alignas(256) static unsigned char host_scratch[size_t(8) << 20];
  *out = host_scratch;
  return LIBRA_OK;
}
}  // namespace libra
