// Kernel-launcher stand-ins for the host-only sanitizer build: the driver never reaches a
// launch (it calls only host entry points); these keep api.cpp linkable without device code.
#include "internal.h"

namespace libra {
hipError_t launch_pack(const KvLayout&, const void*, const void*, int64_t, int64_t, hipStream_t) { return hipErrorUnknown; }
hipError_t launch_unpack(const KvLayout&, void*, void*, int64_t, int64_t, hipStream_t) { return hipErrorUnknown; }
hipError_t launch_gather(const KvLayout&, const int32_t*, int32_t, const int32_t*, int32_t, int32_t, void*, void*, hipStream_t) { return hipErrorUnknown; }
hipError_t launch_cache_write(const KvLayout&, const Plan&, const void*, const void*, const void*, const int32_t*, int32_t, hipStream_t) { return hipErrorUnknown; }
hipError_t launch_decode(const KvLayout&, const Plan&, void*, const void*, const int32_t*, int32_t, float, void*, float*, hipStream_t) { return hipErrorUnknown; }
hipError_t launch_merge(const Plan&, void*, void*, float*, hipStream_t) { return hipErrorUnknown; }
bool merge_launches(const Plan&) { return false; }
hipError_t launch_chunk(const KvLayout&, const Plan&, void*, const void*, const int32_t*, int32_t, float, void*, float*, hipStream_t) { return hipErrorUnknown; }
libra_status measure_xcd_weights(const void*, size_t, int, int32_t*, hipStream_t) { return LIBRA_E_HIP; }
hipError_t launch_page_copy(const KvLayout&, const int32_t*, int64_t, void*, void*, bool, hipStream_t) { return hipErrorUnknown; }
}  // namespace libra
