// A host-only stand-in for the HIP runtime calls that the library's host code makes, for
// the no-allocation check: "device" memory is host memory, copies are memcpy, events are
// counters.  Every allocating call is counted, so a driver can assert which entry points
// allocate.  Not a HIP implementation: it supports exactly what the host sources call.
#include <hip/hip_runtime_api.h>

#include <cstdlib>
#include <cstring>

#include "fake_hip.h"

FakeHipCounters g_fake_hip;

extern "C" {

hipError_t hipGetDeviceCount(int* count) {
  *count = 1;
  return hipSuccess;
}
hipError_t hipGetDevice(int* id) {
  *id = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* pi, hipDeviceAttribute_t, int) {
  *pi = 256;
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "fake hip error"; }

hipError_t hipHostMalloc(void** ptr, size_t size, unsigned int) {
  ++g_fake_hip.host_malloc;
  *ptr = std::malloc(size ? size : 1);
  return *ptr ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipHostFree(void* ptr) {
  ++g_fake_hip.host_free;
  std::free(ptr);
  return hipSuccess;
}
hipError_t hipMalloc(void** ptr, size_t size) {
  ++g_fake_hip.device_malloc;
  *ptr = std::malloc(size ? size : 1);
  return hipSuccess;
}
hipError_t hipFree(void* ptr) {
  ++g_fake_hip.device_free;
  std::free(ptr);
  return hipSuccess;
}

struct FakeEvent { int recorded; };

hipError_t hipEventCreate(hipEvent_t* e) {
  ++g_fake_hip.event_create;
  *e = reinterpret_cast<hipEvent_t>(new FakeEvent{0});
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  ++g_fake_hip.event_destroy;
  delete reinterpret_cast<FakeEvent*>(e);
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) {
  ++g_fake_hip.event_record;
  reinterpret_cast<FakeEvent*>(e)->recorded = 1;
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t) {
  ++g_fake_hip.event_sync;
  return hipSuccess;
}
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t* st, unsigned int) {
  ++g_fake_hip.stream_create;
  *st = reinterpret_cast<hipStream_t>(new int(0));
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned int) {
  ++g_fake_hip.stream_wait;
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  ++g_fake_hip.memcpy_async;
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipPointerGetAttributes(hipPointerAttribute_t* a, const void* p) {
  std::memset(a, 0, sizeof(*a));
  a->type = hipMemoryTypeDevice;
  a->devicePointer = const_cast<void*>(p);
  return hipSuccess;
}

}  // extern "C"
