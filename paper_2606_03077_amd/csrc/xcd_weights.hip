// Per-XCD HBM read rate under full load, as weights for the decode plan's slot placement.
//
// Every workgroup streams its own contiguous block of the caller's buffer with 16-byte
// non-temporal loads (four in flight per lane) for a fixed time on the device's constant
// 100 MHz clock, then records how many loads it issued and on which XCD it ran.  All
// workgroups are resident and reading for the whole interval, so the loads per XCD are
// each XCD's share of the memory system while every XCD competes for it; the host turns
// them into weights.
#include <algorithm>
#include <cmath>
#include <vector>

#include "internal.h"

namespace libra {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;
constexpr int kWorkgroups = 2048;  // 8 per CU: every CU reads for the whole launch

constexpr unsigned long long kTicks = 10000;  // 100 us at 100 MHz

struct Count {
  unsigned long long loads, xcc, sink, pad;
};

__global__ __launch_bounds__(kThreads) void xcd_read_kernel(const u32x4* src, size_t per_wg,
                                                            Count* counts) {
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  const u32x4* p = src + size_t(blockIdx.x) * per_wg;
  u32x4 acc = {0u, 0u, 0u, 0u};
  unsigned long long loads = 0;
  // per_wg is a multiple of kThreads * kUnroll, so every load is inside the block; the
  // block is read again from its start should the interval outlast one pass.
  size_t i = threadIdx.x;
  while (true) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) v[k] = __builtin_nontemporal_load(p + i + k * kThreads);
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) acc ^= v[k];
    loads += kUnroll;
    i += kThreads * kUnroll;
    if (i >= per_wg) i = threadIdx.x;
    if (__builtin_amdgcn_s_memrealtime() - t0 >= kTicks) break;  // wave-uniform
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    Count c;
    c.loads = loads;
    c.xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20) & 0xFu;  // HW_REG_XCC_ID
    c.sink = acc.x ^ acc.y ^ acc.z ^ acc.w;  // keeps the loads
    c.pad = 0;
    counts[blockIdx.x] = c;
  }
}

// Reads [src, src + n16 * 16 bytes) once: workgroup w streams its contiguous block with
// 16-byte non-temporal loads, four in flight per lane, and folds them into one 16-byte
// value per workgroup so that no load is dropped.
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* src, size_t per_wg,
                                                               u32x4* sink) {
  const u32x4* p = src + size_t(blockIdx.x) * per_wg;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t i = threadIdx.x; i < per_wg; i += kThreads * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) v[k] = __builtin_nontemporal_load(p + i + k * kThreads);
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) acc ^= v[k];
  }
  __shared__ u32x4 red[kThreads];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    u32x4 r = {0u, 0u, 0u, 0u};
    for (int t = 0; t < kThreads; ++t) r ^= red[t];
    sink[blockIdx.x] = r;
  }
}

}  // namespace

libra_status measure_hbm_read_rate(const void* buf, size_t bytes, int reps, double* interval_gbps,
                                   double* completion_gbps, hipStream_t s) {
  const size_t chunk = size_t(kThreads) * kUnroll;  // 16-byte elements
  const size_t per_wg = (bytes / 16 / kWorkgroups) / chunk * chunk;
  void* d = nullptr;
  note_alloc_call();
  hipError_t e = hipMalloc(&d, sizeof(Count) * kWorkgroups);
  if (e != hipSuccess) return hip_error(e, "hipMalloc(read-rate counts)");
  Count* d_counts = static_cast<Count*>(d);
  std::vector<Count> h(kWorkgroups);
  hipEvent_t a = nullptr, b = nullptr;
  note_alloc_call();
  note_alloc_call();
  e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  std::vector<double> interval, completion;
  // Completion-timed reads first: consecutive passes over a buffer larger than the
  // 256 MB MALL find none of their lines cached (each pass starts where the previous
  // one's surviving lines are not).  Then the fixed-interval reads.
  for (int r = 0; e == hipSuccess && r <= reps; ++r) {  // pass 0 warms up, not counted
    e = hipEventRecord(a, s);
    if (e == hipSuccess) {
      hipLaunchKernelGGL(stream_read_kernel, dim3(kWorkgroups), dim3(kThreads), 0, s,
                         static_cast<const u32x4*>(buf), per_wg, static_cast<u32x4*>(d));
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipEventRecord(b, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    if (e == hipSuccess && r > 0)
      completion.push_back(double(per_wg) * kWorkgroups * 16.0 / (double(ms) * 1e-3) / 1e9);
  }
  for (int r = 0; e == hipSuccess && r <= reps; ++r) {
    hipLaunchKernelGGL(xcd_read_kernel, dim3(kWorkgroups), dim3(kThreads), 0, s,
                       static_cast<const u32x4*>(buf), per_wg, d_counts);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = hipMemcpyAsync(h.data(), d_counts, sizeof(Count) * kWorkgroups, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess || r == 0) continue;
    // every workgroup read for kTicks of the 100 MHz clock; its first lane's load count
    // stands for each of its lanes, 16 bytes a load
    double loads = 0;
    for (const Count& c : h) loads += double(c.loads);
    interval.push_back(loads * kThreads * 16.0 / (double(kTicks) * 1e-8) / 1e9);
  }
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  note_alloc_call();
  (void)hipFree(d);
  if (e != hipSuccess) return hip_error(e, "HBM read-rate measurement");
  auto median = [](std::vector<double> v) {
    std::sort(v.begin(), v.end());
    return v.size() % 2 ? v[v.size() / 2] : 0.5 * (v[v.size() / 2 - 1] + v[v.size() / 2]);
  };
  *interval_gbps = median(interval);
  *completion_gbps = median(completion);
  return LIBRA_OK;
}

libra_status measure_xcd_weights(const void* buf, size_t bytes, int reps, int32_t* weights,
                                 hipStream_t s) {
  const size_t chunk = size_t(kThreads) * kUnroll;  // 16-byte elements
  const size_t per_wg = (bytes / 16 / kWorkgroups) / chunk * chunk;
  Count* d_counts = nullptr;
  note_alloc_call();
  hipError_t e = hipMalloc(&d_counts, sizeof(Count) * kWorkgroups);
  if (e != hipSuccess) return hip_error(e, "hipMalloc(counts)");
  std::vector<Count> h(kWorkgroups);
  double loads[kNumXcds] = {0};
  libra_status st = LIBRA_OK;
  for (int r = 0; r <= reps; ++r) {  // launch 0 warms up, not counted
    hipLaunchKernelGGL(xcd_read_kernel, dim3(kWorkgroups), dim3(kThreads), 0, s,
                       static_cast<const u32x4*>(buf), per_wg, d_counts);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = hipMemcpyAsync(h.data(), d_counts, sizeof(Count) * kWorkgroups, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      st = hip_error(e, "XCD read calibration");
      break;
    }
    if (r == 0) continue;
    for (const Count& c : h) loads[c.xcc % kNumXcds] += double(c.loads);
  }
  note_alloc_call();
  (void)hipFree(d_counts);
  if (st != LIBRA_OK) return st;
  double most = 0;
  for (int x = 0; x < kNumXcds; ++x) most = std::max(most, loads[x]);
  for (int x = 0; x < kNumXcds; ++x) {
    if (loads[x] <= 0 || most <= 0) {
      weights[x] = 0;  // no workgroup ran there: the plan's default
      continue;
    }
    weights[x] = int32_t(std::clamp(std::lround(1000.0 * loads[x] / most), 1L, 1000L));
  }
  return LIBRA_OK;
}

}  // namespace libra
