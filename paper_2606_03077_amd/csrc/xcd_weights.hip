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

}  // namespace

libra_status measure_xcd_weights(const void* buf, size_t bytes, int reps, int32_t* weights,
                                 hipStream_t s) {
  const size_t chunk = size_t(kThreads) * kUnroll;  // 16-byte elements
  const size_t per_wg = (bytes / 16 / kWorkgroups) / chunk * chunk;
  Count* d_counts = nullptr;
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
