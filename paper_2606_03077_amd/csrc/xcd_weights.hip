// Per-XCD HBM read rate under full load, as weights for the decode plan's slot placement.
//
// Every workgroup streams one contiguous block of the caller's buffer with 16-byte
// non-temporal loads (four in flight per lane) and stamps, on the device's constant
// 100 MHz clock, when it started and finished and on which XCD it ran.  With all XCDs
// reading at once, an XCD whose CUs get a smaller share of the memory system finishes its
// (equal) blocks later; the host turns the per-XCD mean finish times into weights.
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

struct Stamp {
  unsigned long long t0, t1, xcc, sink;
};

__global__ __launch_bounds__(kThreads) void xcd_read_kernel(const u32x4* src, size_t per_wg,
                                                            Stamp* stamps) {
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  const u32x4* p = src + size_t(blockIdx.x) * per_wg;
  u32x4 acc = {0u, 0u, 0u, 0u};
  // per_wg is a multiple of kThreads * kUnroll, so every load is inside the block.
  for (size_t i = threadIdx.x; i < per_wg; i += kThreads * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) v[k] = __builtin_nontemporal_load(p + i + k * kThreads);
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) acc ^= v[k];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    Stamp s;
    s.t0 = t0;
    s.t1 = __builtin_amdgcn_s_memrealtime();
    s.xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20) & 0xFu;  // HW_REG_XCC_ID
    s.sink = acc.x ^ acc.y ^ acc.z ^ acc.w;  // keeps the loads
    stamps[blockIdx.x] = s;
  }
}

}  // namespace

libra_status measure_xcd_weights(const void* buf, size_t bytes, int reps, int32_t* weights,
                                 hipStream_t s) {
  const size_t chunk = size_t(kThreads) * kUnroll;  // 16-byte elements
  const size_t per_wg = (bytes / 16 / kWorkgroups) / chunk * chunk;
  Stamp* d_stamps = nullptr;
  hipError_t e = hipMalloc(&d_stamps, sizeof(Stamp) * kWorkgroups);
  if (e != hipSuccess) return hip_error(e, "hipMalloc(stamps)");
  std::vector<Stamp> h(kWorkgroups);
  double sum[kNumXcds] = {0};
  int64_t cnt[kNumXcds] = {0};
  libra_status st = LIBRA_OK;
  for (int r = 0; r <= reps && st == LIBRA_OK; ++r) {  // launch 0 warms up, not counted
    hipLaunchKernelGGL(xcd_read_kernel, dim3(kWorkgroups), dim3(kThreads), 0, s,
                       static_cast<const u32x4*>(buf), per_wg, d_stamps);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = hipMemcpyAsync(h.data(), d_stamps, sizeof(Stamp) * kWorkgroups, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      st = hip_error(e, "XCD read calibration");
      break;
    }
    if (r == 0) continue;
    unsigned long long base = ~0ull;
    for (const Stamp& x : h) base = std::min(base, x.t0);
    for (const Stamp& x : h) {
      const int xcd = int(x.xcc % kNumXcds);
      sum[xcd] += double(x.t1 - base);
      ++cnt[xcd];
    }
  }
  (void)hipFree(d_stamps);
  if (st != LIBRA_OK) return st;
  double fastest = 0;
  for (int x = 0; x < kNumXcds; ++x)
    if (cnt[x] > 0) {
      const double mean = sum[x] / double(cnt[x]);
      if (fastest == 0 || mean < fastest) fastest = mean;
    }
  for (int x = 0; x < kNumXcds; ++x) {
    if (cnt[x] == 0 || fastest <= 0) {
      weights[x] = 0;  // no workgroup ran there: the plan's default
      continue;
    }
    const double w = 1000.0 * fastest / (sum[x] / double(cnt[x]));
    weights[x] = int32_t(std::clamp(std::lround(w), 1L, 1000L));
  }
  return LIBRA_OK;
}

}  // namespace libra
