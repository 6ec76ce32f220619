// Internal declarations shared by the host code and the HIP kernels of libra.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "libra.h"
#include "tables.h"

namespace libra {

struct Plan {
  int32_t mode = LIBRA_MODE_DECODE;
  int32_t batch = 0, num_q_heads = 0, num_kv_heads = 0, group = 0;
  libra_plan_params params{};
  libra_plan_info info{};
  std::vector<int32_t> units;   // n_units * kUnitInts
  std::vector<int32_t> writes;  // n_write_tiles * kWriteInts (append only)
  std::vector<int32_t> merges;  // n_merge_groups * kMergeInts
  std::vector<int32_t> xcd_map; // (first chunk unit, count) per XCD queue
  int64_t chunk_grid = 0;       // workgroups of the chunk launch: kNumXcds * longest queue

  // Workspace image: [units | writes | merges | xcd map | partial o | partial lse],
  // 256-B aligned.
  size_t off_units = 0, off_writes = 0, off_merges = 0, off_xcd_map = 0, off_part_o = 0,
         off_part_lse = 0;
  size_t ws_bytes = 0;
  size_t upload_bytes = 0;  // bytes of [units | writes | merges | xcd map] from the host
  int64_t pages_needed = 0; // block-table columns the units and writes read (per row, max)
  uint64_t id = 0;          // process-unique, set at creation: which plan a workspace holds

  // Upload state (guarded by upload_mu: calls on one plan may come from several threads).
  // The pinned image and the event come from the library's pool at plan creation and go
  // back to it when the plan is destroyed; both stay null without a visible device.
  std::mutex upload_mu;
  void* pinned = nullptr;         // host staging copy of [units | writes | merges | xcd map]
  size_t pinned_capacity = 0;
  hipEvent_t upload_done = nullptr;
  // Plans with both decode rows and chunk tiles run the two launches concurrently: the
  // decode rows on the device's auxiliary stream, forked from and joined back to the
  // caller's stream by these events (from the pool; null otherwise).
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
};

struct KvLayout {
  libra_kv_layout_desc desc{};
};

// Counts every HIP call of the library that allocates or frees memory or creates an
// event or a stream (libra_alloc_calls reports the total).
void note_alloc_call();

// Error reporting (per thread).
libra_status set_error(libra_status s, const std::string& msg);
libra_status hip_error(hipError_t e, const char* what);

// Plan construction (host, no HIP calls unless num_cus == 0).
libra_status build_plan(const libra_plan_desc& d, const int32_t* seq_lens, const int32_t* q_lens,
                        const libra_plan_params& p, Plan* out);

// Kernel launchers (defined next to their kernels).
hipError_t launch_pack(const KvLayout& L, const void* k_src, const void* v_src, int64_t first,
                       int64_t n, hipStream_t s);
hipError_t launch_unpack(const KvLayout& L, void* k_dst, void* v_dst, int64_t first, int64_t n,
                         hipStream_t s);
hipError_t launch_gather(const KvLayout& L, const int32_t* bt, int32_t stride, const int32_t* cu,
                         int32_t batch, int32_t max_pages, void* k_out, void* v_out, hipStream_t s);
hipError_t launch_cache_write(const KvLayout& L, const Plan& P, const void* ws, const void* k_new,
                              const void* v_new, const int32_t* bt, int32_t stride, hipStream_t s);
hipError_t launch_decode(const KvLayout& L, const Plan& P, void* ws, const void* q,
                         const int32_t* bt, int32_t stride, float scale, void* out, float* lse,
                         hipStream_t s);
// Page-run copies (to_run: cache -> packed run; else packed run -> cache).
hipError_t launch_page_copy(const KvLayout& L, const int32_t* ids, int64_t n, void* k_run,
                            void* v_run, bool to_run, hipStream_t s);
hipError_t launch_merge(const Plan& P, void* ws, void* out, float* lse, hipStream_t s);
bool merge_launches(const Plan& P);  // whether launch_merge enqueues a kernel for P
// Streams buf (reps + 1 launches, the first not counted) and writes per-XCD weights.
libra_status measure_xcd_weights(const void* buf, size_t bytes, int reps, int32_t* weights,
                                 hipStream_t s);
// Streams buf with every CU reading: fixed-interval and completion-timed rates, in GB/s.
libra_status measure_hbm_read_rate(const void* buf, size_t bytes, int reps, double* interval_gbps,
                                   double* completion_gbps, hipStream_t s);
hipError_t launch_chunk(const KvLayout& L, const Plan& P, void* ws, const void* q,
                        const int32_t* bt, int32_t stride, float scale, void* out, float* lse,
                        hipStream_t s);

// The static device scratch of libra_decode_attn_noalloc (csrc/scratch.hip): its size,
// and its address on device `dev` (the calling thread's current device).
size_t scratch_capacity();
libra_status scratch_buffer(int dev, void** out);

}  // namespace libra
