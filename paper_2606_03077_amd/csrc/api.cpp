// extern "C" entry points of libra (declared and documented in include/libra.h).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <iterator>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "internal.h"

namespace libra {

namespace {
thread_local std::string g_last_error;
}

libra_status set_error(libra_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

libra_status hip_error(hipError_t e, const char* what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return LIBRA_E_HIP;
}

namespace {
std::atomic<uint64_t> g_alloc_calls{0};
}

void note_alloc_call() { g_alloc_calls.fetch_add(1, std::memory_order_relaxed); }

namespace {

constexpr size_t kWorkspaceAlign = 256;

// Per-kernel timing: event pairs recorded around launches while enabled.
struct Profiler {
  std::mutex mu;
  bool enabled = false;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> free_events;

  hipEvent_t get() {
    if (!free_events.empty()) {
      hipEvent_t e = free_events.back();
      free_events.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    note_alloc_call();
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Profiler g_prof;

// Brackets one kernel launch with events when profiling is on.
class ProfScope {
 public:
  ProfScope(int kind, hipStream_t s, bool active) : kind_(kind), s_(s) {
    if (!active) return;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    if (!g_prof.enabled) return;
    a_ = g_prof.get();
    b_ = g_prof.get();
    if (a_ && b_ && hipEventRecord(a_, s_) == hipSuccess) return;
    release();
  }
  ~ProfScope() {
    if (!a_) return;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    if (hipEventRecord(b_, s_) == hipSuccess) {
      g_prof.pending.push_back({kind_, a_, b_});
    } else {
      release();
    }
  }

 private:
  void release() {
    if (a_) g_prof.free_events.push_back(a_);
    if (b_) g_prof.free_events.push_back(b_);
    a_ = b_ = nullptr;
  }
  int kind_;
  hipStream_t s_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

libra_status check_layout(const libra_kv_layout_desc* d) {
  if (!d) return set_error(LIBRA_E_INVAL, "layout descriptor is NULL");
  if (d->page_size != kPage) return set_error(LIBRA_E_UNSUPPORTED, "page_size must be 16");
  if (d->head_dim != kDim) return set_error(LIBRA_E_UNSUPPORTED, "head_dim must be 128");
  if (d->dtype != LIBRA_DTYPE_BF16) return set_error(LIBRA_E_UNSUPPORTED, "dtype must be bf16");
  if (d->num_kv_heads <= 0) return set_error(LIBRA_E_INVAL, "num_kv_heads must be > 0");
  if (d->num_kv_heads > LIBRA_MAX_KV_HEADS)
    return set_error(LIBRA_E_UNSUPPORTED, "num_kv_heads must be <= 1024");
  if (d->num_pages <= 0) return set_error(LIBRA_E_INVAL, "num_pages must be > 0");
  if (d->num_pages > (int64_t(1) << 40) / d->num_kv_heads)
    return set_error(LIBRA_E_INVAL, "num_pages * num_kv_heads too large");
  if (!d->k_cache || !d->v_cache) return set_error(LIBRA_E_INVAL, "k_cache / v_cache is NULL");
  if ((reinterpret_cast<uintptr_t>(d->k_cache) | reinterpret_cast<uintptr_t>(d->v_cache)) & 15)
    return set_error(LIBRA_E_INVAL, "k_cache / v_cache must be 16-byte aligned");
  return LIBRA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Which plan's tables each workspace holds, by plan id: a call skips the table upload
// only if its own plan was the last to upload to that workspace, so plans that take
// turns on one workspace never read each other's tables.
struct WorkspaceOwners {
  std::mutex mu;
  std::unordered_map<uintptr_t, uint64_t> owner;
};
WorkspaceOwners g_ws;
std::atomic<uint64_t> g_next_plan_id{1};

// Which plan's tables the static scratch of each device holds (0: none).  Plan ids are
// never reused, so a destroyed plan's id can never match a live plan.
constexpr int kMaxScratchOwners = 64;
std::atomic<uint64_t> g_scratch_owner[kMaxScratchOwners] = {};

bool holds_tables(const void* ws, uint64_t id) {
  std::lock_guard<std::mutex> lk(g_ws.mu);
  auto it = g_ws.owner.find(reinterpret_cast<uintptr_t>(ws));
  return it != g_ws.owner.end() && it->second == id;
}

// Pinned staging images and upload events, owned by the library and reused by plans.
// A plan takes one of each when it is built (libra_splitkv_plan) and returns them when it
// is destroyed, so decode / append calls never allocate, and destroying a plan frees no
// pinned memory (hipHostFree may wait for the device).  The pool never shrinks: it holds
// as many images as plans were alive at once, and is never destroyed (its memory is not
// freed at exit, when the HIP runtime may already be torn down).
struct StagingPool {
  std::mutex mu;
  std::vector<std::pair<size_t, void*>> images;  // (capacity, pinned host memory)
  std::vector<hipEvent_t> events;
};
StagingPool& g_staging = *new StagingPool();

libra_status staging_acquire(Plan& P) {
  std::lock_guard<std::mutex> lk(g_staging.mu);
  if (P.upload_bytes > 0) {
    size_t best = g_staging.images.size();
    for (size_t i = 0; i < g_staging.images.size(); ++i)
      if (g_staging.images[i].first >= P.upload_bytes &&
          (best == g_staging.images.size() ||
           g_staging.images[i].first < g_staging.images[best].first))
        best = i;
    if (best < g_staging.images.size()) {
      P.pinned_capacity = g_staging.images[best].first;
      P.pinned = g_staging.images[best].second;
      g_staging.images.erase(g_staging.images.begin() + static_cast<std::ptrdiff_t>(best));
    } else {
      size_t cap = 4096;
      while (cap < P.upload_bytes) cap *= 2;
      note_alloc_call();
      hipError_t e = hipHostMalloc(&P.pinned, cap, hipHostMallocDefault);
      if (e != hipSuccess) {
        P.pinned = nullptr;
        return hip_error(e, "hipHostMalloc(plan tables)");
      }
      P.pinned_capacity = cap;
    }
  }
  auto take_event = [](hipEvent_t* ev) -> libra_status {
    if (!g_staging.events.empty()) {
      *ev = g_staging.events.back();
      g_staging.events.pop_back();
      return LIBRA_OK;
    }
    note_alloc_call();
    hipError_t e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
    if (e != hipSuccess) {
      *ev = nullptr;
      return hip_error(e, "hipEventCreate(plan)");
    }
    return LIBRA_OK;
  };
  libra_status st = take_event(&P.upload_done);
  if (st != LIBRA_OK) return st;
  if (P.info.n_single > 0 && P.info.n_chunk > 0) {
    st = take_event(&P.fork_ev);
    if (st == LIBRA_OK) st = take_event(&P.join_ev);
    if (st != LIBRA_OK) return st;
  }
  return LIBRA_OK;
}

void staging_release(Plan& P) {
  std::lock_guard<std::mutex> lk(g_staging.mu);
  if (P.pinned) g_staging.images.emplace_back(P.pinned_capacity, P.pinned);
  for (hipEvent_t* ev : {&P.upload_done, &P.fork_ev, &P.join_ev}) {
    if (*ev) g_staging.events.push_back(*ev);
    *ev = nullptr;
  }
  P.pinned = nullptr;
}

// One auxiliary stream per device (default priority, non-blocking), created with the
// first plan that has both decode rows and chunk tiles, and kept until the process ends.
constexpr int kMaxAuxDevices = 64;
std::mutex g_aux_mu;
hipStream_t g_aux_stream[kMaxAuxDevices] = {};

libra_status ensure_aux_stream() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxAuxDevices) return LIBRA_OK;  // such devices run sequentially
  std::lock_guard<std::mutex> lk(g_aux_mu);
  if (!g_aux_stream[dev]) {
    note_alloc_call();
    e = hipStreamCreateWithFlags(&g_aux_stream[dev], hipStreamNonBlocking);
    if (e != hipSuccess) {
      g_aux_stream[dev] = nullptr;
      return hip_error(e, "hipStreamCreate(auxiliary)");
    }
  }
  return LIBRA_OK;
}

// The current device's auxiliary stream, or null if it has none (then run sequentially).
hipStream_t aux_stream() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxAuxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_aux_mu);
  return g_aux_stream[dev];
}

// Fills the plan's pinned image with its tables (at plan creation).
void staging_fill(Plan& P) {
  if (!P.pinned) return;
  char* h = static_cast<char*>(P.pinned);
  std::memset(h, 0, P.upload_bytes);
  auto put = [h](size_t off, const std::vector<int32_t>& v) {
    if (!v.empty()) std::memcpy(h + off, v.data(), v.size() * sizeof(int32_t));
  };
  put(P.off_units, P.units);
  put(P.off_writes, P.writes);
  put(P.off_merges, P.merges);
  put(P.off_xcd_map, P.xcd_map);
}

// Enqueues the copy of the plan's pinned table image to ws and records its event.
// Allocates nothing.  Caller holds P.upload_mu.
libra_status enqueue_tables(Plan& P, void* ws, hipStream_t s) {
  if (!P.upload_done)
    return set_error(LIBRA_E_INVAL,
                     "plan was built without a visible HIP device; it cannot run on one");
  hipError_t e;
  {
    ProfScope ps(LIBRA_KERNEL_UPLOAD, s, true);
    if (P.upload_bytes > 0) {
      e = hipMemcpyAsync(ws, P.pinned, P.upload_bytes, hipMemcpyHostToDevice, s);
      if (e != hipSuccess) return hip_error(e, "hipMemcpyAsync(plan tables)");
    }
  }
  e = hipEventRecord(P.upload_done, s);
  if (e != hipSuccess) return hip_error(e, "hipEventRecord");
  return LIBRA_OK;
}

// Copies the plan's tables into ws unless ws already holds them (or always, if forced).
libra_status upload(Plan& P, void* ws, size_t ws_bytes, hipStream_t s, bool force = true) {
  std::lock_guard<std::mutex> lk(P.upload_mu);
  if (!force && holds_tables(ws, P.id)) return LIBRA_OK;
  if (!ws) return set_error(LIBRA_E_INVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kWorkspaceAlign)
    return set_error(LIBRA_E_INVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < P.ws_bytes)
    return set_error(LIBRA_E_WORKSPACE, "workspace smaller than libra_plan_workspace_bytes");
  libra_status st = enqueue_tables(P, ws, s);
  if (st != LIBRA_OK) return st;
  {
    std::lock_guard<std::mutex> lk2(g_ws.mu);
    g_ws.owner[reinterpret_cast<uintptr_t>(ws)] = P.id;
  }
  return LIBRA_OK;
}

libra_status check_call(const KvLayout* L, const Plan* P, int mode, const void* q,
                        const int32_t* bt, int32_t bt_stride, int32_t batch, int32_t hq,
                        float scale, const void* out) {
  if (!L || !P) return set_error(LIBRA_E_INVAL, "layout or plan is NULL");
  if (P->mode != mode)
    return set_error(LIBRA_E_INVAL, mode == LIBRA_MODE_DECODE ? "plan is not a decode plan"
                                                              : "plan is not an append plan");
  if (batch != P->batch || hq != P->num_q_heads)
    return set_error(LIBRA_E_INVAL, "batch / num_q_heads differ from the plan's");
  if (P->num_kv_heads != L->desc.num_kv_heads)
    return set_error(LIBRA_E_INVAL, "plan and layout disagree on num_kv_heads");
  if (!(scale > 0.f) || !std::isfinite(scale))
    return set_error(LIBRA_E_INVAL, "scale must be positive and finite");
  if (P->info.n_rows > 0) {
    if (!q || !out) return set_error(LIBRA_E_INVAL, "q / out is NULL");
    if (!aligned16(q) || !aligned16(out)) return set_error(LIBRA_E_INVAL, "q / out must be 16-byte aligned");
  }
  const int64_t need = P->pages_needed;
  if (need > 0) {
    if (!bt) return set_error(LIBRA_E_INVAL, "block_table is NULL");
    if (bt_stride < need)
      return set_error(LIBRA_E_INVAL, "bt_stride smaller than the pages the plan's lengths need");
  }
  return LIBRA_OK;
}

// Decode units, chunk units, then the merge of split rows.  `timed` allows per-kernel
// timing events (which may create events while timing is enabled).  When the plan has
// both decode rows and chunk tiles, the chunk launch goes first on `s` and the decode
// launch on the device's auxiliary stream, forked from `s` after everything enqueued
// before and joined back before the merge: the dispatcher then fills the CUs that the
// matrix-core bound chunk tiles free with the HBM-bound decode rows as they come.
std::mutex g_fork_mu;  // record / wait pairs of concurrent callers must not interleave

libra_status launch_attention(const KvLayout& L, const Plan& P, void* ws, const void* q,
                              const int32_t* bt, int32_t stride, float scale, void* out,
                              float* lse, hipStream_t s, bool timed = true) {
  hipError_t e;
  hipStream_t s2 = nullptr;
  if (P.info.n_single > 0 && P.info.n_chunk > 0 && P.fork_ev && P.join_ev) s2 = aux_stream();
  if (s2) {
    {
      std::lock_guard<std::mutex> lk(g_fork_mu);
      e = hipEventRecord(P.fork_ev, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(s2, P.fork_ev, 0);
    }
    if (e != hipSuccess) return hip_error(e, "forking the decode rows");
    {
      ProfScope ps(LIBRA_KERNEL_CHUNK, s, timed);
      e = launch_chunk(L, P, ws, q, bt, stride, scale, out, lse, s);
    }
    if (e != hipSuccess) return hip_error(e, "chunk launch");
    {
      ProfScope ps(LIBRA_KERNEL_DECODE, s2, timed);
      e = launch_decode(L, P, ws, q, bt, stride, scale, out, lse, s2);
    }
    if (e != hipSuccess) return hip_error(e, "decode launch");
    {
      std::lock_guard<std::mutex> lk(g_fork_mu);
      e = hipEventRecord(P.join_ev, s2);
      if (e == hipSuccess) e = hipStreamWaitEvent(s, P.join_ev, 0);
    }
    if (e != hipSuccess) return hip_error(e, "joining the decode rows");
  } else {
    {
      ProfScope ps(LIBRA_KERNEL_DECODE, s, timed && P.info.n_single > 0);
      e = launch_decode(L, P, ws, q, bt, stride, scale, out, lse, s);
    }
    if (e != hipSuccess) return hip_error(e, "decode launch");
    {
      ProfScope ps(LIBRA_KERNEL_CHUNK, s, timed && P.info.n_chunk > 0);
      e = launch_chunk(L, P, ws, q, bt, stride, scale, out, lse, s);
    }
    if (e != hipSuccess) return hip_error(e, "chunk launch");
  }
  {
    ProfScope ps(LIBRA_KERNEL_MERGE, s, timed && merge_launches(P));
    e = launch_merge(P, ws, out, lse, s);
  }
  return e == hipSuccess ? LIBRA_OK : hip_error(e, "merge launch");
}

// The address a kernel uses for a page run: device memory as is, pinned host memory
// through its device mapping (the copy then crosses PCIe inside the kernel).  Memory the
// runtime does not know (pageable host memory) is refused.
bool device_view(const void* p, void** out) {
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();  // clear the runtime's last error; the caller reports its own
    return false;
  }
  if (a.type == hipMemoryTypeDevice) {
    *out = const_cast<void*>(p);
    return true;
  }
  if (a.type == hipMemoryTypeHost && a.devicePointer && a.hostPointer) {
    *out = static_cast<char*>(a.devicePointer) +
           (static_cast<const char*>(p) - static_cast<const char*>(a.hostPointer));
    return true;
  }
  return false;
}

libra_status page_copy(const KvLayout* layout, const int32_t* page_ids, int64_t n_pages,
                       const void* k_run, const void* v_run, bool to_run, void* stream) {
  if (!layout) return set_error(LIBRA_E_INVAL, "layout is NULL");
  if (!k_run && !v_run) return set_error(LIBRA_E_INVAL, "K and V page runs are both NULL");
  if (n_pages < 0 || n_pages > layout->desc.num_pages)
    return set_error(LIBRA_E_INVAL, "n_pages must be in [0, num_pages]");
  if (n_pages == 0) return LIBRA_OK;
  if (!page_ids) return set_error(LIBRA_E_INVAL, "page_ids is NULL");
  if ((k_run && !aligned16(k_run)) || (v_run && !aligned16(v_run)))
    return set_error(LIBRA_E_INVAL, "page runs must be 16-byte aligned");
  void* k_dev = nullptr;
  void* v_dev = nullptr;
  if (k_run && !device_view(k_run, &k_dev))
    return set_error(LIBRA_E_INVAL, "K page run is neither device nor pinned host memory");
  if (v_run && !device_view(v_run, &v_dev))
    return set_error(LIBRA_E_INVAL, "V page run is neither device nor pinned host memory");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    ProfScope ps(to_run ? LIBRA_KERNEL_COPY_OUT : LIBRA_KERNEL_COPY_IN, s, true);
    e = launch_page_copy(*layout, page_ids, n_pages, k_dev, v_dev, to_run, s);
  }
  return e == hipSuccess ? LIBRA_OK : hip_error(e, "page copy launch");
}

}  // namespace
}  // namespace libra

using namespace libra;

struct libra_kv_layout_s : KvLayout {};
struct libra_plan_s : Plan {};

extern "C" {

const char* libra_status_string(libra_status s) {
  switch (s) {
    case LIBRA_OK: return "LIBRA_OK";
    case LIBRA_E_INVAL: return "LIBRA_E_INVAL";
    case LIBRA_E_UNSUPPORTED: return "LIBRA_E_UNSUPPORTED";
    case LIBRA_E_WORKSPACE: return "LIBRA_E_WORKSPACE";
    case LIBRA_E_HIP: return "LIBRA_E_HIP";
    case LIBRA_E_NOMEM: return "LIBRA_E_NOMEM";
  }
  return "LIBRA_E_UNKNOWN";
}

const char* libra_last_error(void) { return g_last_error.c_str(); }

uint64_t libra_alloc_calls(void) { return g_alloc_calls.load(std::memory_order_relaxed); }

libra_status libra_kv_layout_create(const libra_kv_layout_desc* desc, libra_kv_layout* out) {
  if (!out) return set_error(LIBRA_E_INVAL, "out is NULL");
  *out = nullptr;
  libra_status st = check_layout(desc);
  if (st != LIBRA_OK) return st;
  auto* L = new (std::nothrow) libra_kv_layout_s();
  if (!L) return set_error(LIBRA_E_NOMEM, "layout allocation failed");
  L->desc = *desc;
  *out = L;
  return LIBRA_OK;
}

void libra_kv_layout_destroy(libra_kv_layout layout) { delete layout; }

libra_status libra_kv_pack_pages(libra_kv_layout layout, const void* k_src, const void* v_src,
                                 int64_t first_page, int64_t n_pages, void* stream) {
  if (!layout) return set_error(LIBRA_E_INVAL, "layout is NULL");
  if (!k_src && !v_src) return set_error(LIBRA_E_INVAL, "k_src and v_src are both NULL");
  if (first_page < 0 || n_pages < 0 || first_page + n_pages > layout->desc.num_pages)
    return set_error(LIBRA_E_INVAL, "page range outside the cache");
  if ((k_src && !aligned16(k_src)) || (v_src && !aligned16(v_src)))
    return set_error(LIBRA_E_INVAL, "sources must be 16-byte aligned");
  hipError_t e;
  {
    ProfScope ps(LIBRA_KERNEL_PACK, static_cast<hipStream_t>(stream), n_pages > 0);
    e = launch_pack(*layout, k_src, v_src, first_page, n_pages, static_cast<hipStream_t>(stream));
  }
  return e == hipSuccess ? LIBRA_OK : hip_error(e, "pack launch");
}

libra_status libra_kv_unpack_pages(libra_kv_layout layout, void* k_dst, void* v_dst,
                                   int64_t first_page, int64_t n_pages, void* stream) {
  if (!layout) return set_error(LIBRA_E_INVAL, "layout is NULL");
  if (!k_dst && !v_dst) return set_error(LIBRA_E_INVAL, "k_dst and v_dst are both NULL");
  if (first_page < 0 || n_pages < 0 || first_page + n_pages > layout->desc.num_pages)
    return set_error(LIBRA_E_INVAL, "page range outside the cache");
  if ((k_dst && !aligned16(k_dst)) || (v_dst && !aligned16(v_dst)))
    return set_error(LIBRA_E_INVAL, "destinations must be 16-byte aligned");
  hipError_t e;
  {
    ProfScope ps(LIBRA_KERNEL_UNPACK, static_cast<hipStream_t>(stream), n_pages > 0);
    e = launch_unpack(*layout, k_dst, v_dst, first_page, n_pages, static_cast<hipStream_t>(stream));
  }
  return e == hipSuccess ? LIBRA_OK : hip_error(e, "unpack launch");
}

libra_status libra_kv_gather(libra_kv_layout layout, const int32_t* block_table, int32_t bt_stride,
                             const int32_t* cu_seq_lens, int32_t batch, int32_t max_pages,
                             void* k_out, void* v_out, void* stream) {
  if (!layout) return set_error(LIBRA_E_INVAL, "layout is NULL");
  if (batch < 0 || max_pages < 0) return set_error(LIBRA_E_INVAL, "batch / max_pages < 0");
  if (batch == 0 || max_pages == 0) return LIBRA_OK;
  if (!block_table || !cu_seq_lens || !k_out || !v_out)
    return set_error(LIBRA_E_INVAL, "NULL pointer argument");
  if (bt_stride < max_pages) return set_error(LIBRA_E_INVAL, "bt_stride < max_pages");
  if (batch > 65535 || layout->desc.num_kv_heads > 65535)
    return set_error(LIBRA_E_UNSUPPORTED, "batch and num_kv_heads must be <= 65535");
  if (!aligned16(k_out) || !aligned16(v_out))
    return set_error(LIBRA_E_INVAL, "outputs must be 16-byte aligned");
  hipError_t e;
  {
    ProfScope ps(LIBRA_KERNEL_GATHER, static_cast<hipStream_t>(stream), true);
    e = launch_gather(*layout, block_table, bt_stride, cu_seq_lens, batch, max_pages, k_out, v_out,
                      static_cast<hipStream_t>(stream));
  }
  return e == hipSuccess ? LIBRA_OK : hip_error(e, "gather launch");
}

libra_status libra_kv_copy_out(libra_kv_layout layout, const int32_t* page_ids, int64_t n_pages,
                               void* k_dst, void* v_dst, void* stream) {
  return page_copy(layout, page_ids, n_pages, k_dst, v_dst, true, stream);
}

libra_status libra_kv_copy_in(libra_kv_layout layout, const int32_t* page_ids, int64_t n_pages,
                              const void* k_src, const void* v_src, void* stream) {
  return page_copy(layout, page_ids, n_pages, k_src, v_src, false, stream);
}

libra_status libra_splitkv_plan(const libra_plan_desc* desc, const int32_t* seq_lens_host,
                                const int32_t* q_lens_host, const libra_plan_params* params,
                                libra_plan* out) {
  if (!out) return set_error(LIBRA_E_INVAL, "out is NULL");
  *out = nullptr;
  if (!desc) return set_error(LIBRA_E_INVAL, "plan descriptor is NULL");
  const libra_plan_desc& d = *desc;
  if (d.mode != LIBRA_MODE_DECODE && d.mode != LIBRA_MODE_APPEND)
    return set_error(LIBRA_E_INVAL, "mode must be LIBRA_MODE_DECODE or LIBRA_MODE_APPEND");
  if (d.batch < 0) return set_error(LIBRA_E_INVAL, "batch must be >= 0");
  if (d.num_kv_heads <= 0 || d.num_q_heads <= 0 || d.num_q_heads % d.num_kv_heads)
    return set_error(LIBRA_E_INVAL, "num_q_heads must be a positive multiple of num_kv_heads");
  const int G = d.num_q_heads / d.num_kv_heads;
  if (G > LIBRA_MAX_GROUP) return set_error(LIBRA_E_UNSUPPORTED, "num_q_heads / num_kv_heads > 16");
  if (d.batch > 0 && !seq_lens_host) return set_error(LIBRA_E_INVAL, "seq_lens_host is NULL");
  if (d.mode == LIBRA_MODE_DECODE && q_lens_host)
    return set_error(LIBRA_E_INVAL, "decode plans take q_lens_host = NULL");
  if (d.mode == LIBRA_MODE_APPEND && d.batch > 0 && !q_lens_host)
    return set_error(LIBRA_E_INVAL, "append plans need q_lens_host");

  libra_plan_params p{0, 3, 16, 64, 0, {0, 0, 0, 0, 0, 0, 0, 0}};
  if (params) p = *params;
  if (p.num_cus == 0) {
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_error(e, "querying the compute-unit count");
    p.num_cus = cus;
  }
  if (p.num_cus <= 0 || p.units_per_cu <= 0 || p.min_split_pages <= 0 || p.max_splits <= 0 ||
      p.q_tile < 0)
    return set_error(LIBRA_E_INVAL, "plan parameters must be positive");
  for (int x = 0; x < kNumXcds; ++x)
    if (p.xcd_weight[x] < 0 || p.xcd_weight[x] > 1000000)
      return set_error(LIBRA_E_INVAL, "xcd_weight entries must lie in [0, 1000000]");
  if (p.q_tile > kChunkRows / G)
    return set_error(LIBRA_E_UNSUPPORTED, "q_tile larger than floor(256 / G) tokens");

  auto* P = new (std::nothrow) libra_plan_s();
  if (!P) return set_error(LIBRA_E_NOMEM, "plan allocation failed");
  P->id = g_next_plan_id.fetch_add(1);
  libra_status st;
  try {
    st = build_plan(d, seq_lens_host, q_lens_host, p, P);
  } catch (const std::bad_alloc&) {
    st = set_error(LIBRA_E_NOMEM, "plan tables allocation failed");
  }
  if (st != LIBRA_OK) {
    delete P;
    return st;
  }
  // Pinned staging for the table upload, taken here so that no decode / append call
  // allocates.  Without a visible device (host-only use: inspecting a plan) there is none.
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) != hipSuccess || n_dev <= 0) {
    (void)hipGetLastError();
  } else {
    st = staging_acquire(*P);
    if (st == LIBRA_OK && P->fork_ev) st = ensure_aux_stream();
    if (st != LIBRA_OK) {
      staging_release(*P);
      delete P;
      return st;
    }
    staging_fill(*P);
  }
  *out = P;
  return LIBRA_OK;
}

libra_status libra_xcd_read_weights(const void* buf, size_t bytes, int32_t reps,
                                    int32_t* weights, void* stream) {
  if (!buf || !weights) return set_error(LIBRA_E_INVAL, "buf or weights is NULL");
  if (reinterpret_cast<uintptr_t>(buf) % kWorkspaceAlign)
    return set_error(LIBRA_E_INVAL, "buf must be 256-byte aligned");
  if (bytes < (size_t(1) << 30)) return set_error(LIBRA_E_INVAL, "buf must hold at least 1 GiB");
  if (reps < 1 || reps > 100) return set_error(LIBRA_E_INVAL, "reps must lie in [1, 100]");
  return measure_xcd_weights(buf, bytes, reps, weights, static_cast<hipStream_t>(stream));
}

libra_status libra_hbm_read_rate(const void* buf, size_t bytes, int32_t reps,
                                 double* interval_gbps, double* completion_gbps, void* stream) {
  if (!buf || !interval_gbps || !completion_gbps)
    return set_error(LIBRA_E_INVAL, "buf or an output is NULL");
  if (reinterpret_cast<uintptr_t>(buf) % kWorkspaceAlign)
    return set_error(LIBRA_E_INVAL, "buf must be 256-byte aligned");
  if (bytes < (size_t(1) << 28)) return set_error(LIBRA_E_INVAL, "buf must hold at least 256 MiB");
  if (reps < 1 || reps > 100) return set_error(LIBRA_E_INVAL, "reps must lie in [1, 100]");
  return measure_hbm_read_rate(buf, bytes, reps, interval_gbps, completion_gbps,
                               static_cast<hipStream_t>(stream));
}

libra_status libra_plan_get_units(libra_plan plan, const int32_t** units_host, int32_t* n_units) {
  if (!plan || !units_host || !n_units) return set_error(LIBRA_E_INVAL, "NULL argument");
  *units_host = plan->units.data();
  *n_units = plan->info.n_units;
  return LIBRA_OK;
}

libra_status libra_plan_get_info(libra_plan plan, libra_plan_info* info) {
  if (!plan || !info) return set_error(LIBRA_E_INVAL, "NULL argument");
  *info = plan->info;
  return LIBRA_OK;
}

size_t libra_plan_workspace_bytes(libra_plan plan) { return plan ? plan->ws_bytes : 0; }

libra_status libra_plan_upload(libra_plan plan, void* workspace, size_t ws_bytes, void* stream) {
  if (!plan) return set_error(LIBRA_E_INVAL, "plan is NULL");
  return upload(*plan, workspace, ws_bytes, static_cast<hipStream_t>(stream));
}

void libra_plan_destroy(libra_plan plan) {
  if (!plan) return;
  // The pinned image may still be the source of an enqueued copy: wait for that copy
  // (only it, not the device) before the image goes back to the pool.
  if (plan->upload_done) (void)hipEventSynchronize(plan->upload_done);
  {
    std::lock_guard<std::mutex> lk(g_ws.mu);
    for (auto it = g_ws.owner.begin(); it != g_ws.owner.end();)
      it = it->second == plan->id ? g_ws.owner.erase(it) : std::next(it);
  }
  staging_release(*plan);
  delete plan;
}

libra_status libra_decode_attn(libra_kv_layout layout, libra_plan plan, const void* q,
                               const int32_t* block_table, int32_t bt_stride, int32_t batch,
                               int32_t num_q_heads, float scale, void* workspace, size_t ws_bytes,
                               void* out, float* lse, void* stream) {
  libra_status st = check_call(layout, plan, LIBRA_MODE_DECODE, q, block_table, bt_stride, batch,
                               num_q_heads, scale, out);
  if (st != LIBRA_OK) return st;
  if (ws_bytes < plan->ws_bytes)
    return set_error(LIBRA_E_WORKSPACE, "workspace smaller than libra_plan_workspace_bytes");
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = upload(*plan, workspace, ws_bytes, s, false);
  if (st != LIBRA_OK) return st;
  return launch_attention(*layout, *plan, workspace, q, block_table, bt_stride, scale, out, lse, s);
}

libra_status libra_decode_attn_noalloc(libra_kv_layout layout, libra_plan plan, const void* q,
                                       const int32_t* block_table, int32_t bt_stride,
                                       int32_t batch, int32_t num_q_heads, float scale, void* out,
                                       float* lse, void* stream) {
  libra_status st = check_call(layout, plan, LIBRA_MODE_DECODE, q, block_table, bt_stride, batch,
                               num_q_heads, scale, out);
  if (st != LIBRA_OK) return st;
  if (plan->ws_bytes > scratch_capacity())
    return set_error(LIBRA_E_WORKSPACE,
                     "the plan needs " + std::to_string(plan->ws_bytes) +
                         " bytes of scratch; the static scratch holds " +
                         std::to_string(scratch_capacity()) +
                         " bytes (libra_decode_attn takes a workspace of any size)");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchOwners)
    return set_error(LIBRA_E_UNSUPPORTED, "device ordinal outside the scratch table (64 devices)");
  void* ws = nullptr;
  st = scratch_buffer(dev, &ws);
  if (st != LIBRA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    std::lock_guard<std::mutex> lk(plan->upload_mu);
    if (g_scratch_owner[dev].load() != plan->id) {
      st = enqueue_tables(*plan, ws, s);
      if (st != LIBRA_OK) return st;
      g_scratch_owner[dev].store(plan->id);
    }
  }
  return launch_attention(*layout, *plan, ws, q, block_table, bt_stride, scale, out, lse, s,
                          /*timed=*/false);
}

libra_status libra_append_attn(libra_kv_layout layout, libra_plan plan, const void* q,
                               const void* k_new, const void* v_new, const int32_t* block_table,
                               int32_t bt_stride, int32_t batch, int32_t num_q_heads, float scale,
                               void* workspace, size_t ws_bytes, void* out, float* lse,
                               void* stream) {
  libra_status st = check_call(layout, plan, LIBRA_MODE_APPEND, q, block_table, bt_stride, batch,
                               num_q_heads, scale, out);
  if (st != LIBRA_OK) return st;
  if (plan->info.n_rows > 0) {
    if (!k_new || !v_new) return set_error(LIBRA_E_INVAL, "k_new / v_new is NULL");
    if (!aligned16(k_new) || !aligned16(v_new))
      return set_error(LIBRA_E_INVAL, "k_new / v_new must be 16-byte aligned");
  }
  if (ws_bytes < plan->ws_bytes)
    return set_error(LIBRA_E_WORKSPACE, "workspace smaller than libra_plan_workspace_bytes");
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = upload(*plan, workspace, ws_bytes, s, false);
  if (st != LIBRA_OK) return st;
  hipError_t e;
  {
    ProfScope ps(LIBRA_KERNEL_CACHE_WRITE, s, plan->info.n_write_tiles > 0);
    e = launch_cache_write(*layout, *plan, workspace, k_new, v_new, block_table, bt_stride, s);
  }
  if (e != hipSuccess) return hip_error(e, "cache-write launch");
  return launch_attention(*layout, *plan, workspace, q, block_table, bt_stride, scale, out, lse, s);
}

libra_status libra_profile_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.enabled = enable != 0;
  return LIBRA_OK;
}

libra_status libra_profile_collect(libra_kernel_times* out) {
  if (!out) return set_error(LIBRA_E_INVAL, "out is NULL");
  std::memset(out, 0, sizeof(*out));
  std::lock_guard<std::mutex> lk(g_prof.mu);
  libra_status st = LIBRA_OK;
  for (const Profiler::Rec& r : g_prof.pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess && st == LIBRA_OK) st = hip_error(e, "reading kernel timing events");
    out->ms[r.kind] += ms;
    out->launches[r.kind] += 1;
    g_prof.free_events.push_back(r.a);
    g_prof.free_events.push_back(r.b);
  }
  g_prof.pending.clear();
  return st;
}

}  // extern "C"
