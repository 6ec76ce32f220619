// Host-side head reshard of offloaded KV pages (Sec. 5, migration Step 2).
//
// An offloaded request is a packed page run per shard: page i's tiles for the shard's
// heads, back to back, 4096 bytes per (page, head) tile (the library tile layout, which
// does not depend on how many heads a cache holds).  Resharding along heads therefore
// only regroups whole tiles: the copy for page i takes each maximal head range that lies
// in one source shard and one destination shard as a single memcpy.  Pages are split
// across a few host threads when the run is large.
#include <algorithm>
#include <cstring>
#include <thread>
#include <vector>

#include "internal.h"

namespace libra {
namespace {


void reshard_pages(const char* const* src, int hs, char* const* dst, int hd, int heads,
                   int64_t p0, int64_t p1) {
  for (int64_t p = p0; p < p1; ++p) {
    int h = 0;
    while (h < heads) {
      const int i = h / hs, j = h / hd;
      const int run = std::min((i + 1) * hs, (j + 1) * hd) - h;
      std::memcpy(dst[j] + (size_t(p) * hd + (h - j * hd)) * kTileBytes,
                  src[i] + (size_t(p) * hs + (h - i * hs)) * kTileBytes, size_t(run) * kTileBytes);
      h += run;
    }
  }
}

bool overlaps(const char* a, size_t na, const char* b, size_t nb) {
  return a < b + nb && b < a + na;
}

}  // namespace
}  // namespace libra

using namespace libra;

extern "C" libra_status libra_kv_reshard_host(const void* const* src, int32_t n_src,
                                              int32_t heads_per_src, void* const* dst,
                                              int32_t n_dst, int64_t n_pages) {
  if (!src || !dst) return set_error(LIBRA_E_INVAL, "src / dst array is NULL");
  if (n_src <= 0 || n_dst <= 0 || heads_per_src <= 0)
    return set_error(LIBRA_E_INVAL, "n_src, n_dst and heads_per_src must be > 0");
  if (n_pages < 0) return set_error(LIBRA_E_INVAL, "n_pages < 0");
  const int64_t heads64 = int64_t(n_src) * heads_per_src;
  if (heads64 > 65536) return set_error(LIBRA_E_INVAL, "too many heads");
  const int heads = int(heads64);
  if (heads % n_dst != 0) return set_error(LIBRA_E_INVAL, "n_dst must divide the head count");
  const int hd = heads / n_dst;
  const int64_t max_pages = int64_t(1) << 40;
  if (n_pages > max_pages / (int64_t(heads) * int64_t(kTileBytes)))
    return set_error(LIBRA_E_INVAL, "n_pages too large");
  if (n_pages == 0) return LIBRA_OK;
  std::vector<const char*> s(n_src);
  std::vector<char*> d(n_dst);
  const size_t ns = size_t(n_pages) * heads_per_src * kTileBytes;
  const size_t nd = size_t(n_pages) * hd * kTileBytes;
  for (int i = 0; i < n_src; ++i) {
    if (!src[i]) return set_error(LIBRA_E_INVAL, "a source buffer is NULL");
    s[i] = static_cast<const char*>(src[i]);
  }
  for (int j = 0; j < n_dst; ++j) {
    if (!dst[j]) return set_error(LIBRA_E_INVAL, "a destination buffer is NULL");
    d[j] = static_cast<char*>(dst[j]);
    for (int i = 0; i < n_src; ++i)
      if (overlaps(d[j], nd, s[i], ns)) return set_error(LIBRA_E_INVAL, "buffers overlap");
    for (int k = 0; k < j; ++k)
      if (overlaps(d[j], nd, d[k], nd)) return set_error(LIBRA_E_INVAL, "buffers overlap");
  }
  // Threads only pay off for runs of tens of MiB; each takes a contiguous page range.
  const size_t total = size_t(n_pages) * heads * kTileBytes;
  const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
  const int64_t nthreads =
      std::min<int64_t>({int64_t(std::min(hw, 8u)), n_pages, int64_t(total >> 24) + 1});
  if (nthreads <= 1) {
    reshard_pages(s.data(), heads_per_src, d.data(), hd, heads, 0, n_pages);
    return LIBRA_OK;
  }
  std::vector<std::thread> pool;
  pool.reserve(size_t(nthreads));
  for (int64_t t = 0; t < nthreads; ++t) {
    const int64_t p0 = n_pages * t / nthreads, p1 = n_pages * (t + 1) / nthreads;
    try {
      pool.emplace_back(reshard_pages, s.data(), heads_per_src, d.data(), hd, heads, p0, p1);
    } catch (...) {  // no thread available: do this range here
      reshard_pages(s.data(), heads_per_src, d.data(), hd, heads, p0, p1);
    }
  }
  for (auto& th : pool) th.join();
  return LIBRA_OK;
}
