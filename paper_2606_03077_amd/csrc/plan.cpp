// Host construction of the split-KV work plan (rule documented in include/libra.h).
#include <algorithm>
#include <array>
#include <cstring>
#include <queue>

#include "internal.h"

namespace libra {
namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

using Unit = std::array<int32_t, kUnitInts>;

// Rule step 4: split counts that cut the single rows into at most R pieces per KV head
// with the smallest possible largest piece.  Each extra split goes to the row with the
// largest share pages_b / n_b (exact cross-multiplied comparison, ties to the smaller b)
// among the rows that can still be split; a row that cannot be split now never can, as
// only its own split count would change that.  Returns false (nsplit untouched) when the
// rows do not fit in R or the largest piece exceeds 1.5 times the mean share.
bool one_wave_splits(const std::vector<int64_t>& pages, const std::vector<int64_t>& single,
                     int64_t R, const libra_plan_params& p, std::vector<int64_t>& nsplit) {
  if (single.empty() || int64_t(single.size()) > R) return false;
  std::vector<int64_t> n(pages.size(), 1);
  auto before = [&](int64_t a, int64_t b) {  // true if row a's share is served after b's
    const int64_t lhs = pages[a] * n[b], rhs = pages[b] * n[a];
    if (lhs != rhs) return lhs < rhs;
    return a > b;
  };
  std::priority_queue<int64_t, std::vector<int64_t>, decltype(before)> heap(before);
  for (int64_t b : single) heap.push(b);
  int64_t total = int64_t(single.size());
  while (total < R && !heap.empty()) {
    const int64_t b = heap.top();
    heap.pop();
    if (n[b] >= p.max_splits || pages[b] < (n[b] + 1) * int64_t(p.min_split_pages)) continue;
    ++n[b];
    ++total;
    heap.push(b);
  }
  int64_t largest = 0, sum = 0;
  for (int64_t b : single) {
    largest = std::max(largest, ceil_div(pages[b], n[b]));
    sum += pages[b];
  }
  if (__int128(2) * largest * R > __int128(3) * sum) return false;
  for (int64_t b : single) nsplit[b] = n[b];
  return true;
}

// Rule step 11: the units (in step 9's order) are dealt to S slots, each to the slot with
// room that minimises (load + cost) / weight; the r-th unit of slot c is listed at position
// c + r * S.  Slots of one XCD share a weight, so one min-heap of (load, c) per XCD yields
// that XCD's best slot and the eight candidates are compared exactly; this picks the same
// slot as a scan over all of them.
std::vector<Unit> place_on_slots(const std::vector<Unit>& units, const libra_plan_params& p,
                                 int64_t S) {
  const int64_t n = int64_t(units.size());
  auto weight = [&](int64_t c) -> int64_t {
    const int32_t x = p.xcd_weight[c % kNumXcds];
    return x > 0 ? x : 1000;
  };
  auto cap = [&](int64_t c) { return c < n ? (n - 1 - c) / S + 1 : int64_t(0); };
  using Entry = std::pair<int64_t, int64_t>;  // (load, slot)
  std::array<std::priority_queue<Entry, std::vector<Entry>, std::greater<Entry>>, kNumXcds> heaps;
  for (int64_t c = 0; c < std::min(S, n); ++c) heaps[c % kNumXcds].push({0, c});
  std::vector<int64_t> taken(size_t(std::min(S, n)), 0);
  std::vector<Unit> out(units.size());
  for (const Unit& u : units) {
    const int64_t cost = ceil_div(u[U_KV1], kPage) - u[U_KV0] / kPage;
    int best = -1;
    Entry be{0, 0};
    for (int k = 0; k < kNumXcds; ++k) {
      if (heaps[k].empty()) continue;
      const Entry e = heaps[k].top();
      if (best >= 0) {
        const __int128 lhs = __int128(e.first + cost) * weight(be.second);
        const __int128 rhs = __int128(be.first + cost) * weight(e.second);
        if (lhs > rhs || (lhs == rhs && e.second > be.second)) continue;
      }
      best = k;
      be = e;
    }
    heaps[best].pop();
    const int64_t c = be.second;
    out[size_t(c + taken[c] * S)] = u;
    if (++taken[c] < cap(c)) heaps[best].push({be.first + cost, c});
  }
  return out;
}

}  // namespace

libra_status build_plan(const libra_plan_desc& d, const int32_t* seq_lens, const int32_t* q_lens,
                        const libra_plan_params& p, Plan* out) {
  const int64_t B = d.batch;
  const int64_t Hkv = d.num_kv_heads;
  const int64_t G = d.num_q_heads / d.num_kv_heads;
  const bool append = d.mode == LIBRA_MODE_APPEND;

  std::vector<int64_t> L(B), C(B), pages(B), row0(B);
  int64_t rows = 0;
  for (int64_t b = 0; b < B; ++b) {
    L[b] = seq_lens[b];
    C[b] = append ? q_lens[b] : 1;
    if (L[b] < 0) return set_error(LIBRA_E_INVAL, "seq_lens must be >= 0");
    if (append && (C[b] < 1 || C[b] > L[b]))
      return set_error(LIBRA_E_INVAL, "append needs 1 <= q_lens[b] <= seq_lens[b]");
    pages[b] = ceil_div(L[b], kPage);
    row0[b] = rows;
    rows += C[b];
  }
  if (rows > INT32_MAX) return set_error(LIBRA_E_INVAL, "too many query rows");

  // Steps 3-5: one wave of S units per KV head if the single rows can fill it evenly,
  // else the chunk rule.
  std::vector<int64_t> single;
  int64_t W = 0;
  for (int64_t b = 0; b < B; ++b)
    if (C[b] == 1) {
      single.push_back(b);
      W += pages[b] * Hkv;
    }
  const int64_t S = int64_t(p.num_cus) * p.units_per_cu;
  const int64_t chunk = W > 0 ? std::max<int64_t>(p.min_split_pages, ceil_div(W, S))
                              : int64_t(p.min_split_pages);
  std::vector<int64_t> nsplit(B, 1), slot_base(B, -1);
  const bool balanced = one_wave_splits(pages, single, S / Hkv, p, nsplit);
  if (!balanced)
    for (int64_t b : single)
      nsplit[b] = std::min<int64_t>(p.max_splits, std::max<int64_t>(1, ceil_div(pages[b], chunk)));

  // Step 10: partial slots in ascending (b, g).
  int64_t slots = 0;
  for (int64_t b : single) {
    if (nsplit[b] > 1) {
      slot_base[b] = slots;
      slots += nsplit[b] * Hkv;
    }
  }
  if (slots > INT32_MAX) return set_error(LIBRA_E_INVAL, "too many partial slots");

  std::vector<Unit> singles, chunks;
  for (int64_t b = 0; b < B; ++b) {
    if (C[b] != 1) continue;
    const int64_t n = nsplit[b];
    for (int64_t g = 0; g < Hkv; ++g) {
      for (int64_t j = 0; j < n; ++j) {
        const int64_t p0 = (j * pages[b]) / n, p1 = ((j + 1) * pages[b]) / n;
        Unit u{};
        u[U_B] = int32_t(b);
        u[U_G] = int32_t(g);
        u[U_KV0] = int32_t(kPage * p0);
        u[U_KV1] = int32_t(std::min<int64_t>(kPage * p1, L[b]));
        u[U_Q0] = 0;
        u[U_Q1] = 1;
        u[U_SPLIT] = int32_t(j);
        u[U_NSPLIT] = int32_t(n);
        u[U_PART] = n > 1 ? int32_t(slot_base[b] + g * n) : -1;
        u[U_ROW0] = int32_t(row0[b]);
        u[U_KIND] = kKindSingle;
        u[U_PRIOR] = int32_t(L[b] - 1);
        singles.push_back(u);
      }
    }
  }
  std::sort(singles.begin(), singles.end(), [](const Unit& x, const Unit& y) {
    const int64_t tx = x[U_KV1] - x[U_KV0], ty = y[U_KV1] - y[U_KV0];
    if (tx != ty) return tx > ty;
    if (x[U_B] != y[U_B]) return x[U_B] < y[U_B];
    if (x[U_G] != y[U_G]) return x[U_G] < y[U_G];
    return x[U_SPLIT] < y[U_SPLIT];
  });
  if (!singles.empty())  // step 11: CU slots for one wave, else the XCD queues
    singles = place_on_slots(singles, p, balanced ? int64_t(p.num_cus) : int64_t(kNumXcds));

  // Step 7: query tiles of chunk rows.
  const int64_t T = p.q_tile > 0 ? p.q_tile : int64_t(kChunkRows) / G;
  for (int64_t b = 0; b < B; ++b) {
    if (C[b] == 1) continue;
    const int64_t P = L[b] - C[b];
    for (int64_t g = 0; g < Hkv; ++g) {
      for (int64_t q0 = 0; q0 < C[b]; q0 += T) {
        const int64_t q1 = std::min(q0 + T, C[b]);
        Unit u{};
        u[U_B] = int32_t(b);
        u[U_G] = int32_t(g);
        u[U_KV0] = 0;
        u[U_KV1] = int32_t(P + q1);
        u[U_Q0] = int32_t(q0);
        u[U_Q1] = int32_t(q1);
        u[U_SPLIT] = 0;
        u[U_NSPLIT] = 1;
        u[U_PART] = -1;
        u[U_ROW0] = int32_t(row0[b]);
        u[U_KIND] = kKindChunk;
        u[U_PRIOR] = int32_t(P);
        chunks.push_back(u);
      }
    }
  }
  // Step 9 (chunk units): XCD-affine order.  Tiles of one (b, g) read the same keys, so
  // they are kept on one XCD (workgroup w runs on XCD w % kNumXcds) to share its L2,
  // unless the group costs more than an eighth of the launch: it is then cut into
  // contiguous, cost-balanced parts so that every XCD gets work.  Parts by descending
  // cost (ties ascending (b, g, part)) are dealt to the XCD queue with the least
  // accumulated cost (ties to the lowest queue); each queue then lists its parts by
  // descending cost of their longest tile, a part's tiles together and longest first (so
  // the last tiles a CU takes are short, and the tiles that read the same keys run
  // together); queues are listed one after another.  A tile costs its key-loop steps: the kernel spends the
  // same time on a step whatever the number of the tile's query tokens.
  auto cost = [](const Unit& u) { return ceil_div(u[U_KV1] - u[U_KV0], kChunkStepKeys); };
  int64_t total_cost = 0;
  for (const Unit& u : chunks) total_cost += cost(u);
  const int64_t fair = std::max<int64_t>(1, ceil_div(total_cost, kNumXcds));
  struct Part { int64_t cost; int32_t b, g, idx; size_t first, last; };  // [first, last) in part_tiles
  std::vector<Part> parts;
  std::vector<Unit> part_tiles;  // chunks regrouped part by part
  part_tiles.reserve(chunks.size());
  for (size_t i = 0; i < chunks.size();) {  // chunks are built in ascending (b, g, q_begin)
    size_t j = i + 1;
    while (j < chunks.size() && chunks[j][U_B] == chunks[i][U_B] && chunks[j][U_G] == chunks[i][U_G]) ++j;
    int64_t c = 0;
    for (size_t k = i; k < j; ++k) c += cost(chunks[k]);
    const int64_t n = std::min<int64_t>(int64_t(j - i), ceil_div(c, fair));
    int64_t before = 0, cur = -1;
    for (size_t k = i; k < j; ++k) {
      const int64_t idx = int64_t(__int128(before) * n / c);
      if (idx != cur) {
        parts.push_back(Part{0, chunks[k][U_B], chunks[k][U_G], int32_t(idx), part_tiles.size(),
                             part_tiles.size()});
        cur = idx;
      }
      parts.back().cost += cost(chunks[k]);
      parts.back().last += 1;
      part_tiles.push_back(chunks[k]);
      before += cost(chunks[k]);
    }
    i = j;
  }
  std::vector<size_t> porder(parts.size());
  for (size_t k = 0; k < porder.size(); ++k) porder[k] = k;
  std::sort(porder.begin(), porder.end(), [&](size_t a, size_t b) {
    const Part &x = parts[a], &y = parts[b];
    if (x.cost != y.cost) return x.cost > y.cost;
    if (x.b != y.b) return x.b < y.b;
    if (x.g != y.g) return x.g < y.g;
    return x.idx < y.idx;
  });
  // Deal the parts; then each queue lists its parts by descending cost of their longest
  // tile (ties ascending (b, g, part)), a part's tiles together, by descending cost (ties
  // ascending q_begin).
  std::vector<std::vector<size_t>> qparts(kNumXcds);
  int64_t qcost[kNumXcds] = {0};
  for (size_t k : porder) {
    int x = 0;
    for (int y = 1; y < kNumXcds; ++y)
      if (qcost[y] < qcost[x]) x = y;
    qcost[x] += parts[k].cost;
    qparts[x].push_back(k);
  }
  auto tile_order = [&](const Unit& a, const Unit& b) {
    const int64_t ca = cost(a), cb = cost(b);
    if (ca != cb) return ca > cb;
    return a[U_Q0] < b[U_Q0];
  };
  std::vector<int64_t> longest_tile(parts.size(), 0);
  for (size_t k = 0; k < parts.size(); ++k) {
    std::sort(part_tiles.begin() + parts[k].first, part_tiles.begin() + parts[k].last, tile_order);
    longest_tile[k] = cost(part_tiles[parts[k].first]);
  }
  std::vector<std::vector<Unit>> queues(kNumXcds);
  for (int x = 0; x < kNumXcds; ++x) {
    std::sort(qparts[x].begin(), qparts[x].end(), [&](size_t a, size_t b) {
      if (longest_tile[a] != longest_tile[b]) return longest_tile[a] > longest_tile[b];
      const Part &pa = parts[a], &pb = parts[b];
      if (pa.b != pb.b) return pa.b < pb.b;
      if (pa.g != pb.g) return pa.g < pb.g;
      return pa.idx < pb.idx;
    });
    for (size_t k : qparts[x])
      queues[x].insert(queues[x].end(), part_tiles.begin() + parts[k].first,
                       part_tiles.begin() + parts[k].last);
  }
  chunks.clear();
  int32_t xcd_map[2 * kNumXcds];
  int32_t longest = 0;
  for (int x = 0; x < kNumXcds; ++x) {
    xcd_map[2 * x] = int32_t(chunks.size());
    xcd_map[2 * x + 1] = int32_t(queues[x].size());
    longest = std::max<int32_t>(longest, int32_t(queues[x].size()));
    chunks.insert(chunks.end(), queues[x].begin(), queues[x].end());
  }

  Plan& P = *out;
  P.mode = d.mode;
  P.batch = d.batch;
  P.num_q_heads = d.num_q_heads;
  P.num_kv_heads = d.num_kv_heads;
  P.group = int32_t(G);
  P.params = p;
  P.units.clear();
  P.units.reserve((singles.size() + chunks.size()) * kUnitInts);
  for (const Unit& u : singles) P.units.insert(P.units.end(), u.begin(), u.end());
  for (const Unit& u : chunks) P.units.insert(P.units.end(), u.begin(), u.end());

  // Cache-write table (append): every (sequence, page) holding new positions [P_b, L_b).
  P.writes.clear();
  if (append) {
    for (int64_t b = 0; b < B; ++b) {
      const int64_t P0 = L[b] - C[b];
      for (int64_t pg = P0 / kPage; pg * kPage < L[b]; ++pg) {
        const int64_t s0 = std::max<int64_t>(P0, pg * kPage) - pg * kPage;
        const int64_t s1 = std::min<int64_t>(L[b], pg * kPage + kPage) - pg * kPage;
        const int32_t rec[kWriteInts] = {int32_t(b), int32_t(pg), int32_t(s0), int32_t(s1),
                                         int32_t(row0[b] + pg * kPage + s0 - P0), 0, 0, 0};
        P.writes.insert(P.writes.end(), rec, rec + kWriteInts);
      }
    }
  }

  P.xcd_map.assign(xcd_map, xcd_map + 2 * kNumXcds);
  P.chunk_grid = int64_t(kNumXcds) * longest;

  // Split-merge table: every single row with n_b > 1, per KV head, ascending (b, g).
  P.merges.clear();
  for (int64_t b = 0; b < B; ++b) {
    if (C[b] != 1 || nsplit[b] <= 1) continue;
    for (int64_t g = 0; g < Hkv; ++g) {
      const int32_t rec[kMergeInts] = {int32_t(b), int32_t(g), int32_t(nsplit[b]),
                                       int32_t(slot_base[b] + g * nsplit[b]), int32_t(row0[b]),
                                       0, 0, 0};
      P.merges.insert(P.merges.end(), rec, rec + kMergeInts);
    }
  }

  // Block-table columns the kernels read: every unit's pages and every written page.
  P.pages_needed = 0;
  for (size_t i = 0; i < P.units.size(); i += kUnitInts)
    P.pages_needed = std::max<int64_t>(P.pages_needed, ceil_div(P.units[i + U_KV1], kPage));
  for (size_t i = 0; i < P.writes.size(); i += kWriteInts)
    P.pages_needed = std::max<int64_t>(P.pages_needed, int64_t(P.writes[i + W_PAGE]) + 1);

  libra_plan_info& I = P.info;
  std::memset(&I, 0, sizeof(I));
  I.n_single = int32_t(singles.size());
  I.n_chunk = int32_t(chunks.size());
  I.n_units = I.n_single + I.n_chunk;
  I.n_partial_slots = int32_t(slots);
  I.chunk_pages = chunk;
  I.q_tile = int32_t(T);
  I.n_rows = int32_t(rows);
  I.n_write_tiles = int32_t(P.writes.size() / kWriteInts);
  I.num_cus = p.num_cus;
  I.n_merge_groups = int32_t(P.merges.size() / kMergeInts);
  I.balanced = balanced ? 1 : 0;

  size_t off = 0;
  P.off_units = off;
  off = align256(off + P.units.size() * sizeof(int32_t));
  P.off_writes = off;
  off = align256(off + P.writes.size() * sizeof(int32_t));
  P.off_merges = off;
  off = align256(off + P.merges.size() * sizeof(int32_t));
  P.off_xcd_map = off;
  off = align256(off + P.xcd_map.size() * sizeof(int32_t));
  P.upload_bytes = off;
  P.off_part_o = off;
  off = align256(off + size_t(slots) * size_t(G) * kDim * sizeof(float));
  P.off_part_lse = off;
  off = align256(off + size_t(slots) * size_t(G) * sizeof(float));
  P.ws_bytes = std::max<size_t>(off, 256);
  return LIBRA_OK;
}

}  // namespace libra
