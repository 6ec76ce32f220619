// Causality-guided bucket routing on the host (Sec. 5): the prefix tree over tool-return
// histories with residual-length histograms, and the per-tool-return bucket choice.
#include <cmath>
#include <limits>
#include <new>
#include <unordered_map>
#include <vector>

#include "internal.h"

namespace libra {
namespace {

struct TrieNode {
  std::vector<int64_t> counts;                 // per residual-length bin
  int64_t total = 0;
  std::unordered_map<int32_t, int32_t> next;   // tool state -> child node
};

}  // namespace

struct Trie {
  std::vector<int64_t> edges;
  std::vector<TrieNode> nodes;                  // nodes[0] is the root above all prompts
  std::unordered_map<int64_t, int32_t> prompts; // prompt id -> prompt node

  int bins() const { return int(edges.size()) + 1; }

  int bin_of(int64_t residual) const {
    int k = 0;
    while (k < int(edges.size()) && residual >= edges[k]) ++k;
    return k;
  }

  int32_t add_node() {
    nodes.emplace_back();
    nodes.back().counts.assign(size_t(bins()), 0);
    return int32_t(nodes.size() - 1);
  }

  void record(int32_t node, int64_t residual) {
    nodes[node].counts[bin_of(residual)] += 1;
    nodes[node].total += 1;
  }
};

}  // namespace libra

using namespace libra;

struct libra_trie_s : Trie {};

extern "C" {

libra_status libra_trie_create(const int64_t* bin_edges, int32_t n_edges, libra_trie* out) {
  if (!out) return set_error(LIBRA_E_INVAL, "out is NULL");
  if (n_edges < 0 || n_edges > 63) return set_error(LIBRA_E_INVAL, "n_edges must be in [0, 63]");
  if (n_edges > 0 && !bin_edges) return set_error(LIBRA_E_INVAL, "bin_edges is NULL");
  for (int32_t i = 0; i < n_edges; ++i) {
    if (bin_edges[i] <= 0) return set_error(LIBRA_E_INVAL, "bin edges must be > 0");
    if (i > 0 && bin_edges[i] <= bin_edges[i - 1])
      return set_error(LIBRA_E_INVAL, "bin edges must increase strictly");
  }
  libra_trie_s* t = new (std::nothrow) libra_trie_s();
  if (!t) return set_error(LIBRA_E_NOMEM, "trie allocation failed");
  try {
    t->edges.assign(bin_edges, bin_edges + n_edges);
    t->add_node();
  } catch (const std::bad_alloc&) {
    delete t;
    return set_error(LIBRA_E_NOMEM, "trie allocation failed");
  }
  *out = t;
  return LIBRA_OK;
}

void libra_trie_destroy(libra_trie trie) { delete trie; }

libra_status libra_trie_insert(libra_trie trie, int64_t prompt_id, const int32_t* states,
                               int32_t n_states, const int64_t* residual) {
  if (!trie || !residual || (n_states > 0 && !states))
    return set_error(LIBRA_E_INVAL, "NULL argument");
  if (n_states < 0) return set_error(LIBRA_E_INVAL, "n_states < 0");
  for (int32_t k = 0; k <= n_states; ++k)
    if (residual[k] < 0) return set_error(LIBRA_E_INVAL, "residual lengths must be >= 0");
  try {
    trie->record(0, residual[0]);
    auto it = trie->prompts.find(prompt_id);
    int32_t node;
    if (it == trie->prompts.end()) {
      node = trie->add_node();
      trie->prompts.emplace(prompt_id, node);
    } else {
      node = it->second;
    }
    trie->record(node, residual[0]);
    for (int32_t k = 0; k < n_states; ++k) {
      auto c = trie->nodes[node].next.find(states[k]);
      int32_t child;
      if (c == trie->nodes[node].next.end()) {
        child = trie->add_node();
        trie->nodes[node].next.emplace(states[k], child);
      } else {
        child = c->second;
      }
      node = child;
      trie->record(node, residual[k + 1]);
    }
  } catch (const std::bad_alloc&) {
    return set_error(LIBRA_E_NOMEM, "trie insertion ran out of memory");
  }
  return LIBRA_OK;
}

libra_status libra_trie_lookup(libra_trie trie, int64_t prompt_id, const int32_t* states,
                               int32_t n_states, double* hist, int32_t* depth) {
  if (!trie || !hist || !depth || (n_states > 0 && !states))
    return set_error(LIBRA_E_INVAL, "NULL argument");
  if (n_states < 0) return set_error(LIBRA_E_INVAL, "n_states < 0");
  if (trie->nodes[0].total == 0) return set_error(LIBRA_E_INVAL, "the tree is empty");
  int32_t node = 0, d = -1;
  auto it = trie->prompts.find(prompt_id);
  if (it != trie->prompts.end()) {
    node = it->second;
    d = 0;
    for (int32_t k = 0; k < n_states; ++k) {
      auto c = trie->nodes[node].next.find(states[k]);
      if (c == trie->nodes[node].next.end()) break;  // unseen: keep the parent
      node = c->second;
      d = k + 1;
    }
  }
  const TrieNode& n = trie->nodes[node];
  for (int k = 0; k < trie->bins(); ++k) hist[k] = double(n.counts[k]) / double(n.total);
  *depth = d;
  return LIBRA_OK;
}

libra_status libra_route_bucket(const double* hist, int32_t n_bins, const double* t_dec,
                                const double* c_mig, int32_t n_buckets, int32_t current,
                                int32_t* best, double* best_cost) {
  if (!hist || !t_dec || !c_mig || !best || !best_cost)
    return set_error(LIBRA_E_INVAL, "NULL argument");
  if (n_bins < 1 || n_buckets < 1) return set_error(LIBRA_E_INVAL, "n_bins and n_buckets must be > 0");
  if (current < 0 || current >= n_buckets) return set_error(LIBRA_E_INVAL, "current bucket out of range");
  int32_t arg = -1;
  double lo = std::numeric_limits<double>::infinity();
  for (int32_t b = 0; b < n_buckets; ++b) {
    double c = 0.0;
    for (int32_t k = 0; k < n_bins; ++k) c += hist[k] * t_dec[size_t(b) * n_bins + k];
    if (b != current) c += c_mig[size_t(current) * n_buckets + b];
    if (std::isnan(c)) return set_error(LIBRA_E_INVAL, "NaN cost");
    if (arg < 0 || c < lo) {
      lo = c;
      arg = b;
    }
  }
  *best = arg;
  *best_cost = lo;
  return LIBRA_OK;
}

}  // extern "C"
