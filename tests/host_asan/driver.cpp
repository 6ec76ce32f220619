// Host-side fuzz of the library's CPU entry points under AddressSanitizer and
// UndefinedBehaviorSanitizer: split plans, head reshard, cost-evaluator fits and sums,
// RolloutDP (literal and crossing search), the prefix tree and bucket routing.  Inputs
// are seeded; results are checked only for internal consistency here (the Python tests
// compare them with the oracle).  Exits non-zero on the first inconsistency.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "libra.h"

#define CHECK(cond)                                                         \
  do {                                                                      \
    if (!(cond)) {                                                          \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      return 1;                                                             \
    }                                                                       \
  } while (0)

int main() {
  std::mt19937_64 rng(2606);
  auto uni = [&](int64_t lo, int64_t hi) {
    return std::uniform_int_distribution<int64_t>(lo, hi)(rng);
  };

  // Split plans: random batches, decode and append, random parameters.
  for (int it = 0; it < 300; ++it) {
    const int B = int(uni(0, 40));
    const int hkv = int(uni(1, 8));
    const int G = int(uni(1, 16));
    std::vector<int32_t> L(B), C(B);
    for (int b = 0; b < B; ++b) {
      L[b] = int32_t(uni(0, 3) == 0 ? uni(0, 40) : uni(1, 70000));
      C[b] = int32_t(std::max<int64_t>(1, std::min<int64_t>(L[b], uni(0, 2) ? 1 : uni(1, 3000))));
      if (L[b] == 0) C[b] = 1;
    }
    const bool append = it % 2;
    if (append)
      for (int b = 0; b < B; ++b)
        if (L[b] == 0) L[b] = 1;
    libra_plan_desc d{append ? LIBRA_MODE_APPEND : LIBRA_MODE_DECODE, B, hkv * G, hkv};
    const int tpb = G >= 16 ? 1 : 16 / G;
    libra_plan_params p{int32_t(uni(1, 512)), int32_t(uni(1, 8)), int32_t(uni(1, 64)),
                        int32_t(uni(1, 128)), int32_t(uni(0, 1) ? 0 : uni(1, 16 * tpb))};
    for (int x = 0; x < 8; ++x) p.xcd_weight[x] = int32_t(uni(0, 3) == 0 ? 0 : uni(1, 1000000));
    libra_plan plan = nullptr;
    const libra_status st = libra_splitkv_plan(&d, L.data(), append ? C.data() : nullptr, &p, &plan);
    if (st != LIBRA_OK) continue;
    const int32_t* units = nullptr;
    int32_t n = 0;
    CHECK(libra_plan_get_units(plan, &units, &n) == LIBRA_OK);
    libra_plan_info info{};
    CHECK(libra_plan_get_info(plan, &info) == LIBRA_OK);
    CHECK(info.n_units == n && info.n_single + info.n_chunk == n);
    int64_t sum = 0;
    for (int i = 0; i < n; ++i) sum ^= units[i * LIBRA_UNIT_INTS + 3];
    (void)sum;
    for (int i = 0; i < info.n_single; ++i)  // every slot position holds a real unit
      CHECK(units[i * LIBRA_UNIT_INTS + 7] >= 1 && units[i * LIBRA_UNIT_INTS + 10] == 0);
    CHECK(libra_plan_workspace_bytes(plan) >= 256);
    libra_plan_destroy(plan);
  }

  // Head reshard: random shard counts, compared with a direct tile walk.
  for (int it = 0; it < 60; ++it) {
    const int n_src = int(uni(1, 4)), hps = int(uni(1, 4));
    const int H = n_src * hps;
    std::vector<int> divs;
    for (int x = 1; x <= H; ++x)
      if (H % x == 0) divs.push_back(x);
    const int n_dst = divs[size_t(uni(0, int64_t(divs.size()) - 1))];
    const int64_t pages = uni(0, 9);
    const size_t tile = 4096;
    std::vector<std::vector<unsigned char>> src(n_src), dst(n_dst);
    std::vector<const void*> sp(n_src);
    std::vector<void*> dp(n_dst);
    for (int i = 0; i < n_src; ++i) {
      src[i].resize(size_t(pages) * hps * tile + 1);
      for (auto& c : src[i]) c = static_cast<unsigned char>(rng());
      sp[i] = src[i].data();
    }
    const int hd = H / n_dst;
    for (int j = 0; j < n_dst; ++j) {
      dst[j].assign(size_t(pages) * hd * tile + 1, 0);
      dp[j] = dst[j].data();
    }
    CHECK(libra_kv_reshard_host(sp.data(), n_src, hps, dp.data(), n_dst, pages) == LIBRA_OK);
    for (int64_t pg = 0; pg < pages; ++pg)
      for (int h = 0; h < H; ++h) {
        const unsigned char* a = src[h / hps].data() + (size_t(pg) * hps + h % hps) * tile;
        const unsigned char* b = dst[h / hd].data() + (size_t(pg) * hd + h % hd) * tile;
        CHECK(std::memcmp(a, b, tile) == 0);
      }
  }

  // Cost evaluator.
  for (int it = 0; it < 200; ++it) {
    const int n = int(uni(3, 30));
    std::vector<double> Ls(n), Ts(n);
    for (int i = 0; i < n; ++i) {
      Ls[i] = double(uni(0, 50000)) + i;
      Ts[i] = 1e-9 * Ls[i] * Ls[i] + 1e-5 * Ls[i] + 0.01 + 1e-4 * double(uni(0, 100));
    }
    libra_ce_poly poly{};
    if (libra_ce_fit(Ls.data(), Ts.data(), n, &poly) == LIBRA_OK) {
      double mape = -1;
      CHECK(libra_ce_mape(&poly, Ls.data(), Ts.data(), n, &mape) == LIBRA_OK && mape >= 0);
    }
    double s = 0;
    const int64_t a = uni(0, 1 << 20), b = uni(0, 1 << 20);
    CHECK(libra_ce_poly_sum(&poly, a, b, &s) == LIBRA_OK);
    CHECK(std::isfinite(s) || !std::isfinite(poly.gamma));
  }

  // RolloutDP: literal and crossing search agree on the makespan; partitions are valid.
  const int32_t tps[4] = {1, 2, 4, 8};
  for (int it = 0; it < 120; ++it) {
    const int n = int(uni(0, 60)), g = int(uni(0, 20)), nt = int(uni(1, 4));
    std::vector<int64_t> lens(n);
    for (auto& x : lens) x = uni(0, 30000);
    libra_rollout_model m{};
    m.attn_step = libra_ce_poly{0.0, 2.7e-8, 1e-5};
    for (int k = 0; k < 4; ++k) {
      m.linear_step[k] = 3e-3 / (1 << k) + 1e-4;
      m.attn_scale[k] = 1.0 / (1 << k) + 0.02;
    }
    std::vector<int32_t> order(std::max(1, n)), inst(3 * std::max(1, g));
    double ms[2];
    int32_t k[2];
    for (int e = 0; e < 2; ++e) {
      CHECK(libra_rollout_dp(lens.data(), n, g, tps, nt, &m, e, &ms[e], order.data(), inst.data(),
                             &k[e]) == LIBRA_OK);
      int gsum = 0, rsum = 0;
      for (int i = 0; i < k[e]; ++i) {
        gsum += inst[3 * i];
        rsum += inst[3 * i + 2];
        CHECK(inst[3 * i + 1] >= 0 && inst[3 * i + 1] + inst[3 * i + 2] <= n);
      }
      if (std::isfinite(ms[e])) CHECK(gsum == g && rsum == n);
    }
    CHECK(ms[0] == ms[1] || (std::isinf(ms[0]) && std::isinf(ms[1])));
  }

  // Prefix tree and routing.
  for (int it = 0; it < 20; ++it) {
    const int ne = int(uni(0, 6));
    std::vector<int64_t> edges(ne);
    int64_t e = 0;
    for (auto& x : edges) x = (e += uni(1, 5000));
    libra_trie t = nullptr;
    CHECK(libra_trie_create(edges.data(), ne, &t) == LIBRA_OK);
    std::vector<double> hist(size_t(ne) + 1);
    int32_t depth = 0;
    CHECK(libra_trie_lookup(t, 1, nullptr, 0, hist.data(), &depth) == LIBRA_E_INVAL);
    for (int tr = 0; tr < 200; ++tr) {
      const int ns = int(uni(0, 8));
      std::vector<int32_t> st(ns);
      std::vector<int64_t> res(size_t(ns) + 1);
      for (auto& x : st) x = int32_t(uni(0, 15));
      for (auto& x : res) x = uni(0, 40000);
      CHECK(libra_trie_insert(t, uni(0, 20), st.data(), ns, res.data()) == LIBRA_OK);
    }
    for (int q = 0; q < 200; ++q) {
      const int ns = int(uni(0, 10));
      std::vector<int32_t> st(ns);
      for (auto& x : st) x = int32_t(uni(0, 15));
      CHECK(libra_trie_lookup(t, uni(0, 25), st.data(), ns, hist.data(), &depth) == LIBRA_OK);
      double sum = 0;
      for (double h : hist) sum += h;
      CHECK(std::fabs(sum - 1.0) < 1e-12 && depth >= -1 && depth <= ns);
      const int M = int(uni(1, 5));
      std::vector<double> td(size_t(M) * hist.size()), cm(size_t(M) * M);
      for (auto& x : td) x = double(uni(1, 100));
      for (auto& x : cm) x = double(uni(0, 10));
      int32_t best = -1;
      double cost = 0;
      CHECK(libra_route_bucket(hist.data(), int32_t(hist.size()), td.data(), cm.data(), M,
                               int32_t(uni(0, M - 1)), &best, &cost) == LIBRA_OK);
      CHECK(best >= 0 && best < M);
    }
    libra_trie_destroy(t);
  }
  std::printf("host fuzz ok\n");
  return 0;
}
