// Checks which entry points allocate, against the host-only HIP stand-in (fake_hip.cpp):
// plan creation may take pinned staging and an event (from the library's pool); uploads,
// decode and append calls must make no allocating runtime call; destroying a plan returns
// its staging to the pool, so the next plan of the same size allocates nothing either.
// "Device" buffers are host memory; kernel launches are stubbed (stubs.cpp with
// LIBRA_STUB_LAUNCH_OK) and only counted.
#include <cstdio>
#include <cstring>
#include <vector>

#include "fake_hip.h"
#include "libra.h"

#define CHECK(cond)                                                         \
  do {                                                                      \
    if (!(cond)) {                                                          \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      return 1;                                                             \
    }                                                                       \
  } while (0)

namespace {

struct Buffers {
  std::vector<unsigned char> k, v, q, kn, vn, out, bt;
  std::vector<float> lse;
  std::vector<unsigned char> ws;  // over-allocated so that a 256-byte aligned window fits
  void* ws_aligned(size_t bytes) {
    ws.assign(bytes + 512, 0);
    uintptr_t p = reinterpret_cast<uintptr_t>(ws.data());
    return reinterpret_cast<void*>((p + 255) & ~uintptr_t(255));
  }
};

}  // namespace

int main() {
  const int B = 5, hq = 32, hkv = 8;
  const int32_t lens[B] = {3000, 17, 5000, 129, 2048};
  const int32_t qlens[B] = {1, 1, 300, 1, 64};
  int32_t rows = 0;
  for (int b = 0; b < B; ++b) rows += qlens[b];
  const int64_t pages = 5000 / 16 + 8;
  const int32_t stride = int32_t(pages);

  Buffers m;
  m.k.assign(size_t(pages) * hkv * 4096 + 16, 0);
  m.v = m.k;
  m.q.assign(size_t(rows) * hq * 256 + 16, 0);
  m.out = m.q;
  m.kn.assign(size_t(rows) * hkv * 256 + 16, 0);
  m.vn = m.kn;
  m.bt.assign(size_t(B) * stride * 4 + 16, 0);
  m.lse.assign(size_t(rows) * hq + 4, 0.f);
  auto al16 = [](std::vector<unsigned char>& v) {
    uintptr_t p = reinterpret_cast<uintptr_t>(v.data());
    return reinterpret_cast<void*>((p + 15) & ~uintptr_t(15));
  };

  libra_kv_layout_desc desc{pages, 16, hkv, 128, LIBRA_DTYPE_BF16, al16(m.k), al16(m.v)};
  libra_kv_layout lay = nullptr;
  CHECK(libra_kv_layout_create(&desc, &lay) == LIBRA_OK);

  libra_plan_params p{64, 3, 4, 64, 0, {0, 0, 0, 0, 0, 0, 0, 0}};
  libra_plan_desc dd{LIBRA_MODE_DECODE, B, hq, hkv};
  libra_plan_desc da{LIBRA_MODE_APPEND, B, hq, hkv};

  // Plan creation: the only place staging may be allocated.
  const FakeHipCounters before_plans = g_fake_hip;
  libra_plan dec = nullptr, app = nullptr;
  CHECK(libra_splitkv_plan(&dd, lens, nullptr, &p, &dec) == LIBRA_OK);
  CHECK(libra_splitkv_plan(&da, lens, qlens, &p, &app) == LIBRA_OK);
  CHECK(g_fake_hip.host_malloc - before_plans.host_malloc == 2);
  // one upload event each; the append plan (decode rows and chunk tiles) also takes its
  // fork / join events and creates the device's auxiliary stream
  CHECK(g_fake_hip.event_create - before_plans.event_create == 4);
  CHECK(g_fake_hip.stream_create - before_plans.stream_create == 1);

  const size_t wsd = libra_plan_workspace_bytes(dec), wsa = libra_plan_workspace_bytes(app);
  Buffers w1, w2;
  void* ws1 = w1.ws_aligned(wsd > wsa ? wsd : wsa);
  void* ws2 = w2.ws_aligned(wsd > wsa ? wsd : wsa);
  const size_t wsb = wsd > wsa ? wsd : wsa;

  // Hot calls: uploads, decode and append, taking turns on two workspaces.
  const FakeHipCounters before = g_fake_hip;
  CHECK(libra_plan_upload(dec, ws1, wsb, nullptr) == LIBRA_OK);
  for (int it = 0; it < 3; ++it) {
    CHECK(libra_decode_attn(lay, dec, al16(m.q), reinterpret_cast<int32_t*>(al16(m.bt)), stride,
                            B, hq, 0.088f, ws1, wsb, al16(m.out), m.lse.data(),
                            nullptr) == LIBRA_OK);
    CHECK(libra_append_attn(lay, app, al16(m.q), al16(m.kn), al16(m.vn),
                            reinterpret_cast<int32_t*>(al16(m.bt)), stride, B, hq, 0.088f,
                            it % 2 ? ws2 : ws1, wsb, al16(m.out), m.lse.data(),
                            nullptr) == LIBRA_OK);
  }
  const FakeHipCounters& after = g_fake_hip;
  CHECK(after.allocations() == before.allocations());
  CHECK(after.launches > before.launches);          // the calls did reach their launches
  CHECK(after.stream_wait - before.stream_wait == 6);  // fork and join of 3 append calls
  CHECK(after.memcpy_async - before.memcpy_async >= 4);  // tables re-uploaded on turns
  // The uploaded table image is the plan's unit table.
  const int32_t* units = nullptr;
  int32_t n_units = 0;
  CHECK(libra_plan_get_units(app, &units, &n_units) == LIBRA_OK && n_units > 0);
  CHECK(std::memcmp(ws2, units, size_t(n_units) * LIBRA_UNIT_INTS * sizeof(int32_t)) == 0);

  // Destroying plans frees nothing; a new plan of the same size reuses the pool.
  const FakeHipCounters before_destroy = g_fake_hip;
  libra_plan_destroy(dec);
  libra_plan_destroy(app);
  CHECK(g_fake_hip.allocations() == before_destroy.allocations());
  libra_plan dec2 = nullptr;
  CHECK(libra_splitkv_plan(&dd, lens, nullptr, &p, &dec2) == LIBRA_OK);
  CHECK(g_fake_hip.allocations() == before_destroy.allocations());
  CHECK(libra_decode_attn(lay, dec2, al16(m.q), reinterpret_cast<int32_t*>(al16(m.bt)), stride, B,
                          hq, 0.088f, ws1, wsb, al16(m.out), nullptr, nullptr) == LIBRA_OK);
  CHECK(g_fake_hip.allocations() == before_destroy.allocations());
  // The static-scratch variant: no allocating call on its first call or later ones; its
  // tables go to the scratch once per plan, and a plan too large for it is refused.
  const FakeHipCounters before_static = g_fake_hip;
  for (int it = 0; it < 3; ++it)
    CHECK(libra_decode_attn_noalloc(lay, dec2, al16(m.q), reinterpret_cast<int32_t*>(al16(m.bt)),
                                    stride, B, hq, 0.088f, al16(m.out), m.lse.data(),
                                    nullptr) == LIBRA_OK);
  CHECK(g_fake_hip.allocations() == before_static.allocations());
  CHECK(g_fake_hip.memcpy_async - before_static.memcpy_async == 1);
  CHECK(g_fake_hip.launches > before_static.launches);
  CHECK(libra_decode_attn_noalloc(lay, dec2, al16(m.q), reinterpret_cast<int32_t*>(al16(m.bt)),
                                  stride, B, hq, -1.f, al16(m.out), nullptr,
                                  nullptr) == LIBRA_E_INVAL);
  {
    // 40 rows of 65,536 tokens cut into 64 splits each: 40 * 8 * 64 partial slots of
    // 4 * 129 * 4 bytes, over 8 MiB of scratch.
    std::vector<int32_t> big(40, 65536);
    libra_plan_params pb{4096, 3, 1, 64, 0, {0, 0, 0, 0, 0, 0, 0, 0}};
    libra_plan_desc db{LIBRA_MODE_DECODE, 40, hq, hkv};
    libra_plan bigp = nullptr;
    CHECK(libra_splitkv_plan(&db, big.data(), nullptr, &pb, &bigp) == LIBRA_OK);
    CHECK(libra_plan_workspace_bytes(bigp) > (size_t(8) << 20));
    const long copies = g_fake_hip.memcpy_async, launches = g_fake_hip.launches;
    CHECK(libra_decode_attn_noalloc(lay, bigp, al16(m.q), reinterpret_cast<int32_t*>(al16(m.bt)),
                                    65536 / 16, 40, hq, 0.088f, al16(m.out), nullptr,
                                    nullptr) != LIBRA_OK);
    CHECK(g_fake_hip.memcpy_async == copies && g_fake_hip.launches == launches);
    libra_plan_destroy(bigp);
  }
  libra_plan_destroy(dec2);
  libra_kv_layout_destroy(lay);
  std::printf("no-alloc ok: %ld launches, %ld table copies\n", g_fake_hip.launches,
              g_fake_hip.memcpy_async);
  return 0;
}
