// Causal attention of an appended chunk (e.g. a tool output) over the paged KV cache.
//
// One 256-thread workgroup per chunk unit (sequence b, KV head g, new tokens [q0, q1)).
// Query rows are (token, head) pairs of the G heads sharing KV head g; they are packed
// into 16-wide matrix columns, tpb = max(1, 16 / G) tokens per column block.  Each of
// the 4 waves owns 4 column blocks (64 columns), so a workgroup covers up to 16 * tpb
// tokens.  Keys are visited one page pair at a time; the pair's four 4 KiB tiles (K and
// V of both pages) are staged in LDS, double-buffered, and shared by the 4 waves:
// every K/V byte fetched from HBM feeds 64 query columns per wave.  The math per pair
// and column block is the decode kernel's:
//   S^T = K . Q^T (4 mfma 16x16x32 per page), online softmax in base 2,
//   O^T += V^T . P^T (8 mfma 16x16x32 over the 32 keys of the pair).
// Column c of block nb in wave w is token q0 + (4 w + nb) * tpb + c / G, head c % G; it
// sees keys k <= P_b + token (causal, itself included).
#include <cmath>

#include "internal.h"

namespace libra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kNB = 4;               // column blocks per wave
constexpr int kTileU4 = kTileBytes / 16;  // uint4 per tile (256)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = static_cast<__bf16>(lo);
  const __bf16 b = static_cast<__bf16>(hi);
  return uint32_t(__builtin_bit_cast(uint16_t, a)) | (uint32_t(__builtin_bit_cast(uint16_t, b)) << 16);
}

struct ChunkArgs {
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* units;
  const int32_t* bt;
  const uint16_t* q;
  uint16_t* out;
  float* lse;
  int64_t bt_stride;
  int hkv;
  int hq;
  int group;
  float sl2;
};

__global__ __launch_bounds__(kThreads) void chunk_kernel(ChunkArgs A) {
  // [buffer][KA, KB, VA, VB][256 x uint4]
  __shared__ uint4 lds[2][4][kTileU4];

  const int32_t* u = A.units + size_t(blockIdx.x) * kUnitInts;
  const int b = u[U_B], g = u[U_G], kv1 = u[U_KV1];
  const int q0 = u[U_Q0], q1 = u[U_Q1], row0 = u[U_ROW0], prior = u[U_PRIOR];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, quad = lane >> 4;
  const int G = A.group;
  const int tpb = G >= 16 ? 1 : 16 / G;

  // Per column block: token, head, key limit and Q operand.
  int tok[kNB], lim[kNB];
  bf16x8 qop[kNB][4];
  const int head = col % G;
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int t = q0 + (kNB * wave + nb) * tpb + col / G;
    const bool ok = col < tpb * G && t < q1;
    tok[nb] = ok ? t : -1;
    lim[nb] = ok ? prior + t : -1;  // last visible key position
    const uint4* qrow = reinterpret_cast<const uint4*>(
        A.q + (size_t(row0 + (ok ? t : 0)) * A.hq + size_t(g) * G + head) * kDim);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (ok) v = qrow[4 * i + quad];
      qop[nb][i] = as_bf16x8(v);
    }
  }

  float m[kNB], l[kNB];
  f32x4 acc[kNB][8];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    m[nb] = -INFINITY;
    l[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int npages = (kv1 + kPage - 1) / kPage;
  const int npairs = (npages + 1) >> 1;
  const int32_t* btrow = A.bt + int64_t(b) * A.bt_stride;
  const size_t head_off = size_t(g) * kTileElems;
  const size_t page_stride = size_t(A.hkv) * kTileElems;

  auto fetch = [&](int pair, uint4 (&r)[4]) {
    const int pa = 2 * pair;
    const size_t ba = size_t(btrow[pa]) * page_stride + head_off;
    r[0] = reinterpret_cast<const uint4*>(A.k_cache + ba)[tid];
    r[2] = reinterpret_cast<const uint4*>(A.v_cache + ba)[tid];
    if (pa + 1 < npages) {
      const size_t bb = size_t(btrow[pa + 1]) * page_stride + head_off;
      r[1] = reinterpret_cast<const uint4*>(A.k_cache + bb)[tid];
      r[3] = reinterpret_cast<const uint4*>(A.v_cache + bb)[tid];
    } else {
      r[1] = make_uint4(0, 0, 0, 0);
      r[3] = make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf, const uint4 (&r)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) lds[buf][i][tid] = r[i];
  };

  uint4 stage[4];
  if (npairs > 0) {
    fetch(0, stage);
    stash(0, stage);
  }
  __syncthreads();

  for (int n = 0; n < npairs; ++n) {
    const int buf = n & 1;
    if (n + 1 < npairs) fetch(n + 1, stage);

    // This pair's operands, read from LDS in the same lane order as the tiles.
    uint4 ka[4], kb[4], va[4], vb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ka[i] = lds[buf][0][i * 64 + lane];
      kb[i] = lds[buf][1][i * 64 + lane];
      va[i] = lds[buf][2][i * 64 + lane];
      vb[i] = lds[buf][3][i * 64 + lane];
    }
    const int key_a = 2 * n * kPage;  // first key of page A
    // Zero V of slots at or past kv1 (never-written or NaN-poisoned slots).
    if (key_a + 2 * kPage > kv1) {
#pragma unroll
      for (int pgi = 0; pgi < 2; ++pgi) {
        const int keep = min(max(kv1 - key_a - pgi * kPage - 4 * quad, 0), 4);
        const uint32_t m0 = keep >= 2 ? 0xFFFFFFFFu : (keep == 1 ? 0x0000FFFFu : 0u);
        const uint32_t m1 = keep >= 4 ? 0xFFFFFFFFu : (keep == 3 ? 0x0000FFFFu : 0u);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint4& v = pgi == 0 ? va[i] : vb[i];
          v.x &= m0;
          v.y &= m1;
          v.z &= m0;
          v.w &= m1;
        }
      }
    }

#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka[i]), qop[nb][i], sa, 0, 0, 0);
        sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kb[i]), qop[nb][i], sb, 0, 0, 0);
      }
      float x[8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ka_pos = key_a + 4 * quad + r;
        x[r] = ka_pos <= lim[nb] ? sa[r] * A.sl2 : -INFINITY;
        x[4 + r] = ka_pos + kPage <= lim[nb] ? sb[r] * A.sl2 : -INFINITY;
      }
      float mx = x[0];
#pragma unroll
      for (int i = 1; i < 8; ++i) mx = fmaxf(mx, x[i]);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m[nb], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m[nb] - m_use);
      float p[8], ps = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        p[i] = __builtin_amdgcn_exp2f(x[i] - m_use);
        ps += p[i];
      }
      l[nb] = l[nb] * alpha + ps;
      m[nb] = m_new;
      uint4 pb;
      pb.x = pack_bf16x2(p[0], p[1]);
      pb.y = pack_bf16x2(p[2], p[3]);
      pb.z = pack_bf16x2(p[4], p[5]);
      pb.w = pack_bf16x2(p[6], p[7]);
      const bf16x8 pop = as_bf16x8(pb);
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const uint4 a4 = va[db >> 1], b4 = vb[db >> 1];
        const uint4 vo = (db & 1) ? make_uint4(a4.z, a4.w, b4.z, b4.w)
                                  : make_uint4(a4.x, a4.y, b4.x, b4.y);
        acc[nb][db] *= alpha;
        acc[nb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vo), pop, acc[nb][db], 0, 0, 0);
      }
    }

    if (n + 1 < npairs) stash(buf ^ 1, stage);
    __syncthreads();
  }

  // Epilogue: every column is owned by one wave; normalise and store.
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    float ls = l[nb];
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    if (tok[nb] < 0) continue;
    const float inv = ls > 0.f ? 1.f / ls : 0.f;
    const size_t orow = (size_t(row0 + tok[nb]) * A.hq + size_t(g) * G + head);
    uint16_t* op = A.out + orow * kDim + 4 * quad;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      uint2 w;
      w.x = pack_bf16x2(acc[nb][db][0] * inv, acc[nb][db][1] * inv);
      w.y = pack_bf16x2(acc[nb][db][2] * inv, acc[nb][db][3] * inv);
      *reinterpret_cast<uint2*>(op + db * 16) = w;
    }
    if (A.lse && quad == 0)
      A.lse[orow] = ls > 0.f ? (m[nb] + log2f(ls)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_chunk(const KvLayout& L, const Plan& P, void* ws, const void* q,
                        const int32_t* bt, int32_t stride, float scale, void* out, float* lse,
                        hipStream_t s) {
  const int n = P.info.n_chunk;
  if (n == 0) return hipSuccess;
  char* w = static_cast<char*>(ws);
  ChunkArgs A;
  A.k_cache = static_cast<const uint16_t*>(L.desc.k_cache);
  A.v_cache = static_cast<const uint16_t*>(L.desc.v_cache);
  A.units = reinterpret_cast<const int32_t*>(w + P.off_units) + size_t(P.info.n_single) * kUnitInts;
  A.bt = bt;
  A.q = static_cast<const uint16_t*>(q);
  A.out = static_cast<uint16_t*>(out);
  A.lse = lse;
  A.bt_stride = stride;
  A.hkv = P.num_kv_heads;
  A.hq = P.num_q_heads;
  A.group = P.group;
  A.sl2 = scale * kLog2e;
  hipLaunchKernelGGL(chunk_kernel, dim3(unsigned(n)), dim3(kThreads), 0, s, A);
  return hipGetLastError();
}

}  // namespace libra
