// Causal attention of an appended chunk (e.g. a tool output) over the paged KV cache.
//
// One 512-thread workgroup (8 waves, two per SIMD) per chunk unit (sequence b, KV head
// g, new tokens [q0, q1)).  Query rows are the (token, head) pairs of the G heads sharing
// KV head g, token-major; wave w owns the 32 rows 32 w .. 32 w + 31 as the 32 columns of
// its matrix products, so a workgroup covers 256 rows, i.e. floor(256 / G) tokens.
// Keys are visited 64 at a time (a step: four pages, two page pairs).  The step's four
// K tiles and four V tiles are copied from memory straight into a four-stage LDS ring
// three steps ahead (global_load_lds_dwordx4, 16 bytes per lane, the tiles in their
// stored order, no registers), shared by the 8 waves.  Per page pair and wave, on
// v_mfma_f32_32x32x16_bf16:
//   S^T[32 keys x 32 rows] = K . Q^T: 8 MFMAs over the 128 channels; lane (key m, half
//     h) reads K granule (2 c + h) * 16 + m % 16 of page 2P + m / 16 for channels
//     16 c + 8 h .. + 7, and holds scores of keys 8 (r / 4) + 4 h + r % 4 (r = 0..15)
//     for its row;
//   O^T[128 channels x 32 rows] += V^T . P^T: per page, 4 MFMAs (32-channel blocks) over
//     the page's 16 keys.  A lane's probabilities of one page, keys {4h..4h+3, 8+4h..
//     11+4h} in that order, are its B operand as they come out of the scores; the
//     matching A operand, channel d's values at those keys, is V granule 128 h + d of
//     the stored tile (one 16-byte LDS read; the 32 lanes of one half read 512 contiguous
//     bytes, free of bank conflicts), which is why V tiles are stored in that order.
// Each wave works through a step by page pairs: the pair's K operands for step n + 1
// are read from LDS first, then the pair's probabilities are formed (exps) while they
// land, then step n + 1's scores of the pair (a dependent chain of 8 MFMAs) are issued
// interleaved with the pair's 8 independent PV products.
// Softmax runs online in base 2 against a running maximum that is set exactly on the
// first step and afterwards moved only when needed: the probabilities of a page pair
// are taken against the current maximum, and if any lane's sum of them exceeds 2^kTau
// (which any probability above 2^kTau forces), a wave-wide vote moves the maximum to
// the pair's own, rescales the accumulators and takes them again, before a product uses
// them.  Probabilities therefore stay at most 2^kTau, and the result is exact after the
// final normalisation; no per-step maximum is taken.  Causal masks are applied only on
// steps that reach past the tile's first token.  Row r = 32 w + column of the tile is
// token q0 + r / G, head r % G; it sees keys k <= P_b + token.
// Units arrive in per-XCD queues: workgroup w takes tile w / 8 of queue w % 8, so the
// tiles of one (b, g), which read the same keys, run on one XCD and share its L2; each
// queue holds its longest tiles first.  Wave priority is 1 through the first page pair of
// a step and 0 through the second (see the note at the key loop).
#include <cmath>
#include <type_traits>

#include "internal.h"

namespace libra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
static_assert(kChunkRows == 32 * kWaves, "the plan's tile rows are the kernel's");
constexpr int kStepPages = 4;    // pages (16 keys each) per softmax step
static_assert(kStepPages * kPage == kChunkStepKeys, "the plan's tile cost counts these steps");
constexpr int kTau = 8;           // lazy-rescale threshold, base-2 logits
constexpr float kSumTau = float(1 << kTau);  // probabilities stay at most 2^kTau
constexpr int kMaxIds = 4096;     // block-table entries staged in LDS (64K keys)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 x) { return __builtin_bit_cast(bf16x8, x); }
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

struct ChunkArgs {
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* units;
  const int32_t* xcd_map;
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

// Row (M index) of element r of a 32x32 accumulator in a lane of half h.
__device__ __forceinline__ constexpr int acc_row(int r, int h) { return 8 * (r / 4) + 4 * h + (r % 4); }

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void chunk_kernel(ChunkArgs A) {
  // K and V stages: [page of the step][256 x uint4], the tiles as stored.  One array per
  // stage: the direct memory-to-LDS copies into one stage then never make the compiler
  // wait before LDS reads of another.
  __shared__ __align__(16) uint4 ldk0[kStepPages][256];
  __shared__ __align__(16) uint4 ldk1[kStepPages][256];
  __shared__ __align__(16) uint4 ldk2[kStepPages][256];
  __shared__ __align__(16) uint4 ldk3[kStepPages][256];
  __shared__ __align__(16) uint4 ldv0[kStepPages][256];
  __shared__ __align__(16) uint4 ldv1[kStepPages][256];
  __shared__ __align__(16) uint4 ldv2[kStepPages][256];
  __shared__ __align__(16) uint4 ldv3[kStepPages][256];
  __shared__ __align__(16) int lds_ids[kMaxIds];
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  auto kst = [&](auto s_tag) -> uint4 (&)[kStepPages][256] {
    constexpr int st = decltype(s_tag)::value & 3;
    if constexpr (st == 0) return ldk0;
    else if constexpr (st == 1) return ldk1;
    else if constexpr (st == 2) return ldk2;
    else return ldk3;
  };
  auto vst = [&](auto s_tag) -> uint4 (&)[kStepPages][256] {
    constexpr int st = decltype(s_tag)::value & 3;
    if constexpr (st == 0) return ldv0;
    else if constexpr (st == 1) return ldv1;
    else if constexpr (st == 2) return ldv2;
    else return ldv3;
  };

  const int xcd = blockIdx.x % kNumXcds;
  const int slot = blockIdx.x / kNumXcds;
  if (slot >= A.xcd_map[2 * xcd + 1]) return;
  const int32_t* u = A.units + size_t(A.xcd_map[2 * xcd] + slot) * kUnitInts;
  const int b = u[U_B], g = u[U_G], kv1 = u[U_KV1];
  const int q0 = u[U_Q0], q1 = u[U_Q1], row0 = u[U_ROW0], prior = u[U_PRIOR];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 31, hh = lane >> 5;  // accumulator column (tile row), lane half
  const int G = A.group;

  // Tile row of this lane's column: r = 32 wave + col; token q0 + r / G, head r % G.
  const int r_tile = 32 * wave + col;
  const int t_tok = q0 + r_tile / G;
  const int head = r_tile % G;
  const bool ok = t_tok < q1;
  const int tok = ok ? t_tok : -1;
  const int lim = ok ? prior + t_tok : -1;
  // Q operand of MFMA c (channels 16 c .. 16 c + 15): lane (col, hh) holds channels
  // 16 c + 8 hh .. + 7 of its row.
  bf16x8 qop[8];
  {
    const uint4* qrow = reinterpret_cast<const uint4*>(
        A.q + (size_t(row0 + (ok ? t_tok : 0)) * A.hq + size_t(g) * G + head) * kDim);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (ok) v = qrow[2 * c + hh];
      qop[c] = as_bf16x8(v);
    }
  }

  float m = -INFINITY, l = 0.f;
  f32x16 acc[4];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;

  const int npages = (kv1 + kPage - 1) / kPage;
  const int nsteps = (npages + kStepPages - 1) / kStepPages;
  const int32_t* btrow = A.bt + int64_t(b) * A.bt_stride;
  const uint32_t page_bytes = uint32_t(A.hkv) * kTileBytes;
  const int first_tok = prior + q0;
  const int mask_key0 = min(first_tok - (kStepPages * kPage - 1), kv1 - kStepPages * kPage);

  const char* k_lane = reinterpret_cast<const char*>(A.k_cache) + size_t(g) * kTileBytes +
                       size_t(lane) * 16;
  const char* v_lane = reinterpret_cast<const char*>(A.v_cache) + size_t(g) * kTileBytes +
                       size_t(lane) * 16;
  // K and V of `step` straight into LDS stage stage_tag & 3: wave w moves 1 KiB chunks
  // 2 w and 2 w + 1 of the step's four K tiles and of its four V tiles (16 B per lane at
  // the chunk's LDS base + 16 lane, the tile as stored).  Both chunks lie in page w / 2 of
  // the step, so a wave needs one page id: from the staged row (a broadcast LDS read), or
  // from global memory past it (uniform and rare).  Pages past the end re-read the last
  // page (the id row is padded with it), so the copies stay branch-free; their keys are
  // >= kv1, so they are masked and their V zeroed.  The wave index is made scalar, so the
  // page, the LDS targets and the byte offsets are scalar arithmetic.  Four vector-memory
  // operations per wave per step, in a fixed order; the waits count them.
  auto copy_kv = [&](int step, auto stage_tag) {
    const int j = wave >> 1;
    const int p = step * kStepPages + j;
    const int id = p < kMaxIds ? __builtin_amdgcn_readfirstlane(lds_ids[p])
                               : __builtin_amdgcn_readfirstlane(btrow[min(p, npages - 1)]);
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const int i = (2 * wave + c2) & 3;
      const uint64_t off = uint64_t(uint32_t(id)) * page_bytes + i * 1024;
      const uint32_t dk = uint32_t(reinterpret_cast<uintptr_t>(&kst(stage_tag)[j][i * 64]));
      const char* ksrc = k_lane + off;
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(dk), "v"(ksrc)
                   : "memory", "m0");
      const uint32_t dv = uint32_t(reinterpret_cast<uintptr_t>(&vst(stage_tag)[j][i * 64]));
      const char* vsrc = v_lane + off;
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(dv), "v"(vsrc)
                   : "memory", "m0");
    }
  };

  // Stage the page ids once (padded to whole steps with the last id), so that each
  // prefetch is one dependent load, not two.
  const int nids = min(nsteps * kStepPages, kMaxIds);
  for (int i = tid; i < nids; i += kThreads) lds_ids[i] = btrow[min(i, npages - 1)];
  __syncthreads();

  // Scores S^T (32 keys of page pair P x 32 rows) from K stage: K operand of MFMA c,
  // lane (key m, hh): slot m % 16 of page 2P + m / 16, channels 16 c + 8 hh .. + 7, the
  // K granule (2 c + hh) * 16 + slot.
  auto qk_pair = [&](auto stage_tag, int P, f32x16& s) {
    f32x16 a;
#pragma unroll
    for (int r = 0; r < 16; ++r) a[r] = 0.f;
    const int j = 2 * P + (col >> 4);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const uint4 kr = kst(stage_tag)[j][(2 * c + hh) * 16 + (col & 15)];
      a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kr), qop[c], a, 0, 0, 0);
    }
    s = a;
  };

  // Causal / length mask of step n; on the first step (exact) also the running maximum
  // (later steps check their probabilities instead, in pair()).
  auto prepare = [&](int key0, f32x16 (&s)[2], float& neg_m, bool exact) {
    if (key0 > mask_key0) {
#pragma unroll
      for (int P = 0; P < 2; ++P)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + 32 * P + acc_row(r, hh) > lim) s[P][r] = -INFINITY;
    }
    if (exact) {
      float mloc = -INFINITY;
#pragma unroll
      for (int P = 0; P < 2; ++P)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[P][r]);
      float mc = fmaxf(mloc * A.sl2, m);
      m = fmaxf(mc, __shfl_xor(mc, 32));
    }
    neg_m = m == -INFINITY ? 0.f : -m;
  };
  // Moves the running maximum to cover page pair P's scores (rare): rescales l and the
  // accumulators by 2^(m_old - m_new).
  auto rescale = [&](const f32x16& sp, float& neg_m) {
    float mloc = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sp[r]);
    float mc = fmaxf(mloc * A.sl2, m);
    mc = fmaxf(mc, __shfl_xor(mc, 32));
    const float alpha = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mc);
    l *= alpha;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[cb] *= alpha;
    m = mc;
    neg_m = m == -INFINITY ? 0.f : -m;
  };

  // Page pair P of step n: probabilities (consuming s[P]), step n + 1's scores of the
  // pair (from stage kread, unless last) and O^T += V^T P^T over the pair's two pages
  // from V stage vread.  V operand of page j, channel block cb: lane (channel
  // 32 cb + col, hh) reads granule 128 hh + 32 cb + col, keys in the order of the P
  // operand (element p: slot 8 (p / 4) + 4 hh + p % 4), which is the score layout.
  auto pair = [&](int P, auto kread, auto vread, int key0, f32x16 (&s)[2], float& neg_m,
                  auto last_tag) {
    constexpr bool kLast = decltype(last_tag)::value;
    uint4 kpre[8];
    if constexpr (!kLast) {
#pragma unroll
      for (int c = 0; c < 8; ++c) kpre[c] = kst(kread)[2 * P + (col >> 4)][(2 * c + hh) * 16 + (col & 15)];
    }
    // Probabilities against the current maximum.  A probability above 2^kTau (the
    // maximum is stale by more than kTau, or this is a new row's first real score)
    // makes this lane's sum of the pair exceed 2^kTau: the wave then moves the maximum
    // to the pair's own and takes them again, before any product has used them.
    float p[16], ps;
    auto take = [&]() {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(fmaf(s[P][r], A.sl2, neg_m));
      const float t0 = (p[0] + p[1]) + (p[2] + p[3]), t1 = (p[4] + p[5]) + (p[6] + p[7]);
      const float t2 = (p[8] + p[9]) + (p[10] + p[11]), t3 = (p[12] + p[13]) + (p[14] + p[15]);
      ps = (t0 + t1) + (t2 + t3);
    };
    take();
    if (__ballot(!(ps <= kSumTau))) {
      rescale(s[P], neg_m);
      take();
    }
    l += ps;
    uint4 pa, pb;
    pa.x = pack_bf16x2(p[0], p[1]);
    pa.y = pack_bf16x2(p[2], p[3]);
    pa.z = pack_bf16x2(p[4], p[5]);
    pa.w = pack_bf16x2(p[6], p[7]);
    pb.x = pack_bf16x2(p[8], p[9]);
    pb.y = pack_bf16x2(p[10], p[11]);
    pb.z = pack_bf16x2(p[12], p[13]);
    pb.w = pack_bf16x2(p[14], p[15]);
    // Step n + 1's scores of the pair (a chain of 8 dependent MFMAs) interleaved with the
    // pair's PV products (8 independent ones), so the chain's latency is covered.
    f32x16 qs;
#pragma unroll
    for (int r = 0; r < 16; ++r) qs[r] = 0.f;
    uint32_t mk[2][4];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int e = 0; e < 4; ++e) mk[jj][e] = ~0u;
    if constexpr (kLast) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int valid = kv1 - key0 - (2 * P + jj) * kPage;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int s0 = 8 * ((2 * e) / 4) + 4 * hh + (2 * e) % 4;
          const int s1 = 8 * ((2 * e + 1) / 4) + 4 * hh + (2 * e + 1) % 4;
          mk[jj][e] = (s0 < valid ? 0x0000FFFFu : 0u) | (s1 < valid ? 0xFFFF0000u : 0u);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      if constexpr (!kLast) {
        qs = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kpre[c]), qop[c], qs, 0, 0, 0);
      }
      const int jj = c >> 2, cb = c & 3;
      uint4 vo = vst(vread)[2 * P + jj][128 * hh + 32 * cb + col];
      if constexpr (kLast) {
        vo.x &= mk[jj][0];
        vo.y &= mk[jj][1];
        vo.z &= mk[jj][2];
        vo.w &= mk[jj][3];
      }
      acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vo), as_bf16x8(jj == 0 ? pa : pb),
                                                        acc[cb], 0, 0, 0);
    }
    if constexpr (!kLast) s[P] = qs;
  };

  if (nsteps > 0) copy_kv(0, S0{});
  if (nsteps > 1) copy_kv(1, S1{});
  if (nsteps > 2) copy_kv(2, S2{});
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // Wave priority: 1 from a step's opening barrier through its first page pair, 0 for the
  // second.  The two waves of a SIMD otherwise share issue by age, so the older one ran
  // each step's pairs ~40% faster than its partner and then idled at the barrier while
  // the younger finished alone; dropping the priority of a wave once it is half-way
  // through lets a lagging partner catch up within the step.
  __builtin_amdgcn_s_setprio(1);

  f32x16 sc[2];
  if (nsteps > 0) {
    qk_pair(S0{}, 0, sc[0]);
    qk_pair(S0{}, 1, sc[1]);
  }
  // Step n: copies of step n + 3 into the stage last read in step n - 1; at its end only
  // those four copies may be in flight (vmcnt(4)): step n + 1's V and step n + 2's K
  // have landed.
  auto step = [&](int n, auto r_tag) {
    constexpr int r = decltype(r_tag)::value;
    using KRead = std::integral_constant<int, (r + 1) & 3>;
    using VRead = std::integral_constant<int, r>;
    using Copy = std::integral_constant<int, (r + 3) & 3>;
    const int key0 = n * kStepPages * kPage;
    copy_kv(min(n + 3, nsteps - 1), Copy{});
    float neg_m;
    prepare(key0, sc, neg_m, n == 0);
    pair(0, KRead{}, VRead{}, key0, sc, neg_m, std::false_type{});
    __builtin_amdgcn_s_setprio(0);
    pair(1, KRead{}, VRead{}, key0, sc, neg_m, std::false_type{});
    __builtin_amdgcn_s_waitcnt(0xF74);
    __syncthreads();
    __builtin_amdgcn_s_setprio(1);
  };
  int n0 = 0;
  for (; n0 + 4 < nsteps; n0 += 4) {
    step(n0, S0{});
    step(n0 + 1, S1{});
    step(n0 + 2, S2{});
    step(n0 + 3, S3{});
  }
  if (n0 + 1 < nsteps) {
    step(n0, S0{});
    if (n0 + 2 < nsteps) {
      step(n0 + 1, S1{});
      if (n0 + 3 < nsteps) step(n0 + 2, S2{});
    }
  }
  if (nsteps > 0) {
    const int key0 = (nsteps - 1) * kStepPages * kPage;
    float neg_m;
    prepare(key0, sc, neg_m, nsteps == 1);
    switch ((nsteps - 1) & 3) {
      case 0:
        pair(0, S0{}, S0{}, key0, sc, neg_m, std::true_type{});
        pair(1, S0{}, S0{}, key0, sc, neg_m, std::true_type{});
        break;
      case 1:
        pair(0, S0{}, S1{}, key0, sc, neg_m, std::true_type{});
        pair(1, S0{}, S1{}, key0, sc, neg_m, std::true_type{});
        break;
      case 2:
        pair(0, S0{}, S2{}, key0, sc, neg_m, std::true_type{});
        pair(1, S0{}, S2{}, key0, sc, neg_m, std::true_type{});
        break;
      default:
        pair(0, S0{}, S3{}, key0, sc, neg_m, std::true_type{});
        pair(1, S0{}, S3{}, key0, sc, neg_m, std::true_type{});
        break;
    }
  }

  // Epilogue: row col's sum over both lane halves; each lane stores its 16 channels per
  // channel block (runs of 4 at 32 cb + 8 e + 4 hh).
  float ls = l + __shfl_xor(l, 32);
  if (tok < 0) return;
  const float inv = ls > 0.f ? 1.f / ls : 0.f;
  const size_t orow = size_t(row0 + tok) * A.hq + size_t(g) * G + head;
  uint16_t* op = A.out + orow * kDim;
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint2 w;
      w.x = pack_bf16x2(acc[cb][4 * e] * inv, acc[cb][4 * e + 1] * inv);
      w.y = pack_bf16x2(acc[cb][4 * e + 2] * inv, acc[cb][4 * e + 3] * inv);
      *reinterpret_cast<uint2*>(op + 32 * cb + 8 * e + 4 * hh) = w;
    }
  if (A.lse && hh == 0) A.lse[orow] = ls > 0.f ? (m + log2f(ls)) * kLn2 : -INFINITY;
}

}  // namespace

hipError_t launch_chunk(const KvLayout& L, const Plan& P, void* ws, const void* q,
                        const int32_t* bt, int32_t stride, float scale, void* out, float* lse,
                        hipStream_t s) {
  if (P.info.n_chunk == 0) return hipSuccess;
  char* w = static_cast<char*>(ws);
  ChunkArgs A;
  A.k_cache = static_cast<const uint16_t*>(L.desc.k_cache);
  A.v_cache = static_cast<const uint16_t*>(L.desc.v_cache);
  A.units = reinterpret_cast<const int32_t*>(w + P.off_units) + size_t(P.info.n_single) * kUnitInts;
  A.xcd_map = reinterpret_cast<const int32_t*>(w + P.off_xcd_map);
  A.bt = bt;
  A.q = static_cast<const uint16_t*>(q);
  A.out = static_cast<uint16_t*>(out);
  A.lse = lse;
  A.bt_stride = stride;
  A.hkv = P.num_kv_heads;
  A.hq = P.num_q_heads;
  A.group = P.group;
  A.sl2 = scale * kLog2e;
  hipLaunchKernelGGL(chunk_kernel, dim3(unsigned(P.chunk_grid)), dim3(kThreads), 0, s, A);
  return hipGetLastError();
}

}  // namespace libra
