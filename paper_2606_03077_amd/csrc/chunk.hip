// Causal attention of an appended chunk (e.g. a tool output) over the paged KV cache.
//
// One 512-thread workgroup (8 waves) per chunk unit (sequence b, KV head g, new tokens
// [q0, q1)).  Query rows are the (token, head) pairs of the G heads sharing KV head g,
// token-major, packed 16 to a matrix column block whatever G is (a block may hold the
// end of one token's heads and the start of the next's); each wave owns 2 column blocks,
// so a workgroup covers 256 rows, i.e. up to floor(256 / G) tokens.  Keys are visited
// 64 at a time and staged in LDS (four stages), shared by the 8 waves: the step's four
// 4 KiB K tiles are copied from memory straight into LDS three steps ahead
// (global_load_lds_dwordx4, no registers), its four V tiles are loaded into registers
// two steps ahead and written to LDS interleaved by page pair, so that each PV operand
// is a single 16-byte LDS read.  Each wave works through a step by page pairs: the
// pair's probabilities, the next step's scores of the same two pages (written over the
// ones just consumed, so one score set suffices) and the pair's PV, which lets exps
// overlap score and PV MFMAs.  Per page and column block:
//   S^T = K . Q^T (4 mfma 16x16x32), and per page pair O^T += V^T . P^T (8 mfma 16x16x32
//   over 32 keys).
// Softmax runs online in base 2.  The running maximum is only moved (and the
// accumulators rescaled) when a step's scores exceed it by more than 2^kTau, which a
// wave-wide vote detects; otherwise probabilities are taken against the old maximum
// (at most 2^kTau, exact in the final normalisation).  Causal masks are applied only on
// steps that reach past the tile's first token.  Column c of block nb in wave w is row
// r = 16 (2 w + nb) + c of the tile: token q0 + r / G, head r % G; it sees keys
// k <= P_b + token.
// Units arrive in per-XCD queues: workgroup w takes tile w / 8 of queue w % 8, so the
// tiles of one (b, g), which read the same keys, run on one XCD and share its L2.
#include <cmath>
#include <type_traits>

#include "internal.h"

namespace libra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kNB = 2;           // column blocks per wave
static_assert(kChunkRows == 16 * kNB * kWaves, "the plan's tile rows are the kernel's");
constexpr int kStepPages = 4;    // pages (16 keys each) per softmax step
constexpr float kTau = 8.f;      // lazy-rescale threshold, base-2 logits
constexpr int kMaxIds = 4096;    // block-table entries staged in LDS (64K keys)
constexpr int kBufs = 4;         // LDS stages, indexed by step & 3
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 x) { return __builtin_bit_cast(bf16x8, x); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats to bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

struct ChunkArgs {
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* units;    // chunk units, queue by queue
  const int32_t* xcd_map;  // (first unit, count) per XCD queue
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

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void chunk_kernel(ChunkArgs A) {
  // K: [buffer][page of the step][256 x uint4], the tile as stored.
  // V: [buffer][page pair][t][half][lane] x {page 2h bytes, page 2h+1 bytes}: for channel
  // block db = 2 t + half, lane l's 16 bytes are exactly its PV A operand (4 slots of
  // each page of the pair), so the PV loop reads operands with one ds_read_b128.
  // One array per K stage: the direct memory-to-LDS copies of one stage then never
  // make the compiler wait before LDS reads of another.
  __shared__ __align__(16) uint4 ldk0[kStepPages][256];
  __shared__ __align__(16) uint4 ldk1[kStepPages][256];
  __shared__ __align__(16) uint4 ldk2[kStepPages][256];
  __shared__ __align__(16) uint4 ldk3[kStepPages][256];
  __shared__ __align__(16) uint2 ldv[kBufs][kStepPages / 2][4][2][64][2];
  __shared__ __align__(16) int lds_ids[kMaxIds];  // the tile's block-table row
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  // K stage s & 3 (s a compile-time step index).
  auto kst = [&](auto s_tag) -> uint4 (&)[kStepPages][256] {
    constexpr int st = decltype(s_tag)::value & 3;
    if constexpr (st == 0) return ldk0;
    else if constexpr (st == 1) return ldk1;
    else if constexpr (st == 2) return ldk2;
    else return ldk3;
  };

  const int xcd = blockIdx.x % kNumXcds;
  const int slot = blockIdx.x / kNumXcds;
  if (slot >= A.xcd_map[2 * xcd + 1]) return;  // this queue is shorter than the longest
  const int32_t* u = A.units + size_t(A.xcd_map[2 * xcd] + slot) * kUnitInts;
  const int b = u[U_B], g = u[U_G], kv1 = u[U_KV1];
  const int q0 = u[U_Q0], q1 = u[U_Q1], row0 = u[U_ROW0], prior = u[U_PRIOR];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, quad = lane >> 4;
  const int G = A.group;

  int tok[kNB], lim[kNB], head[kNB];
  bf16x8 qop[kNB][4];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int r = (kNB * wave + nb) * 16 + col;  // row of the tile, token-major
    const int t = q0 + r / G;
    head[nb] = r % G;
    const bool ok = t < q1;
    tok[nb] = ok ? t : -1;
    lim[nb] = ok ? prior + t : -1;  // last visible key position
    const uint4* qrow = reinterpret_cast<const uint4*>(
        A.q + (size_t(row0 + (ok ? t : 0)) * A.hq + size_t(g) * G + head[nb]) * kDim);
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
  const int nsteps = (npages + kStepPages - 1) / kStepPages;
  const int32_t* btrow = A.bt + int64_t(b) * A.bt_stride;
  // Page p of head g starts p * page_bytes past the head's first tile (one 32 x 32 ->
  // 64-bit multiply-add per load; num_kv_heads <= 1024 keeps it in 32 bits).
  const uint32_t page_bytes = uint32_t(A.hkv) * kTileBytes;
  const int first_tok = prior + q0;   // smallest query position of the tile
  // Steps whose first key is past this need the causal / length mask.
  const int mask_key0 = min(first_tok - (kStepPages * kPage - 1), kv1 - kStepPages * kPage);

  // Staging of step `step` (its 4 page ids come from LDS in one broadcast read; pages
  // past the end re-read the last page, the id row being padded with it, so the loads
  // stay branch-free; their keys are >= kv1, so they are masked and their V zeroed).
  // K goes from memory straight into LDS stage step & 3: wave w moves 1 KiB chunks 2w and
  // 2w + 1 of the step's four 4 KiB K tiles with global_load_lds_dwordx4 (each lane 16 B,
  // written at the chunk's LDS base + 16 * lane, i.e. the tile as stored).  V comes into
  // registers: thread t holds uint4 `elem` = t % 256 of both pages of pair t / 256, and
  // stash() writes them interleaved (one 16-byte LDS store per half).
  const int vpair = tid >> 8;          // page pair of the step this thread stages V for
  const int elem = tid & 255;          // uint4 index inside a tile
  const char* v_lane = reinterpret_cast<const char*>(A.v_cache) + size_t(g) * kTileBytes +
                       size_t(elem) * 16;
  const char* k_lane = reinterpret_cast<const char*>(A.k_cache) + size_t(g) * kTileBytes +
                       size_t(lane) * 16;
  // The step's 4 page ids (from LDS, one broadcast read; global memory past the staged
  // row, uniform and rare).
  auto step_ids = [&](int step, int (&ids)[kStepPages]) {
    const int p0 = step * kStepPages;
    if (p0 + kStepPages <= kMaxIds) {
      const int4 v = *reinterpret_cast<const int4*>(&lds_ids[p0]);
      ids[0] = v.x;
      ids[1] = v.y;
      ids[2] = v.z;
      ids[3] = v.w;
    } else {
#pragma unroll
      for (int j = 0; j < kStepPages; ++j)
        ids[j] = __builtin_amdgcn_readfirstlane(btrow[min(p0 + j, npages - 1)]);
    }
  };
  // V of `step` into registers (compiler-tracked loads).
  auto fetch_v = [&](int step, uint4 (&r)[2]) {
    int ids[kStepPages];
    step_ids(step, ids);
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
      r[jj] = *reinterpret_cast<const uint4*>(
          v_lane + uint64_t(uint32_t(ids[2 * vpair + jj])) * page_bytes);
  };
  // K of `step` straight into LDS stage stage_tag & 3 (global_load_lds_dwordx4: lane l's
  // 16 bytes land at the chunk's LDS base, held in m0, + 16 l).  Written as inline
  // assembly so that the compiler does not guard every later LDS access with a wait for
  // these copies; their completion is ordered by hand: vmcnt counts them in issue order
  // with the other vector-memory loads, and the wait before each barrier covers them.
  auto copy_k = [&](int step, auto stage_tag) {
    int ids[kStepPages];
    step_ids(step, ids);
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const int c = 2 * wave + c2;  // chunk: page c / 4, quarter c % 4
      const int j = c >> 2, i = c & 3;
      const char* src = k_lane + uint64_t(uint32_t(ids[j])) * page_bytes + i * 1024;
      const uint32_t dst = __builtin_amdgcn_readfirstlane(
          uint32_t(reinterpret_cast<uintptr_t>(&kst(stage_tag)[j][i * 64])));
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(dst), "v"(src)
                   : "memory", "m0");
    }
  };
  auto stash = [&](int step, const uint4 (&r)[2]) {
    const int t = elem >> 6, ln = elem & 63;
    *reinterpret_cast<uint4*>(&ldv[step & 3][vpair][t][0][ln][0]) =
        make_uint4(r[0].x, r[0].y, r[1].x, r[1].y);
    *reinterpret_cast<uint4*>(&ldv[step & 3][vpair][t][1][ln][0]) =
        make_uint4(r[0].z, r[0].w, r[1].z, r[1].w);
  };

  // Stage the page ids once (padded to whole steps with the last id), so that each
  // prefetch is one dependent load, not two.
  const int nids = min(nsteps * kStepPages, kMaxIds);
  for (int i = tid; i < nids; i += kThreads) lds_ids[i] = btrow[min(i, npages - 1)];
  __syncthreads();

  // Scores S^T = K . Q^T of page j of a stage, both column blocks.
  auto qk_page = [&](auto stage_tag, int j, f32x4 (&sj)[kNB]) {
    uint4 kr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) kr[i] = kst(stage_tag)[j][i * 64 + lane];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[i]), qop[nb][i], a, 0, 0, 0);
      sj[nb] = a;
    }
  };

  // Step n's causal mask and running-maximum update (small, with branches): gives the
  // exponent offset -m of each column block.
  auto prepare = [&](int key0, f32x4 (&s)[kStepPages][kNB], float (&neg_m)[kNB]) {
    if (key0 > mask_key0) {
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int j = 0; j < kStepPages; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (key0 + j * kPage + 4 * quad + r > lim[nb]) s[j][nb][r] = -INFINITY;
    }
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      float mloc = -INFINITY;
#pragma unroll
      for (int j = 0; j < kStepPages; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) mloc = fmaxf(mloc, s[j][nb][r]);
      const float xmax = mloc * A.sl2;
      if (__ballot(xmax > m[nb] + kTau)) {  // wave-uniform, rare after the first steps
        float mc = fmaxf(xmax, m[nb]);
        mc = fmaxf(mc, __shfl_xor(mc, 16));
        mc = fmaxf(mc, __shfl_xor(mc, 32));
        const float alpha = m[nb] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[nb] - mc);
        l[nb] *= alpha;
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[nb][db] *= alpha;
        m[nb] = mc;
      }
      neg_m[nb] = m[nb] == -INFINITY ? 0.f : -m[nb];
    }
  };

  // Page pair h of step n: the probabilities of its two pages (consuming s[2h] and
  // s[2h + 1]), step n + 1's scores of the same two pages written back into them (from
  // stage kbuf; skipped on the last step), and O^T += V^T P^T over the pair's 32 keys
  // from stage vbuf.  Exps of one pair overlap the previous pair's PV and this pair's
  // score MFMAs.  On the last step, V of slots at or past kv1 (never written, possibly
  // NaN) is zeroed in the operands.
  auto pair = [&](int h, auto kstage_tag, int vbuf, int key0, f32x4 (&s)[kStepPages][kNB],
                  const float (&neg_m)[kNB], auto last_tag) {
    constexpr bool kLast = decltype(last_tag)::value;
    bf16x8 pop[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      float p[2][4];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          p[jj][r] = __builtin_amdgcn_exp2f(fmaf(s[2 * h + jj][nb][r], A.sl2, neg_m[nb]));
      l[nb] += ((p[0][0] + p[0][1]) + (p[0][2] + p[0][3])) + ((p[1][0] + p[1][1]) + (p[1][2] + p[1][3]));
      uint4 pb;
      pb.x = pack_bf16x2(p[0][0], p[0][1]);
      pb.y = pack_bf16x2(p[0][2], p[0][3]);
      pb.z = pack_bf16x2(p[1][0], p[1][1]);
      pb.w = pack_bf16x2(p[1][2], p[1][3]);
      pop[nb] = as_bf16x8(pb);
    }
    if constexpr (!kLast) {
      qk_page(kstage_tag, 2 * h, s[2 * h]);
      qk_page(kstage_tag, 2 * h + 1, s[2 * h + 1]);
    }
    uint4 vo[8];
#pragma unroll
    for (int db = 0; db < 8; ++db)
      vo[db] = *reinterpret_cast<const uint4*>(&ldv[vbuf][h][db >> 1][db & 1][lane][0]);
    if constexpr (kLast) {
      const int ka = min(max(kv1 - key0 - 2 * h * kPage - 4 * quad, 0), 4);
      const int kb = min(max(kv1 - key0 - (2 * h + 1) * kPage - 4 * quad, 0), 4);
      const uint32_t ma0 = ka >= 2 ? ~0u : (ka == 1 ? 0x0000FFFFu : 0u);
      const uint32_t ma1 = ka >= 4 ? ~0u : (ka == 3 ? 0x0000FFFFu : 0u);
      const uint32_t mb0 = kb >= 2 ? ~0u : (kb == 1 ? 0x0000FFFFu : 0u);
      const uint32_t mb1 = kb >= 4 ? ~0u : (kb == 3 ? 0x0000FFFFu : 0u);
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        vo[db].x &= ma0;
        vo[db].y &= ma1;
        vo[db].z &= mb0;
        vo[db].w &= mb1;
      }
    }
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb)
        acc[nb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vo[db]), pop[nb], acc[nb][db], 0, 0, 0);
  };

  // Software pipeline over steps, three LDS stages: while step n's probabilities are
  // formed and multiplied into V, step n + 1's scores are computed from its K (the two
  // are independent, so matrix and vector work interleave within each wave) and steps
  // n + 2 and n + 3 are in flight from memory.
  // Staging registers come in two sets: step n + 3 is loaded into one while step n + 2,
  // loaded a whole step earlier, waits in the other to be written to LDS at the end of
  // step n, so each load has two steps of compute to land.
  uint4 stage_a[2], stage_b[2];
  if (nsteps > 0) {
    copy_k(0, S0{});
    fetch_v(0, stage_a);
    stash(0, stage_a);
  }
  if (nsteps > 1) {
    copy_k(1, S1{});
    fetch_v(1, stage_a);
    stash(1, stage_a);
  }
  if (nsteps > 2) copy_k(2, S2{});
  // Every load issued so far (Q operands, the first stages, the direct K copies) has
  // landed: the loop's wait counts then only track the in-loop prefetch.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (nsteps > 2) fetch_v(2, stage_a);

  // One score set: each page's scores are replaced by the next step's as soon as its
  // probabilities are taken.
  f32x4 sc[kStepPages][kNB];
  if (nsteps > 0)
#pragma unroll
    for (int j = 0; j < kStepPages; ++j) qk_page(S0{}, j, sc[j]);
  // Every step before the last: no V tail to clear.  `landing` holds V of step n + 2,
  // `flying` receives V of step n + 3; the staging sets swap roles every step.  Step n
  // starts the K copy of step n + 3 (into stage n + 3, last read in step n - 2) and
  // loads V of step n + 3 between its two page pairs.  Before the closing barrier, at
  // most the two V loads of step n + 3 may still be in flight: every older load (K of
  // step n + 3 and everything of step n + 2) has landed: vmcnt(2) (vmcnt bits 3:0, expcnt
  // 6:4 and lgkmcnt 11:8 left open).  The step index modulo 4 is a compile-time tag, so
  // every K stage is a fixed array.
  using Stage = uint4[2];
  auto step = [&](int n, auto r_tag, Stage& landing, Stage& flying) {
    constexpr int r = decltype(r_tag)::value;  // n & 3
    using KRead = std::integral_constant<int, (r + 1) & 3>;
    using KCopy = std::integral_constant<int, (r + 3) & 3>;
    const int key0 = n * kStepPages * kPage;
    // Unconditional (past the end it re-loads the final step's pages, unused, into
    // stages no one reads any more), so that the waits count the same loads every step.
    copy_k(min(n + 3, nsteps - 1), KCopy{});
    float neg_m[kNB];
    prepare(key0, sc, neg_m);
    pair(0, KRead{}, r, key0, sc, neg_m, std::false_type{});
    fetch_v(min(n + 3, nsteps - 1), flying);
    pair(1, KRead{}, r, key0, sc, neg_m, std::false_type{});
    if (n + 2 < nsteps) stash(n + 2, landing);
    __builtin_amdgcn_s_waitcnt(0xF72);
    __syncthreads();
  };
  int n0 = 0;
  for (; n0 + 4 < nsteps; n0 += 4) {
    step(n0, S0{}, stage_a, stage_b);
    step(n0 + 1, S1{}, stage_b, stage_a);
    step(n0 + 2, S2{}, stage_a, stage_b);
    step(n0 + 3, S3{}, stage_b, stage_a);
  }
  // Up to three more steps before the last (n0 is a multiple of 4 here).
  if (n0 + 1 < nsteps) {
    step(n0, S0{}, stage_a, stage_b);
    if (n0 + 2 < nsteps) {
      step(n0 + 1, S1{}, stage_b, stage_a);
      if (n0 + 3 < nsteps) step(n0 + 2, S2{}, stage_a, stage_b);
    }
  }
  if (nsteps > 0) {
    const int key0 = (nsteps - 1) * kStepPages * kPage;
    float neg_m[kNB];
    prepare(key0, sc, neg_m);
    pair(0, S0{}, (nsteps - 1) & 3, key0, sc, neg_m, std::true_type{});
    pair(1, S0{}, (nsteps - 1) & 3, key0, sc, neg_m, std::true_type{});
  }

  // Epilogue: every column is owned by one wave; normalise and store.
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    float ls = l[nb];
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    if (tok[nb] < 0) continue;
    const float inv = ls > 0.f ? 1.f / ls : 0.f;
    const size_t orow = (size_t(row0 + tok[nb]) * A.hq + size_t(g) * G + head[nb]);
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
