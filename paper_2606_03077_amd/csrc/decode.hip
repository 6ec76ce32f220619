// Decode attention over the paged KV cache, one 256-thread workgroup per plan unit.
//
// A unit is (sequence b, KV head g, KV range [kv0, kv1)).  Its pages are shared out to
// the 4 wavefronts in contiguous quarters.  For each page a wave issues four 16-byte K
// loads and eight 8-byte V loads per lane (the layout makes each K load one contiguous
// 1 KiB wave-wide read, each V load two 256 B runs) one page ahead of the math, then on
// the matrix cores:
//
//   S^T[16 slots x 16 heads] = K[16 x 128] . Q^T[128 x 16]    (4 x mfma 16x16x32)
//   O^T[128 x 16 heads]     += V^T[128 x 16 slots] . P^T[16 x 16]  (8 x mfma 16x16x16)
//
// The G query heads sharing KV head g are the 16 matrix columns (zero-padded when
// G < 16).  The QK^T result layout (lane = column + 16 * key-quad) is exactly the
// B-operand layout of the PV product, so P never leaves registers.  Latency is hidden
// by occupancy (several workgroups per CU) rather than deep per-wave buffering.  Softmax runs online
// in base 2 with the scale folded in; column maxima use two cross-lane shuffles.
// The 4 waves' (max, sum, accumulator) are merged through LDS.  A unit that covers the
// whole row writes bf16 O and the float32 LSE; a split writes a float32 partial, and
// merge_kernel (merge.hip), launched next on the same stream, combines the partials of
// each split row by their log-sum-exps (the launch boundary orders the two without
// device-wide cache flushes inside either kernel).
#include <cmath>

#include "internal.h"

namespace libra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#ifndef LIBRA_DECODE_WAVES
#define LIBRA_DECODE_WAVES 4
#endif
constexpr int kWaves = LIBRA_DECODE_WAVES;
constexpr int kThreads = 64 * kWaves;
#ifndef LIBRA_DECODE_DEPTH
#define LIBRA_DECODE_DEPTH 2
#endif
#ifndef LIBRA_DECODE_WAVES_PER_EU
#define LIBRA_DECODE_WAVES_PER_EU 3
#endif
constexpr int kDepth = LIBRA_DECODE_DEPTH;  // pages of K/V held in registers per wave
constexpr int kRedStride = 132;  // padded row of the LDS accumulator exchange
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct PageRegs {
  uint4 k[4];  // K tile, 16 B per lane per 1 KiB quarter
  uint2 v[8];  // V: this lane's 4 slots of one channel for each 16-channel block
};

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 x) { return __builtin_bit_cast(bf16x8, x); }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// K/V bytes are read exactly once per call: non-temporal loads keep them from
// displacing reusable lines and measurably raise the sustained random-tile read rate.
__device__ __forceinline__ uint4 stream_load(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint2 stream_load2(const uint2* p) {
  const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
  return make_uint2(v.x, v.y);
}

// V of lane (i, quad) for channel block db: slots 4 quad .. + 3 of channel 16 db + i, the
// half quad / 2 of granule 128 (quad % 2) + 16 db + i (8 bytes; a wave reads two runs of
// 256 contiguous bytes per block).
__device__ __forceinline__ void load_page(PageRegs& r, const uint4* kt, const uint2* vt, int lane) {
#pragma unroll
  for (int i = 0; i < 4; ++i) r.k[i] = stream_load(kt + i * 64 + lane);
  const int col = lane & 15, quad = lane >> 4;
#pragma unroll
  for (int db = 0; db < 8; ++db)
    r.v[db] = stream_load2(vt + 2 * (128 * (quad & 1) + 16 * db + col) + (quad >> 1));
}

// Zero V of slots >= valid (slot = 4 * quad + r): keeps NaN/garbage of unused slots
// out of the PV product, where a zero probability alone would not.
__device__ __forceinline__ void clear_v_slots(PageRegs& r, int quad, int valid) {
  const int keep = min(max(valid - 4 * quad, 0), 4);  // slots of this lane that hold tokens
  if (keep == 4) return;
  // each 8-byte half holds slots 4q+0..3 as bf16 pairs (x: r0,r1  y: r2,r3)
  const uint32_t m0 = keep >= 2 ? 0xFFFFFFFFu : (keep == 1 ? 0x0000FFFFu : 0u);
  const uint32_t m1 = keep >= 4 ? 0xFFFFFFFFu : (keep == 3 ? 0x0000FFFFu : 0u);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    r.v[i].x &= m0;
    r.v[i].y &= m1;
  }
}

__device__ __forceinline__ f32x4 qk_page(const PageRegs& r, const bf16x8 (&qop)[4]) {
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 4; ++i) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(r.k[i]), qop[i], s, 0, 0, 0);
  return s;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats to bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

struct Softmax {
  float m;  // running max (base-2 logits), uniform over the 4 lanes of a column
  float l;  // this lane's share of the running sum
};

typedef short bf16x4_bits __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x4_bits as_bf16x4(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(bf16x4_bits, make_uint2(lo, hi));
}

// One page: scores, online softmax update, PV accumulate.
//   S^T[16 slots x 16 heads]: 4 x mfma 16x16x32 (k = channels);
//   O^T[128 x 16 heads] += V^T[128 x 16 slots] . P^T: 8 x mfma 16x16x16 (k = slots),
// whose B operand (lane = head + 16 * quad, slots 4 quad .. + 3) is exactly the score
// tile's accumulator layout, so probabilities never leave registers.
__device__ __forceinline__ void process_page(const PageRegs& r, int valid, int quad,
                                             const bf16x8 (&qop)[4], float sl2, Softmax& sm,
                                             f32x4 (&acc)[8]) {
  const f32x4 s = qk_page(r, qop);
  float x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = 4 * quad + i < valid ? s[i] * sl2 : -INFINITY;
  float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(sm.m, mx);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = __builtin_amdgcn_exp2f(sm.m - m_use);
  float p[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(x[i] - m_use);
  sm.l = sm.l * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
  sm.m = m_new;
  const bf16x4_bits pop = as_bf16x4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]));
#pragma unroll
  for (int db = 0; db < 8; ++db) {
    const bf16x4_bits vop = as_bf16x4(r.v[db].x, r.v[db].y);
    acc[db] *= alpha;
    acc[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, pop, acc[db], 0, 0, 0);
  }
}

struct DecodeArgs {
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* units;
  const int32_t* bt;
  const uint16_t* q;
  uint16_t* out;
  float* lse;
  float* part_o;
  float* part_lse;
  int64_t bt_stride;
  int hkv;
  int hq;
  int group;
  float sl2;  // scale * log2(e)
};

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(LIBRA_DECODE_WAVES_PER_EU, 8))) void decode_kernel(DecodeArgs A) {
  __shared__ float red_m[kWaves][16];
  __shared__ float red_l[kWaves][16];
  __shared__ __align__(16) float red_o[kWaves][16][kRedStride];

  const int32_t* u = A.units + size_t(blockIdx.x) * kUnitInts;
  const int b = u[U_B], g = u[U_G], kv0 = u[U_KV0], kv1 = u[U_KV1];
  const int nsplit = u[U_NSPLIT], part = u[U_PART], row = u[U_ROW0], split = u[U_SPLIT];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, quad = lane >> 4;
  const int G = A.group;

  // Q operand: lane (col, quad) holds head col's channels 8 * (4 i + quad) .. + 7 at step i.
  bf16x8 qop[4];
  {
    const uint4* qrow = reinterpret_cast<const uint4*>(
        A.q + (size_t(row) * A.hq + size_t(g) * G + col) * kDim);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (col < G) v = qrow[4 * i + quad];
      qop[i] = as_bf16x8(v);
    }
  }

  // This wave's pages: a contiguous quarter of the unit's pages.
  const int p0 = kv0 / kPage;
  const int p1 = (kv1 + kPage - 1) / kPage;
  const int np = p1 - p0;
  const int w0 = p0 + (wave * np) / kWaves;
  const int nw = p0 + ((wave + 1) * np) / kWaves - w0;

  Softmax sm{-INFINITY, 0.f};
  f32x4 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nw > 0) {
    const int32_t* btrow = A.bt + int64_t(b) * A.bt_stride + w0;
    // Page ids in 64-entry windows, the next window loaded one window ahead.
    int ids_cur = lane < nw ? btrow[lane] : 0;
    int ids_nxt = lane + 64 < nw ? btrow[lane + 64] : 0;
    int win = 0;  // first page index (relative to w0) held by ids_cur
    const size_t head_off = size_t(g) * kTileElems;
    const size_t page_stride = size_t(A.hkv) * kTileElems;
    auto issue = [&](int k, PageRegs& r) {
      if (k - win >= 64) {  // wave-uniform: advance the id window
        ids_cur = ids_nxt;
        win += 64;
        ids_nxt = lane + win + 64 < nw ? btrow[lane + win + 64] : 0;
      }
      const int64_t page = __builtin_amdgcn_readlane(ids_cur, k - win);
      const size_t base = size_t(page) * page_stride + head_off;
      load_page(r, reinterpret_cast<const uint4*>(A.k_cache + base),
                reinterpret_cast<const uint2*>(A.v_cache + base), lane);
    };
    auto consume = [&](PageRegs& r, int k) {
      const int valid = min(kPage, kv1 - (w0 + k) * kPage);
      if (valid < kPage) clear_v_slots(r, quad, valid);
      process_page(r, valid, quad, qop, A.sl2, sm, acc);
    };

    // Ring of kDepth pages: page k + kDepth is issued into the registers page k has
    // just been consumed from, so kDepth - 1 pages stay in flight during the math.
    PageRegs ring[kDepth];
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
      if (j < nw) issue(j, ring[j]);
    for (int k = 0; k < nw; k += kDepth) {
#pragma unroll
      for (int j = 0; j < kDepth; ++j) {
        if (k + j < nw) {
          consume(ring[j], k + j);
          if (k + j + kDepth < nw) issue(k + j + kDepth, ring[j]);
        }
      }
    }
  }

  // Column sum over the 4 key quads.
  float lsum = sm.l;
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (quad == 0) {
    red_m[wave][col] = sm.m;
    red_l[wave][col] = lsum;
  }
  __syncthreads();
  float M = red_m[0][col];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) M = fmaxf(M, red_m[w][col]);
  const float f = (M == -INFINITY || sm.m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(sm.m - M);
#pragma unroll
  for (int db = 0; db < 8; ++db) {
    *reinterpret_cast<f32x4*>(&red_o[wave][col][db * 16 + quad * 4]) = acc[db] * f;
  }
  __syncthreads();

  // The first 256 threads each finish 8 channels of one column (head).
  if (tid >= 256) return;
  const int hcol = tid >> 4, c8 = (tid & 15) * 8;
  float Mh = red_m[0][hcol];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) Mh = fmaxf(Mh, red_m[w][hcol]);
  float Lh = 0.f;
  if (Mh != -INFINITY) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = red_m[w][hcol];
      if (mw != -INFINITY) Lh += __builtin_amdgcn_exp2f(mw - Mh) * red_l[w][hcol];
    }
  }
  float o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += red_o[w][hcol][c8 + i];
    o[i] = Lh > 0.f ? s / Lh : 0.f;
  }
  const float lse2 = Lh > 0.f ? Mh + log2f(Lh) : -INFINITY;
  const size_t head = size_t(g) * G + hcol;

  if (nsplit == 1) {
    if (hcol < G) {
      uint4 ov;
      ov.x = pack_bf16x2(o[0], o[1]);
      ov.y = pack_bf16x2(o[2], o[3]);
      ov.z = pack_bf16x2(o[4], o[5]);
      ov.w = pack_bf16x2(o[6], o[7]);
      *reinterpret_cast<uint4*>(A.out + (size_t(row) * A.hq + head) * kDim + c8) = ov;
      if (A.lse && (tid & 15) == 0) A.lse[size_t(row) * A.hq + head] = lse2 * kLn2;
    }
    return;
  }

  // Split: store this range's normalised float32 partial and its base-2 log-sum-exp;
  // merge_kernel combines the splits after this launch.
  const size_t slot = size_t(part) + split;
  if (hcol < G) {
    float* po = A.part_o + (slot * G + hcol) * kDim + c8;
    *reinterpret_cast<f32x4*>(po) = f32x4{o[0], o[1], o[2], o[3]};
    *reinterpret_cast<f32x4*>(po + 4) = f32x4{o[4], o[5], o[6], o[7]};
    if ((tid & 15) == 0) A.part_lse[slot * G + hcol] = lse2;
  }
}

}  // namespace

hipError_t launch_decode(const KvLayout& L, const Plan& P, void* ws, const void* q,
                         const int32_t* bt, int32_t stride, float scale, void* out, float* lse,
                         hipStream_t s) {
  const int n = P.info.n_single;
  if (n == 0) return hipSuccess;
  char* w = static_cast<char*>(ws);
  DecodeArgs A;
  A.k_cache = static_cast<const uint16_t*>(L.desc.k_cache);
  A.v_cache = static_cast<const uint16_t*>(L.desc.v_cache);
  A.units = reinterpret_cast<const int32_t*>(w + P.off_units);
  A.bt = bt;
  A.q = static_cast<const uint16_t*>(q);
  A.out = static_cast<uint16_t*>(out);
  A.lse = lse;
  A.part_o = reinterpret_cast<float*>(w + P.off_part_o);
  A.part_lse = reinterpret_cast<float*>(w + P.off_part_lse);
  A.bt_stride = stride;
  A.hkv = P.num_kv_heads;
  A.hq = P.num_q_heads;
  A.group = P.group;
  A.sl2 = scale * kLog2e;
  hipLaunchKernelGGL(decode_kernel, dim3(unsigned(n)), dim3(kThreads), 0, s, A);
  return hipGetLastError();
}

}  // namespace libra
