// Log-sum-exp merge of split rows: the float32 partials that decode units wrote for
// the pieces of one (sequence, KV head) row become its bf16 output and float32 LSE.
//
// One 256-thread block per split row.  Its threads form ngroups = max(1, 256 / (16 G))
// groups of 16 G threads; in a group, thread t finishes channels 8 (t % 16) .. + 7 of
// query head t / 16 of the group.  Group k folds splits k, k + ngroups, k + 2 ngroups, ...
// eight at a time (all loads of a batch in flight together) with a running maximum, so a
// row of n splits takes about n / (8 ngroups) dependent rounds of loads; the groups'
// (max, sum, accumulator) then combine through LDS in group order.  With M = max_j lse_j
// (base 2): lse = M + log2(sum_j 2^(lse_j - M)), o = sum_j 2^(lse_j - lse) o_j; empty
// splits (lse_j = -inf) add nothing.
#include <cmath>

#include "internal.h"

namespace libra {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kBatch = 8;
constexpr float kLn2 = 0.6931471805599453f;

// Two floats to bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

struct MergeArgs {
  const int32_t* merges;
  const float* part_o;
  const float* part_lse;
  uint16_t* out;
  float* lse;
  int hq;
  int group;
};

__global__ __launch_bounds__(kThreads) void merge_kernel(MergeArgs A) {
  __shared__ float red_m[kThreads];
  __shared__ float red_w[kThreads];
  __shared__ float red_acc[kThreads][9];  // padded row

  const int32_t* m = A.merges + size_t(blockIdx.x) * kMergeInts;
  const int g = m[M_G], n = m[M_N], part = m[M_PART], row = m[M_ROW];
  const int G = A.group;
  const int per = 16 * G;
  const int ngroups = max(1, kThreads / per);
  const int tid = threadIdx.x;
  const int grp = tid / per, t = tid - grp * per;
  const int hcol = t >> 4, c8 = (t & 15) * 8;

  float M = -INFINITY, wsum = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (grp < ngroups) {
    for (int j0 = grp; j0 < n; j0 += kBatch * ngroups) {
      float lj[kBatch];
      f32x4 x0[kBatch], x1[kBatch];
#pragma unroll
      for (int jj = 0; jj < kBatch; ++jj) {
        const int j = j0 + jj * ngroups;
        lj[jj] = -INFINITY;
        x0[jj] = x1[jj] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (j < n) {
          const size_t slot = size_t(part + j) * G + hcol;
          lj[jj] = A.part_lse[slot];
          const float* po = A.part_o + slot * kDim + c8;
          x0[jj] = *reinterpret_cast<const f32x4*>(po);
          x1[jj] = *reinterpret_cast<const f32x4*>(po + 4);
        }
      }
      float Mc = M;
#pragma unroll
      for (int jj = 0; jj < kBatch; ++jj) Mc = fmaxf(Mc, lj[jj]);
      if (Mc == -INFINITY) continue;
      const float r = __builtin_amdgcn_exp2f(M - Mc);  // 0 while M = -inf
      wsum *= r;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] *= r;
#pragma unroll
      for (int jj = 0; jj < kBatch; ++jj) {
        const float w = __builtin_amdgcn_exp2f(lj[jj] - Mc);  // 0 for empty or absent splits
        wsum += w;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[i] += w * x0[jj][i];
          acc[4 + i] += w * x1[jj][i];
        }
      }
      M = Mc;
    }
  }
  if (ngroups > 1) {  // block-uniform
    red_m[tid] = M;
    red_w[tid] = wsum;
#pragma unroll
    for (int i = 0; i < 8; ++i) red_acc[tid][i] = acc[i];
    __syncthreads();
    if (grp != 0) return;
    for (int k = 1; k < ngroups; ++k) {
      const int o = k * per + t;
      const float Mk = red_m[o];
      const float Mn = fmaxf(M, Mk);
      if (Mn == -INFINITY) continue;
      const float a = __builtin_amdgcn_exp2f(M - Mn), b = __builtin_amdgcn_exp2f(Mk - Mn);
      wsum = wsum * a + red_w[o] * b;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = acc[i] * a + red_acc[o][i] * b;
      M = Mn;
    }
  } else if (grp != 0) {
    return;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  uint4 ov;
  ov.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  ov.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  ov.z = pack_bf16x2(acc[4] * inv, acc[5] * inv);
  ov.w = pack_bf16x2(acc[6] * inv, acc[7] * inv);
  const size_t head = size_t(g) * G + hcol;
  *reinterpret_cast<uint4*>(A.out + (size_t(row) * A.hq + head) * kDim + c8) = ov;
  if (A.lse && (tid & 15) == 0)
    A.lse[size_t(row) * A.hq + head] = wsum > 0.f ? (M + log2f(wsum)) * kLn2 : -INFINITY;
}

}  // namespace

bool merge_launches(const Plan& P) { return P.info.n_merge_groups > 0; }

hipError_t launch_merge(const Plan& P, void* ws, void* out, float* lse, hipStream_t s) {
  const int n = P.info.n_merge_groups;
  if (!merge_launches(P)) return hipSuccess;
  char* w = static_cast<char*>(ws);
  MergeArgs A;
  A.merges = reinterpret_cast<const int32_t*>(w + P.off_merges);
  A.part_o = reinterpret_cast<const float*>(w + P.off_part_o);
  A.part_lse = reinterpret_cast<const float*>(w + P.off_part_lse);
  A.out = static_cast<uint16_t*>(out);
  A.lse = lse;
  A.hq = P.num_q_heads;
  A.group = P.group;
  hipLaunchKernelGGL(merge_kernel, dim3(unsigned(n)), dim3(kThreads), 0, s, A);
  return hipGetLastError();
}

}  // namespace libra
