// Paged KV layout kernels: pack / unpack whole pages, block-table gather, and the
// append-time cache write of new tokens.  All of them move bf16 bytes only.
//
// A (page, head) tile is 16 slots x 128 channels.  Logical order is slot-major
// (element s * 128 + d); the library order puts each element where the attention
// kernels' 16-byte lane loads expect it (see k_off / v_off).  Every kernel stages one
// tile per 256-thread block: thread t owns logical slot t / 16 and channels
// 8 * (t % 16) .. + 7, and 16 contiguous bytes of the library-order tile at 16 t.
#include <algorithm>

#include "internal.h"

namespace libra {
namespace {

constexpr int kThreads = 256;

// Position of (slot s, channel d) inside a K tile, in bf16 elements.
__device__ __forceinline__ int k_off(int s, int d) { return ((d >> 3) * 16 + s) * 8 + (d & 7); }

// Position of (slot s, channel d) inside a V tile, in bf16 elements: 16-byte granule
// 128 h + d holds channel d's slots {4 h .. 4 h + 3, 8 + 4 h .. 11 + 4 h}, h = (s / 4) % 2.
__device__ __forceinline__ int v_off(int s, int d) {
  return (128 * ((s >> 2) & 1) + d) * 8 + (s >> 3) * 4 + (s & 3);
}

__device__ __forceinline__ size_t tile_elem(int64_t page, int g, int hkv) {
  return (size_t(page) * hkv + g) * kTileElems;
}

// Scatter 8 logical channels (packed in a uint4) of slot s into an LDS V tile.
__device__ __forceinline__ void v_scatter8(uint16_t* lds, int s, int d0, uint4 val) {
  const uint16_t* e = reinterpret_cast<const uint16_t*>(&val);
#pragma unroll
  for (int i = 0; i < 8; ++i) lds[v_off(s, d0 + i)] = e[i];
}

__device__ __forceinline__ uint4 v_gather8(const uint16_t* lds, int s, int d0) {
  uint4 r;
  uint16_t* e = reinterpret_cast<uint16_t*>(&r);
#pragma unroll
  for (int i = 0; i < 8; ++i) e[i] = lds[v_off(s, d0 + i)];
  return r;
}

// grid.x = tiles (page, head) in [first * hkv, (first + n) * hkv)
__global__ __launch_bounds__(kThreads) void pack_kernel(const uint16_t* __restrict__ k_src,
                                                        const uint16_t* __restrict__ v_src,
                                                        uint16_t* __restrict__ k_dst,
                                                        uint16_t* __restrict__ v_dst,
                                                        int64_t first_tile) {
  __shared__ __align__(16) uint16_t vt[kTileElems];
  const int t = threadIdx.x;
  const int s = t >> 4, d0 = (t & 15) * 8;
  const size_t src = size_t(blockIdx.x) * kTileElems;
  const size_t dst = size_t(first_tile + blockIdx.x) * kTileElems;
  if (k_src) {
    const uint4 k = *reinterpret_cast<const uint4*>(k_src + src + s * kDim + d0);
    *reinterpret_cast<uint4*>(k_dst + dst + k_off(s, d0)) = k;
  }
  if (v_src) {
    const uint4 v = *reinterpret_cast<const uint4*>(v_src + src + s * kDim + d0);
    v_scatter8(vt, s, d0, v);
    __syncthreads();
    *reinterpret_cast<uint4*>(v_dst + dst + t * 8) = *reinterpret_cast<const uint4*>(vt + t * 8);
  }
}

__global__ __launch_bounds__(kThreads) void unpack_kernel(const uint16_t* __restrict__ k_src,
                                                          const uint16_t* __restrict__ v_src,
                                                          uint16_t* __restrict__ k_dst,
                                                          uint16_t* __restrict__ v_dst,
                                                          int64_t first_tile) {
  __shared__ __align__(16) uint16_t vt[kTileElems];
  const int t = threadIdx.x;
  const int s = t >> 4, d0 = (t & 15) * 8;
  const size_t src = size_t(first_tile + blockIdx.x) * kTileElems;
  const size_t dst = size_t(blockIdx.x) * kTileElems;
  if (k_dst) {
    *reinterpret_cast<uint4*>(k_dst + dst + s * kDim + d0) =
        *reinterpret_cast<const uint4*>(k_src + src + k_off(s, d0));
  }
  if (v_dst) {
    *reinterpret_cast<uint4*>(vt + t * 8) = *reinterpret_cast<const uint4*>(v_src + src + t * 8);
    __syncthreads();
    *reinterpret_cast<uint4*>(v_dst + dst + s * kDim + d0) = v_gather8(vt, s, d0);
  }
}

// grid = (max_pages, batch, hkv); block (p, b, g) copies page p of sequence b, head g.
__global__ __launch_bounds__(kThreads) void gather_kernel(
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ bt, int32_t stride, const int32_t* __restrict__ cu, int hkv,
    uint16_t* __restrict__ k_out, uint16_t* __restrict__ v_out) {
  __shared__ __align__(16) uint16_t vt[kTileElems];
  const int p = blockIdx.x, b = blockIdx.y, g = blockIdx.z;
  const int64_t row0 = cu[b];
  const int64_t len = int64_t(cu[b + 1]) - row0;
  if (int64_t(p) * kPage >= len) return;  // uniform per block
  const int t = threadIdx.x;
  const int s = t >> 4, d0 = (t & 15) * 8;
  const int64_t page = bt[int64_t(b) * stride + p];
  const size_t base = tile_elem(page, g, hkv);
  *reinterpret_cast<uint4*>(vt + t * 8) = *reinterpret_cast<const uint4*>(v_cache + base + t * 8);
  __syncthreads();
  const int64_t tok = int64_t(p) * kPage + s;
  if (tok < len) {
    const size_t o = (size_t(row0 + tok) * hkv + g) * kDim + d0;
    *reinterpret_cast<uint4*>(k_out + o) =
        *reinterpret_cast<const uint4*>(k_cache + base + k_off(s, d0));
    *reinterpret_cast<uint4*>(v_out + o) = v_gather8(vt, s, d0);
  }
}

// grid = (n_write_tiles, hkv).  Record w = (b, logical page, slot0, slot1, row of slot0).
// K elements of a slot are contiguous, so new K rows are stored directly; a V slot is
// spread over the tile, so the V tile is read, patched in LDS and written back whole.
__global__ __launch_bounds__(kThreads) void cache_write_kernel(
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ writes, const int32_t* __restrict__ bt, int32_t stride, int hkv,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new) {
  __shared__ __align__(16) uint16_t vt[kTileElems];
  const int32_t* w = writes + size_t(blockIdx.x) * kWriteInts;
  const int g = blockIdx.y;
  const int b = w[W_B], pg = w[W_PAGE], s0 = w[W_SLOT0], s1 = w[W_SLOT1], row = w[W_ROW];
  const int64_t page = bt[int64_t(b) * stride + pg];
  const size_t base = tile_elem(page, g, hkv);
  const int t = threadIdx.x;
  const int s = t >> 4, d0 = (t & 15) * 8;
  // A page whose 16 slots are all new is overwritten whole: its old V tile is not read.
  // s0 and s1 are uniform over the block, so the barrier below is reached by all threads.
  if (s1 - s0 < kPage)
    *reinterpret_cast<uint4*>(vt + t * 8) = *reinterpret_cast<const uint4*>(v_cache + base + t * 8);
  __syncthreads();
  if (s >= s0 && s < s1) {
    const size_t src = (size_t(row + s - s0) * hkv + g) * kDim + d0;
    *reinterpret_cast<uint4*>(k_cache + base + k_off(s, d0)) =
        *reinterpret_cast<const uint4*>(k_new + src);
    v_scatter8(vt, s, d0, *reinterpret_cast<const uint4*>(v_new + src));
  }
  __syncthreads();
  *reinterpret_cast<uint4*>(v_cache + base + t * 8) = *reinterpret_cast<const uint4*>(vt + t * 8);
}

// Moves whole (page, head) tiles between the cache and a packed page run (request
// offload and reload): run tile r = i * hkv + g holds tile g of page ids[i].  A tile is
// 256 lanes x 16 bytes, so each block-iteration moves one K and one V tile; blocks stride
// over the run.  Ids outside [0, num_pages) are skipped.
template <bool kToRun>
__global__ __launch_bounds__(kThreads) void page_copy_kernel(uint4* __restrict__ k_cache,
                                                             uint4* __restrict__ v_cache,
                                                             const int32_t* __restrict__ ids,
                                                             int64_t num_pages, int hkv,
                                                             int64_t tiles,
                                                             uint4* __restrict__ k_run,
                                                             uint4* __restrict__ v_run) {
  const int t = threadIdx.x;
  for (int64_t r = blockIdx.x; r < tiles; r += gridDim.x) {
    const int64_t i = r / hkv;
    const int g = int(r - i * hkv);
    const int64_t page = ids[i];
    if (page < 0 || page >= num_pages) continue;  // uniform per block
    const size_t c = (size_t(page) * hkv + g) * kThreads + t;
    const size_t q = size_t(r) * kThreads + t;
    if (kToRun) {
      if (k_run) k_run[q] = k_cache[c];
      if (v_run) v_run[q] = v_cache[c];
    } else {
      if (k_run) k_cache[c] = k_run[q];
      if (v_run) v_cache[c] = v_run[q];
    }
  }
}

}  // namespace

// One workgroup per tile; a 1-D grid holds at most 2^32 - 1 work-items, so long page
// ranges go in launches of kMaxTilesPerLaunch tiles (the long-tailed batch packs in 3).
constexpr int64_t kMaxTilesPerLaunch = int64_t(1) << 18;

hipError_t launch_pack(const KvLayout& L, const void* k_src, const void* v_src, int64_t first,
                       int64_t n, hipStream_t s) {
  const int hkv = L.desc.num_kv_heads;
  const int64_t tiles = n * hkv;
  const uint16_t* ks = static_cast<const uint16_t*>(k_src);
  const uint16_t* vs = static_cast<const uint16_t*>(v_src);
  for (int64_t t0 = 0; t0 < tiles; t0 += kMaxTilesPerLaunch) {
    const int64_t nt = std::min(kMaxTilesPerLaunch, tiles - t0);
    const size_t off = size_t(t0) * kTileElems;
    hipLaunchKernelGGL(pack_kernel, dim3(unsigned(nt)), dim3(kThreads), 0, s, ks ? ks + off : ks,
                       vs ? vs + off : vs, static_cast<uint16_t*>(L.desc.k_cache),
                       static_cast<uint16_t*>(L.desc.v_cache), first * hkv + t0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_unpack(const KvLayout& L, void* k_dst, void* v_dst, int64_t first, int64_t n,
                         hipStream_t s) {
  const int hkv = L.desc.num_kv_heads;
  const int64_t tiles = n * hkv;
  uint16_t* kd = static_cast<uint16_t*>(k_dst);
  uint16_t* vd = static_cast<uint16_t*>(v_dst);
  for (int64_t t0 = 0; t0 < tiles; t0 += kMaxTilesPerLaunch) {
    const int64_t nt = std::min(kMaxTilesPerLaunch, tiles - t0);
    const size_t off = size_t(t0) * kTileElems;
    hipLaunchKernelGGL(unpack_kernel, dim3(unsigned(nt)), dim3(kThreads), 0, s,
                       static_cast<const uint16_t*>(L.desc.k_cache),
                       static_cast<const uint16_t*>(L.desc.v_cache), kd ? kd + off : kd,
                       vd ? vd + off : vd, first * hkv + t0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_gather(const KvLayout& L, const int32_t* bt, int32_t stride, const int32_t* cu,
                         int32_t batch, int32_t max_pages, void* k_out, void* v_out,
                         hipStream_t s) {
  if (batch == 0 || max_pages == 0) return hipSuccess;
  const int hkv = L.desc.num_kv_heads;
  hipLaunchKernelGGL(gather_kernel, dim3(unsigned(max_pages), unsigned(batch), unsigned(hkv)),
                     dim3(kThreads), 0, s, static_cast<const uint16_t*>(L.desc.k_cache),
                     static_cast<const uint16_t*>(L.desc.v_cache), bt, stride, cu, hkv,
                     static_cast<uint16_t*>(k_out), static_cast<uint16_t*>(v_out));
  return hipGetLastError();
}

hipError_t launch_cache_write(const KvLayout& L, const Plan& P, const void* ws, const void* k_new,
                              const void* v_new, const int32_t* bt, int32_t stride,
                              hipStream_t s) {
  const int n = P.info.n_write_tiles;
  if (n == 0) return hipSuccess;
  const int hkv = L.desc.num_kv_heads;
  const int32_t* writes =
      reinterpret_cast<const int32_t*>(static_cast<const char*>(ws) + P.off_writes);
  hipLaunchKernelGGL(cache_write_kernel, dim3(unsigned(n), unsigned(hkv)), dim3(kThreads), 0, s,
                     static_cast<uint16_t*>(L.desc.k_cache), static_cast<uint16_t*>(L.desc.v_cache),
                     writes, bt, stride, hkv, static_cast<const uint16_t*>(k_new),
                     static_cast<const uint16_t*>(v_new));
  return hipGetLastError();
}

hipError_t launch_page_copy(const KvLayout& L, const int32_t* ids, int64_t n, void* k_run,
                            void* v_run, bool to_run, hipStream_t s) {
  const int hkv = L.desc.num_kv_heads;
  const int64_t tiles = n * hkv;
  if (tiles == 0) return hipSuccess;
  const unsigned blocks = unsigned(std::min<int64_t>(tiles, 16384));
  auto kern = to_run ? page_copy_kernel<true> : page_copy_kernel<false>;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(kThreads), 0, s,
                     static_cast<uint4*>(L.desc.k_cache), static_cast<uint4*>(L.desc.v_cache), ids,
                     L.desc.num_pages, hkv, tiles, static_cast<uint4*>(k_run),
                     static_cast<uint4*>(v_run));
  return hipGetLastError();
}

}  // namespace libra
