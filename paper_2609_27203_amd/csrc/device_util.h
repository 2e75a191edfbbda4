// Wavefront and workgroup helpers shared by the HIP sources (wave64).
#pragma once
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>
#include <stdint.h>

#include "kernels.h"

namespace xlh {
namespace k {

// ============================================================ index probes
// Segment of key value v in an index: on success *seg is the s with rows
// off[s] .. off[s + 1]; false when no row has key v.
__device__ __forceinline__ bool index_segment(const IndexProbe& ix, uint32_t v, uint32_t* seg) {
  const uint32_t kk = v - (uint32_t)ix.key_lo;
  if (!ix.keys) {
    *seg = kk;
    return kk < ix.key_range;
  }
  uint32_t lo = 0, len = ix.key_range;  // first distinct key >= kk
  while (len > 0) {
    const uint32_t half = len >> 1;
    if (ix.keys[lo + half] < kk) {
      lo += half + 1;
      len -= half + 1;
    } else {
      len = half;
    }
  }
  *seg = lo;
  return lo < ix.key_range && ix.keys[lo] == kk;
}

// ============================================================ wave helpers
__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ u64 lanemask_lt() { return (1ull << lane_id()) - 1ull; }

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t t = __shfl_up(x, d, 64);
    if (lane >= d) x += t;
  }
  return x;
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan_t(T x) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    T t = __shfl_up(x, d, 64);
    if (lane >= d) x += t;
  }
  return x;
}

// Wavefront-local LDS ordering: LDS operations of one wave complete in issue
// order; this keeps the compiler from moving accesses across the point.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// SplitMix64 finalizer (Steele, Lea, Flood 2014): a bijective 64-bit mixer.
__device__ __forceinline__ u64 mix64(u64 x) {
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

__device__ __forceinline__ u64 atomic_load_agent(const u64* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

static inline unsigned grid_for(int64_t n, int per_block, int cap = 1 << 20) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

// Exclusive scan of one value per thread over the workgroup (s_w holds one
// word per wavefront); *total receives the workgroup's sum.
__device__ __forceinline__ uint32_t block_excl_scan_u32(uint32_t x, uint32_t* total, uint32_t* s_w) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(x);
  if (lane == 63) s_w[w] = incl;
  __syncthreads();
  uint32_t pre = 0, tot = 0;
  for (int k = 0; k < (int)(blockDim.x >> 6); ++k) {
    const uint32_t y = s_w[k];
    if (k < w) pre += y;
    tot += y;
  }
  __syncthreads();
  *total = tot;
  return pre + incl - x;
}

// Workgroups of `threads` threads and `lds` dynamic LDS bytes of kernel k
// that the current device keeps resident at once.
// The answer is cached per (kernel, shape, device): a round-by-round launch
// asks again every round.
template <typename Kernel>
static inline hipError_t resident_blocks(Kernel k, int threads, size_t lds, int* out) {
  struct Entry {
    const void* k;
    int threads;
    size_t lds;
    int dev, blocks;
  };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  {
    std::lock_guard<std::mutex> g(mu);
    for (const Entry& c : cache)
      if (c.k == (const void*)k && c.threads == threads && c.lds == lds && c.dev == dev) {
        *out = c.blocks;
        return hipSuccess;
      }
  }
  int cus = 0, per_cu = 0;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, threads, lds);
  if (e != hipSuccess) return e;
  *out = std::max(1, cus * std::max(1, per_cu));
  std::lock_guard<std::mutex> g(mu);
  cache.push_back(Entry{(const void*)k, threads, lds, dev, *out});
  return hipSuccess;
}

}  // namespace k
}  // namespace xlh
