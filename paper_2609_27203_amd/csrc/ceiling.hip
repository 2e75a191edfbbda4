// On-chip ceiling of the frontier kernel's per-candidate step, for pricing
// that kernel against what the chip can do (a measurement kernel: it derives
// nothing).  The frontier kernel keeps each first key's rows in LDS, so its
// candidates cost no HBM traffic; what each one costs is a 4-byte load from
// an index column that L2 holds (an out-neighbour when pushing, an in-edge
// source when pulling), then a test of that value's bit in a 2 KB row in LDS
// and, when the bit is clear, an LDS atomic OR.  This kernel does exactly
// that step with nothing else in the way: every lane keeps CE_UNROLL loads
// in flight, no load depends on an earlier one and no workgroup waits at a
// barrier.  It takes the frontier kernel's workgroup size and LDS footprint,
// so it runs at the same occupancy.  Addresses are either independent
// pseudo-random slots of the column (a pull's in-edge lists, a push's small
// rows) or 64 consecutive slots per wavefront (a push's large rows).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace {

constexpr int CE_THREADS = 256;
constexpr int CE_UNROLL = 8;
constexpr uint32_t CE_ROW_WORDS = 512;  // one 2 KB bitmap row (16,384 targets)

__global__ __launch_bounds__(CE_THREADS) void candidate_ceiling_k(const uint32_t* col, uint32_t mask, uint32_t iters,
                                                                   int consecutive, unsigned long long* out) {
  extern __shared__ uint32_t row[];  // the first CE_ROW_WORDS words are the row; the rest only sets occupancy
  for (uint32_t i = threadIdx.x; i < CE_ROW_WORDS; i += CE_THREADS) row[i] = 0u;
  __syncthreads();
  const uint32_t lane = threadIdx.x & 63u;
  const uint64_t wave = ((uint64_t)blockIdx.x * CE_THREADS + threadIdx.x) >> 6;
  uint32_t x = (uint32_t)(blockIdx.x * CE_THREADS + threadIdx.x) * 0x9E3779B9u + 0x7F4A7C15u;
  uint32_t set = 0;
  for (uint32_t it = 0; it < iters; ++it) {
    uint32_t y[CE_UNROLL];
#pragma unroll
    for (int u = 0; u < CE_UNROLL; ++u) {
      uint32_t idx;
      if (consecutive) {
        idx = (uint32_t)(((wave * iters + it) * CE_UNROLL + (uint32_t)u) * 64u + lane) & mask;
      } else {
        x = x * 1664525u + 1013904223u;  // the 32-bit LCG of Numerical Recipes
        idx = (x >> 7) & mask;
      }
      y[u] = col[idx];
    }
#pragma unroll
    for (int u = 0; u < CE_UNROLL; ++u) {
      const uint32_t b = y[u] & (CE_ROW_WORDS * 32u - 1u);
      const uint32_t bit = 1u << (b & 31u);
      if (!(row[b >> 5] & bit)) {
        atomicOr(&row[b >> 5], bit);
        ++set;
      }
    }
  }
  __syncthreads();
  uint32_t c = 0;
  for (uint32_t i = threadIdx.x; i < CE_ROW_WORDS; i += CE_THREADS) c += (uint32_t)__popc(row[i]);
  if (c + set) atomicAdd(out, (unsigned long long)(c + set));
}

}  // namespace

extern "C" {

// Runs the ceiling kernel once on `stream` over the device column `col`
// (n_pow2 entries, a power of two; values are taken modulo 16,384), with
// 256-thread workgroups holding lds_bytes of LDS each (at least 2 KB), as
// many as fit on the device at once, `iters` steps of CE_UNROLL candidates
// per thread.  `out` is 8 bytes of device memory the kernel sums the set
// bits into (keeps its work observable).  Writes the candidates processed
// and the kernel's duration (HIP events on the stream; the call waits for
// it).  Returns 0, or a HIP error code.
int xlh_candidate_ceiling(const uint32_t* col, uint64_t n_pow2, uint32_t iters, int consecutive, size_t lds_bytes,
                          unsigned long long* out, void* stream, unsigned long long* candidates, float* ms) {
  if (!col || n_pow2 == 0 || (n_pow2 & (n_pow2 - 1)) != 0 || n_pow2 > (1ull << 32) || !out || !candidates ||
      !ms || lds_bytes < CE_ROW_WORDS * 4)
    return (int)hipErrorInvalidValue;
  hipStream_t s = (hipStream_t)stream;
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, candidate_ceiling_k, CE_THREADS, lds_bytes);
  if (e != hipSuccess) return (int)e;
  const unsigned grid = (unsigned)std::max(1, cus * std::max(1, per_cu));
  hipEvent_t e0 = nullptr, e1 = nullptr;
  e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  if (e == hipSuccess) {
    candidate_ceiling_k<<<grid, CE_THREADS, lds_bytes, s>>>(col, (uint32_t)(n_pow2 - 1), iters, consecutive, out);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(ms, e0, e1);
  if (e == hipSuccess) *candidates = (unsigned long long)grid * CE_THREADS * iters * CE_UNROLL;
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return (int)e;
}

}  // extern "C"
