// Worst-case-optimal triangle join on gfx950 (see WcojArgs): per driver row
// (x, y) of a, the Z values of b(y) and c(x) are intersected by probing each
// value of the shorter list into the longer one, so a row costs
// min(|b(y)|, |c(x)|) probes instead of the |b(y)| candidates a binary join
// a ⋈ b followed by a lookup in c produces (the generic-join bound of the
// worst-case-optimal join papers the paper cites, Sec. 4 "Worst-case-optimal
// joins").  Work is split into fixed chunks of WC_CHUNK probes per wavefront
// over the prefix sum of the rows' probe counts, so hot rows with long lists
// spread over many wavefronts.  Two passes over the same chunks: count hits
// per chunk, then (after a scan of the counts) write them in order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_util.h"
#include "kernels.h"

namespace xlh {
namespace k {

constexpr int WC_THREADS = 256;
constexpr int WC_WAVES = WC_THREADS / 64;

__device__ __forceinline__ uint32_t seg_len(const IndexProbe& ix, uint32_t v, uint32_t* beg) {
  uint32_t kk;
  if (!index_segment(ix, v, &kk)) {
    *beg = 0;
    return 0;
  }
  *beg = ix.off[kk];
  return ix.off[kk + 1] - *beg;
}

__global__ void wcoj_work_k(WcojArgs a) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.na;
       i += (int64_t)gridDim.x * blockDim.x) {
    uint32_t b0, c0;
    const uint32_t l1 = seg_len(a.ib, a.ay[i], &b0), l2 = seg_len(a.ic, a.ax[i], &c0);
    a.work[i] = l2 == 0 ? 0u : a.probe_shorter ? (l1 < l2 ? l1 : l2) : l1;
  }
}

hipError_t wcoj_work(const WcojArgs& a, hipStream_t s) {
  if (a.na <= 0) return hipSuccess;
  wcoj_work_k<<<grid_for(a.na, 256, 65536), 256, 0, s>>>(a);
  return hipGetLastError();
}

__global__ void nonzero_flags_k(const uint32_t* v, int64_t n, uint32_t* flag) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    flag[i] = v[i] != 0;
}

hipError_t nonzero_flags(const uint32_t* v, int64_t n, uint32_t* flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  nonzero_flags_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(v, n, flag);
  return hipGetLastError();
}

__global__ void wcoj_compact_k(const uint32_t* work, const uint32_t* pos, int64_t n, uint32_t* crow,
                               unsigned long long* cw) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    if (work[i]) {
      crow[pos[i]] = (uint32_t)i;
      cw[pos[i]] = work[i];
    }
}

hipError_t wcoj_compact(const uint32_t* work, const uint32_t* pos, int64_t n, uint32_t* crow,
                        unsigned long long* cw, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  wcoj_compact_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(work, pos, n, crow, cw);
  return hipGetLastError();
}

// One wavefront per chunk of WC_CHUNK items, 64 per step.  Per step the
// wavefront finds the row of its first item by a binary search over cofs;
// the step's items lie in that row and the next 63 (every listed row has at
// least one item), whose starts and list bounds are staged in LDS, and each
// lane finds its row there by a six-step search.
template <bool MAT>
__global__ __launch_bounds__(WC_THREADS) void wcoj_probe_k(WcojArgs a) {
  __shared__ u64 s_start[WC_WAVES][64];
  __shared__ uint32_t s_x[WC_WAVES][64], s_y[WC_WAVES][64];
  __shared__ uint32_t s_sb[WC_WAVES][64], s_sl[WC_WAVES][64], s_lb[WC_WAVES][64], s_ll[WC_WAVES][64];
  __shared__ uint8_t s_sc[WC_WAVES][64];  // 1: the short list is c's
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const u64 nchunks = (a.items + WC_CHUNK - 1) / WC_CHUNK;
  for (u64 g = (u64)blockIdx.x * WC_WAVES + w; g < nchunks; g += (u64)gridDim.x * WC_WAVES) {
    uint32_t hits = 0;  // this chunk's hits so far (wave-uniform)
    const uint32_t base_out = MAT ? a.chunk_off[g] : 0u;
    for (int st = 0; st < WC_CHUNK / 64; ++st) {
      const u64 b = g * WC_CHUNK + (u64)st * 64;
      if (b >= a.items) break;
      // row of item b: the last q with cofs[q] <= b
      int64_t lo = 0, hi = a.nz;
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (a.cofs[mid] <= b) lo = mid;
        else hi = mid;
      }
      const int64_t q = lo + lane;
      if (q < a.nz) {
        const uint32_t i = a.crow[q];
        const uint32_t x = a.ax[i], y = a.ay[i];
        uint32_t b0, c0;
        const uint32_t l1 = seg_len(a.ib, y, &b0), l2 = seg_len(a.ic, x, &c0);
        const bool c_short = a.probe_shorter && l2 < l1;
        s_start[w][lane] = a.cofs[q];
        s_x[w][lane] = x;
        s_y[w][lane] = y;
        s_sc[w][lane] = c_short;
        s_sb[w][lane] = c_short ? c0 : b0;
        s_sl[w][lane] = c_short ? l2 : l1;
        s_lb[w][lane] = c_short ? b0 : c0;
        s_ll[w][lane] = c_short ? l1 : l2;
      } else {
        s_start[w][lane] = ~0ull;
      }
      wave_lds_sync();
      const u64 item = b + (u64)lane;
      bool hit = false;
      uint32_t z = 0;
      int r = 0;
      if (item < a.items) {
#pragma unroll
        for (int step = 32; step > 0; step >>= 1)
          if (s_start[w][r + step] <= item) r += step;
        const uint32_t j = (uint32_t)(item - s_start[w][r]);
        const bool c_short = s_sc[w][r];
        const uint32_t* sh = c_short ? a.cz : a.bz;
        const uint32_t* lg = c_short ? a.bz : a.cz;
        z = sh[s_sb[w][r] + j];
        // binary search of z among the long list's values (ascending int32)
        const uint32_t e0 = s_lb[w][r];
        uint32_t l = 0, h = s_ll[w][r];
        while (l < h) {
          const uint32_t m = (l + h) >> 1;
          if ((int32_t)lg[e0 + m] < (int32_t)z) l = m + 1;
          else h = m;
        }
        hit = l < s_ll[w][r] && lg[e0 + l] == z;
      }
      const u64 hm = __ballot(hit);
      if (MAT && hit) {
        const uint32_t o = base_out + hits + (uint32_t)__popcll(hm & lanemask_lt());
        a.out0[o] = s_x[w][r];
        a.out1[o] = s_y[w][r];
        a.out2[o] = z;
      }
      hits += (uint32_t)__popcll(hm);
      wave_lds_sync();
    }
    if (!MAT && lane == 0) a.chunk_cnt[g] = hits;
  }
}

hipError_t wcoj_probe(const WcojArgs& a, bool materialize, hipStream_t s) {
  if (a.items == 0 || a.nz <= 0) return hipSuccess;
  const u64 nchunks = (a.items + WC_CHUNK - 1) / WC_CHUNK;
  const unsigned grid = (unsigned)std::min<u64>((nchunks + WC_WAVES - 1) / WC_WAVES, 1u << 16);
  if (materialize) wcoj_probe_k<true><<<grid, WC_THREADS, 0, s>>>(a);
  else wcoj_probe_k<false><<<grid, WC_THREADS, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace k
}  // namespace xlh
