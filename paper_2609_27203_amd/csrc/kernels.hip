// HIP kernels for gfx950 (CDNA4, wave64).  Every hot loop here is bound by
// memory traffic or by atomics, never by arithmetic; nothing is a dense
// contraction, so no matrix-core instructions are used.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kernels.h"
#include "device_util.h"

namespace xlh {
namespace k {


// ============================================================ scan
constexpr int SC_THREADS = 256;
constexpr int SC_ITEMS = 16;
constexpr int SC_TILE = SC_THREADS * SC_ITEMS;

template <typename T>
__device__ T block_excl_scan(T x, T* total) {
  __shared__ T s_w[SC_THREADS / 64];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  T incl = wave_incl_scan_t<T>(x);
  if (lane == 63) s_w[w] = incl;
  __syncthreads();
  T pre = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < SC_THREADS / 64; ++i) {
    T y = s_w[i];
    if (i < w) pre += y;
    tot += y;
  }
  __syncthreads();
  *total = tot;
  return pre + incl - x;
}

template <typename T>
__global__ __launch_bounds__(SC_THREADS) void scan_reduce_k(const T* in, int64_t n, T* partial) {
  const int64_t base = (int64_t)blockIdx.x * SC_TILE;
  T acc = 0;
#pragma unroll
  for (int i = 0; i < SC_ITEMS; ++i) {
    int64_t idx = base + (int64_t)i * SC_THREADS + threadIdx.x;
    if (idx < n) acc += in[idx];
  }
  T tot;
  block_excl_scan<T>(acc, &tot);
  if (threadIdx.x == 0) partial[blockIdx.x] = tot;
}

// Each thread owns SC_ITEMS consecutive elements.
template <typename T>
__global__ __launch_bounds__(SC_THREADS) void scan_apply_k(const T* in, T* out, int64_t n,
                                                            const T* partial, T* total) {
  const int64_t base = (int64_t)blockIdx.x * SC_TILE + (int64_t)threadIdx.x * SC_ITEMS;
  T v[SC_ITEMS];
  T acc = 0;
#pragma unroll
  for (int i = 0; i < SC_ITEMS; ++i) {
    int64_t idx = base + i;
    v[i] = idx < n ? in[idx] : (T)0;
    acc += v[i];
  }
  T tot;
  T pre = block_excl_scan<T>(acc, &tot);
  pre += partial ? partial[blockIdx.x] : (T)0;
#pragma unroll
  for (int i = 0; i < SC_ITEMS; ++i) {
    int64_t idx = base + i;
    if (idx < n) out[idx] = pre;
    pre += v[i];
  }
  if (total && blockIdx.x == gridDim.x - 1 && threadIdx.x == SC_THREADS - 1) *total = pre;
}

// Arrays up to SC_ONE_MAX elements are scanned by one workgroup walking its
// tiles in order (one launch instead of three: for a few tens of thousands
// of elements the launches, not the bytes, set the time).
// Each thread owns SC_ONE_ITEMS consecutive elements of each of SC_ONE_SUB
// sub-tiles, so one load instruction of a wavefront covers a contiguous 1 KB
// (u32); a step loads all four sub-tiles at once and ranks them with one
// workgroup scan of four sums per thread.
constexpr int SC_ONE_THREADS = 1024;
constexpr int SC_ONE_ITEMS = 4;
constexpr int SC_ONE_SUB = 4;
constexpr int64_t SC_ONE_MAX = 65536;

template <typename T>
__global__ __launch_bounds__(SC_ONE_THREADS) void scan_one_k(const T* in, T* out, int64_t n, T* total) {
  __shared__ T s_w[SC_ONE_SUB][SC_ONE_THREADS / 64];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  constexpr int64_t SUB = (int64_t)SC_ONE_THREADS * SC_ONE_ITEMS;
  T carry = 0;
  for (int64_t b = 0; b < n; b += SUB * SC_ONE_SUB) {
    T v[SC_ONE_SUB][SC_ONE_ITEMS], acc[SC_ONE_SUB], incl[SC_ONE_SUB];
#pragma unroll
    for (int k = 0; k < SC_ONE_SUB; ++k) {
      const int64_t base = b + k * SUB + (int64_t)threadIdx.x * SC_ONE_ITEMS;
      acc[k] = 0;
#pragma unroll
      for (int i = 0; i < SC_ONE_ITEMS; ++i) {
        v[k][i] = base + i < n ? in[base + i] : (T)0;
        acc[k] += v[k][i];
      }
    }
#pragma unroll
    for (int k = 0; k < SC_ONE_SUB; ++k) {
      incl[k] = wave_incl_scan_t<T>(acc[k]);
      if (lane == 63) s_w[k][w] = incl[k];
    }
    __syncthreads();
    T run = carry;
#pragma unroll
    for (int k = 0; k < SC_ONE_SUB; ++k) {
      T pre = 0, tot = 0;
      for (int j = 0; j < SC_ONE_THREADS / 64; ++j) {
        const T y = s_w[k][j];
        if (j < w) pre += y;
        tot += y;
      }
      T o = run + pre + incl[k] - acc[k];
      const int64_t base = b + k * SUB + (int64_t)threadIdx.x * SC_ONE_ITEMS;
#pragma unroll
      for (int i = 0; i < SC_ONE_ITEMS; ++i) {
        if (base + i < n) out[base + i] = o;
        o += v[k][i];
      }
      run += tot;
    }
    __syncthreads();
    carry = run;
  }
  if (total && threadIdx.x == 0) *total = carry;
}

// Arrays of SC_TILE+1 to SC_WIDE_MAX elements, 16-byte aligned and written
// to a separate array: one launch of one workgroup per tile.  Each workgroup
// sums every element before its tile itself (at most SC_WIDE_MAX elements,
// read with 16-byte loads issued a batch at a time) instead of waiting for
// the tiles before it, so no workgroup depends on another.  Within a tile,
// thread t owns one 16-byte vector of each of four sub-tiles (one load
// instruction of a wavefront covers a contiguous 1 KB) and the four sums per
// thread are ranked by one workgroup scan.
constexpr int SC_W_THREADS = 1024;
constexpr int SC_W_SUB = 4;
constexpr int SC_W_BATCH = 16;
constexpr int64_t SC_WIDE_MAX = 131072;

template <typename T>
struct alignas(16) ScVec {
  T e[16 / sizeof(T)];
};

template <typename T>
__global__ __launch_bounds__(SC_W_THREADS) void scan_wide_k(const T* in, T* out, int64_t n, T* total) {
  constexpr int PER = 16 / sizeof(T);
  constexpr int64_t SUBV = SC_W_THREADS;                  // vectors per sub-tile
  constexpr int64_t TILE = SUBV * SC_W_SUB * PER;         // elements per workgroup
  __shared__ T s_w[SC_W_SUB][SC_W_THREADS / 64];
  __shared__ T s_p[SC_W_THREADS / 64];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const ScVec<T>* inv = (const ScVec<T>*)in;
  ScVec<T>* outv = (ScVec<T>*)out;
  const int64_t v0 = (int64_t)blockIdx.x * (TILE / PER);  // first vector of the tile
  ScVec<T> v[SC_W_SUB];
  T acc[SC_W_SUB];
#pragma unroll
  for (int k = 0; k < SC_W_SUB; ++k) {
    const int64_t vi = v0 + k * SUBV + threadIdx.x;
    const int64_t e0 = vi * PER;
    if (e0 + PER <= n) {
      v[k] = inv[vi];
    } else {
#pragma unroll
      for (int i = 0; i < PER; ++i) v[k].e[i] = e0 + i < n ? in[e0 + i] : (T)0;
    }
    acc[k] = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[k] += v[k].e[i];
  }
  // the elements before the tile: whole vectors, since the tile starts at a
  // multiple of TILE elements
  T pre = 0;
  for (int64_t q0 = threadIdx.x; q0 < v0; q0 += (int64_t)SC_W_THREADS * SC_W_BATCH) {
    ScVec<T> x[SC_W_BATCH];
#pragma unroll
    for (int u = 0; u < SC_W_BATCH; ++u) {
      const int64_t q = q0 + (int64_t)u * SC_W_THREADS;
      if (q < v0) {
        x[u] = inv[q];
      } else {
#pragma unroll
        for (int i = 0; i < PER; ++i) x[u].e[i] = 0;
      }
    }
#pragma unroll
    for (int u = 0; u < SC_W_BATCH; ++u)
#pragma unroll
      for (int i = 0; i < PER; ++i) pre += x[u].e[i];
  }
  T incl[SC_W_SUB];
#pragma unroll
  for (int k = 0; k < SC_W_SUB; ++k) {
    incl[k] = wave_incl_scan_t<T>(acc[k]);
    if (lane == 63) s_w[k][w] = incl[k];
  }
  const T pw = wave_incl_scan_t<T>(pre);
  if (lane == 63) s_p[w] = pw;
  __syncthreads();
  T run = 0;
  for (int j = 0; j < SC_W_THREADS / 64; ++j) run += s_p[j];
#pragma unroll
  for (int k = 0; k < SC_W_SUB; ++k) {
    T before = 0, tot = 0;
    for (int j = 0; j < SC_W_THREADS / 64; ++j) {
      const T y = s_w[k][j];
      if (j < w) before += y;
      tot += y;
    }
    T o = run + before + incl[k] - acc[k];
    const int64_t vi = v0 + k * SUBV + threadIdx.x;
    const int64_t e0 = vi * PER;
    ScVec<T> r;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      r.e[i] = o;
      o += v[k].e[i];
    }
    if (e0 + PER <= n) {
      outv[vi] = r;
    } else {
#pragma unroll
      for (int i = 0; i < PER; ++i)
        if (e0 + i < n) out[e0 + i] = r.e[i];
    }
    run += tot;
  }
  if (total && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *total = run;
}

size_t scan_temp_bytes(int64_t n) {
  size_t bytes = 0;
  int64_t m = n;
  while (m > SC_TILE) {
    m = (m + SC_TILE - 1) / SC_TILE;
    bytes += ((size_t)m * 8 + 255) & ~(size_t)255;
  }
  return bytes + 256;
}

template <typename T>
static hipError_t scan_rec(const T* in, T* out, int64_t n, T* total, char* temp, hipStream_t s) {
  if (n <= 0) {
    if (total) return hipMemsetAsync(total, 0, sizeof(T), s);
    return hipSuccess;
  }
  if (n <= SC_TILE) {
    scan_apply_k<T><<<1, SC_THREADS, 0, s>>>(in, out, n, nullptr, total);
    return hipGetLastError();
  }
  // the one-launch wide form reads elements of other tiles, so it needs a
  // separate output array; both arrays 16-byte aligned for its vector loads
  const uintptr_t ia = (uintptr_t)in, oa = (uintptr_t)out;
  const bool apart = oa >= ia + (uintptr_t)n * sizeof(T) || ia >= oa + (uintptr_t)n * sizeof(T);
  if (n <= SC_WIDE_MAX && apart && ((ia | oa) & 15) == 0) {
    constexpr int64_t tile = (int64_t)SC_W_THREADS * SC_W_SUB * (16 / sizeof(T));
    scan_wide_k<T><<<(unsigned)((n + tile - 1) / tile), SC_W_THREADS, 0, s>>>(in, out, n, total);
    return hipGetLastError();
  }
  if (n <= SC_ONE_MAX) {
    scan_one_k<T><<<1, SC_ONE_THREADS, 0, s>>>(in, out, n, total);
    return hipGetLastError();
  }
  int64_t nb = (n + SC_TILE - 1) / SC_TILE;
  T* partial = (T*)temp;
  char* next = temp + (((size_t)nb * 8 + 255) & ~(size_t)255);
  scan_reduce_k<T><<<(unsigned)nb, SC_THREADS, 0, s>>>(in, n, partial);
  hipError_t e = scan_rec<T>(partial, partial, nb, nullptr, next, s);
  if (e != hipSuccess) return e;
  scan_apply_k<T><<<(unsigned)nb, SC_THREADS, 0, s>>>(in, out, n, partial, total);
  return hipGetLastError();
}

hipError_t scan_exclusive_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total,
                              void* temp, hipStream_t s) {
  return scan_rec<uint32_t>(in, out, n, total, (char*)temp, s);
}
hipError_t scan_exclusive_u64(const u64* in, u64* out, int64_t n, u64* total, void* temp,
                              hipStream_t s) {
  return scan_rec<u64>(in, out, n, total, (char*)temp, s);
}

// ============================================================ radix sort
// LSD radix sort with 8-bit digits.  Per pass: a per-tile digit histogram
// (LDS atomics; the tile's counts are also added to the pass's 256 digit
// totals), the digit-major offsets (one workgroup per digit scans that
// digit's row of tile counts and adds the keys of all smaller digits), and a
// stable scatter.  In the scatter each wavefront ranks its keys with a
// ballot-based match of equal digits and running per-wave digit counters in
// LDS, so the pass is stable without a block-wide sort.
// Tiles of RS_THREADS * ITEMS keys: 16 items per thread for large inputs,
// 4 for small ones so that a few hundred thousand keys still spread over
// every CU.
constexpr int RS_THREADS = 256;
constexpr int RS_WAVES = RS_THREADS / 64;
constexpr int RS_SMALL_ITEMS = 4;
constexpr int64_t RS_SMALL_N = (int64_t)1 << 22;  // below this, small tiles

template <typename K, int RS_ITEMS>
__global__ __launch_bounds__(RS_THREADS) void rs_hist_k(const K* keys, int64_t n, int shift,
                                                         uint32_t dmask, uint32_t* hist,
                                                         uint32_t nblocks, uint32_t* totals) {
  constexpr int RS_TILE = RS_THREADS * RS_ITEMS;
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * RS_TILE;
#pragma unroll
  for (int i = 0; i < RS_ITEMS; ++i) {
    int64_t idx = base + (int64_t)i * RS_THREADS + threadIdx.x;
    if (idx < n) atomicAdd(&h[(uint32_t)(keys[idx] >> shift) & dmask], 1u);
  }
  __syncthreads();
  const uint32_t c = h[threadIdx.x];
  hist[(size_t)threadIdx.x * nblocks + blockIdx.x] = c;
  if (c) atomicAdd(&totals[threadIdx.x], c);
}

// Workgroup d: row d of the histogram table (digit d's count in each tile)
// becomes digit d's output offset in each tile: the number of keys with a
// smaller digit plus digit d's count in the earlier tiles.  Workgroup 0 also
// clears the digit totals of the next pass.
__global__ __launch_bounds__(RS_THREADS) void rs_offsets_k(uint32_t* hist, uint32_t nblocks,
                                                           const uint32_t* totals, uint32_t* next_totals) {
  __shared__ uint32_t s_w[RS_THREADS / 64];
  __shared__ uint32_t s_base;
  const uint32_t d = blockIdx.x;
  uint32_t t;
  const uint32_t below = block_excl_scan_u32(totals[threadIdx.x], &t, s_w);
  if (threadIdx.x == d) s_base = below;
  __syncthreads();
  uint32_t carry = s_base;
  uint32_t* row = hist + (size_t)d * nblocks;
  for (uint32_t b0 = 0; b0 < nblocks; b0 += RS_THREADS) {
    const uint32_t b = b0 + threadIdx.x;
    const uint32_t v = b < nblocks ? row[b] : 0u;
    const uint32_t p = block_excl_scan_u32(v, &t, s_w);
    if (b < nblocks) row[b] = carry + p;
    carry += t;
  }
  if (d == 0) next_totals[threadIdx.x] = 0u;
}

template <typename K, int RS_ITEMS>
__global__ __launch_bounds__(RS_THREADS) void rs_scatter_k(const K* kin, const uint32_t* vin,
                                                            K* kout, uint32_t* vout, int64_t n,
                                                            int shift, int nbits,
                                                            const uint32_t* off,
                                                            uint32_t nblocks) {
  constexpr int RS_TILE = RS_THREADS * RS_ITEMS;
  __shared__ uint32_t cnt[RS_WAVES][256];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < RS_WAVES * 256; i += RS_THREADS) (&cnt[0][0])[i] = 0;
  __syncthreads();
  const uint32_t dmask = (1u << nbits) - 1u;
  const int64_t sub = (int64_t)blockIdx.x * RS_TILE + (int64_t)w * 64 * RS_ITEMS;
  K key[RS_ITEMS];
  uint32_t val[RS_ITEMS], rank[RS_ITEMS], dig[RS_ITEMS];
#pragma unroll
  for (int i = 0; i < RS_ITEMS; ++i) {
    const int64_t idx = sub + (int64_t)i * 64 + lane;
    const bool valid = idx < n;
    key[i] = valid ? kin[idx] : (K)0;
    val[i] = (valid && vin) ? vin[idx] : 0u;
    const uint32_t d = (uint32_t)(key[i] >> shift) & dmask;
    u64 peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (d >> b) & 1u;
      const u64 bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    if (!valid) peers = 0;
    const uint32_t lt = __popcll(peers & lanemask_lt());
    const uint32_t before = cnt[w][d];
    wave_lds_sync();
    rank[i] = before + lt;
    dig[i] = valid ? d : 0xffffffffu;
    if (valid && lt == 0) cnt[w][d] = before + (uint32_t)__popcll(peers);
    wave_lds_sync();
  }
  __syncthreads();
  // the tile's keys in output order in LDS (digit, then wave, then rank), so
  // each digit's run goes out as consecutive stores
  __shared__ K sk[RS_TILE];
  __shared__ uint32_t sv[RS_TILE];
  __shared__ uint32_t toff[256], s_w[RS_WAVES];
  {
    uint32_t t = 0;
    for (int ww = 0; ww < RS_WAVES; ++ww) t += cnt[ww][threadIdx.x];
    uint32_t tot;
    toff[threadIdx.x] = block_excl_scan_u32(t, &tot, s_w);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < RS_ITEMS; ++i) {
    const uint32_t d = dig[i];
    if (d == 0xffffffffu) continue;
    uint32_t pre = 0;
    for (int ww = 0; ww < w; ++ww) pre += cnt[ww][d];
    const uint32_t lp = toff[d] + pre + rank[i];
    sk[lp] = key[i];
    sv[lp] = val[i];
  }
  __syncthreads();
  const int64_t t0 = (int64_t)blockIdx.x * RS_TILE;
  const uint32_t tile_n = (uint32_t)min((int64_t)RS_TILE, n - t0);
  for (uint32_t q = threadIdx.x; q < tile_n; q += RS_THREADS) {
    const K k = sk[q];
    const uint32_t d = (uint32_t)(k >> shift) & dmask;
    const uint32_t pos = off[(size_t)d * nblocks + blockIdx.x] + (q - toff[d]);
    kout[pos] = k;
    if (vout) vout[pos] = sv[q];
  }
}

// Inputs of at most SS_MAX keys are sorted by one workgroup in LDS: every
// 8-bit pass of the same stable LSD order runs in one launch instead of
// three launches per pass.  Wavefront w owns positions [256w, 256w + 256),
// four 64-key runs; a pass ranks each key among the equal digits of its
// wavefront with the ballot match used by the scatter above, offsets each
// (digit, wavefront) count in digit-major order, and scatters the keys to
// their new positions in LDS.  The result is written back in place.
constexpr int SS_THREADS = 1024;
constexpr int SS_WAVES = SS_THREADS / 64;
constexpr int SS_ITEMS = 4;
constexpr int64_t SS_MAX = (int64_t)SS_THREADS * SS_ITEMS;

template <typename K>
__global__ __launch_bounds__(SS_THREADS) void sort_small_k(K* keys, uint32_t* vals, int n, int bits) {
  __shared__ K sk[SS_MAX];
  __shared__ uint32_t sv[SS_MAX];
  __shared__ uint32_t cnt[SS_WAVES][256];
  __shared__ uint32_t s_w[SS_WAVES];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  K key[SS_ITEMS];
  uint32_t val[SS_ITEMS];
#pragma unroll
  for (int j = 0; j < SS_ITEMS; ++j) {
    const int p = w * 64 * SS_ITEMS + j * 64 + lane;
    key[j] = p < n ? keys[p] : (K)0;
    val[j] = (p < n && vals) ? vals[p] : 0u;
  }
  for (int shift = 0; shift < bits; shift += 8) {
    const int nbits = bits - shift < 8 ? bits - shift : 8;
    const uint32_t dmask = (1u << nbits) - 1u;
    for (int i = threadIdx.x; i < SS_WAVES * 256; i += SS_THREADS) (&cnt[0][0])[i] = 0;
    __syncthreads();
    uint32_t rank[SS_ITEMS], dig[SS_ITEMS];
#pragma unroll
    for (int j = 0; j < SS_ITEMS; ++j) {
      const bool valid = w * 64 * SS_ITEMS + j * 64 + lane < n;
      const uint32_t d = (uint32_t)(key[j] >> shift) & dmask;
      u64 peers = __ballot(valid);
      for (int b = 0; b < nbits; ++b) {
        const bool bit = (d >> b) & 1u;
        const u64 bal = __ballot(bit);
        peers &= bit ? bal : ~bal;
      }
      if (!valid) peers = 0;
      const uint32_t lt = __popcll(peers & lanemask_lt());
      const uint32_t before = cnt[w][d];
      wave_lds_sync();
      rank[j] = before + lt;
      dig[j] = d;
      if (valid && lt == 0) cnt[w][d] = before + (uint32_t)__popcll(peers);
      wave_lds_sync();
    }
    __syncthreads();
    // digit d's total, then the digit-major offsets of every (digit, wavefront)
    uint32_t tot = 0;
    if (threadIdx.x < 256)
      for (int ww = 0; ww < SS_WAVES; ++ww) tot += cnt[ww][threadIdx.x];
    const uint32_t incl = wave_incl_scan_t<uint32_t>(tot);
    if (lane == 63) s_w[w] = incl;
    __syncthreads();
    uint32_t run = incl - tot;
    for (int ww = 0; ww < w; ++ww) run += s_w[ww];
    if (threadIdx.x < 256)
      for (int ww = 0; ww < SS_WAVES; ++ww) {
        const uint32_t c = cnt[ww][threadIdx.x];
        cnt[ww][threadIdx.x] = run;
        run += c;
      }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SS_ITEMS; ++j) {
      if (w * 64 * SS_ITEMS + j * 64 + lane < n) {
        const uint32_t pos = cnt[w][dig[j]] + rank[j];
        sk[pos] = key[j];
        sv[pos] = val[j];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SS_ITEMS; ++j) {
      const int p = w * 64 * SS_ITEMS + j * 64 + lane;
      if (p < n) {
        key[j] = sk[p];
        val[j] = sv[p];
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < SS_ITEMS; ++j) {
    const int p = w * 64 * SS_ITEMS + j * 64 + lane;
    if (p < n) {
      keys[p] = key[j];
      if (vals) vals[p] = val[j];
    }
  }
}

static int64_t rs_tile(int64_t n) { return (int64_t)RS_THREADS * (n < RS_SMALL_N ? RS_SMALL_ITEMS : 16); }

size_t radix_temp_bytes(int64_t n) {
  int64_t nb = (n + rs_tile(n) - 1) / rs_tile(n);
  if (nb < 1) nb = 1;
  size_t hist = (((size_t)nb * 256 * 4) + 255) & ~(size_t)255;
  return hist + 2 * 256 * 4;  // + the digit totals of two consecutive passes
}

template <typename K>
static hipError_t radix_sort_t(K* keys, uint32_t* vals, K* keys_alt, uint32_t* vals_alt,
                               int64_t n, int bits, void* temp, hipStream_t s, int* in_alt) {
  *in_alt = 0;
  if (n <= 1 || bits <= 0) return hipSuccess;
  if (n <= SS_MAX) {
    sort_small_k<K><<<1, SS_THREADS, 0, s>>>(keys, vals, (int)n, bits);
    return hipGetLastError();
  }
  const bool small = n < RS_SMALL_N;
  const uint32_t nb = (uint32_t)((n + rs_tile(n) - 1) / rs_tile(n));
  uint32_t* hist = (uint32_t*)temp;
  uint32_t* totals = (uint32_t*)((char*)temp + ((((size_t)nb * 256 * 4) + 255) & ~(size_t)255));
  hipError_t e = hipMemsetAsync(totals, 0, 256 * 4, s);
  if (e != hipSuccess) return e;
  int pass = 0;
  K* ka = keys;
  K* kb = keys_alt;
  uint32_t* va = vals;
  uint32_t* vb = vals ? vals_alt : nullptr;
  for (int shift = 0; shift < bits; shift += 8, ++pass) {
    const int nbits = bits - shift < 8 ? bits - shift : 8;
    uint32_t* tot = totals + 256 * (pass & 1);
    uint32_t* tot_next = totals + 256 * ((pass + 1) & 1);
    if (small)
      rs_hist_k<K, RS_SMALL_ITEMS><<<nb, RS_THREADS, 0, s>>>(ka, n, shift, (1u << nbits) - 1u, hist, nb, tot);
    else
      rs_hist_k<K, 16><<<nb, RS_THREADS, 0, s>>>(ka, n, shift, (1u << nbits) - 1u, hist, nb, tot);
    rs_offsets_k<<<256, RS_THREADS, 0, s>>>(hist, nb, tot, tot_next);
    if (small)
      rs_scatter_k<K, RS_SMALL_ITEMS><<<nb, RS_THREADS, 0, s>>>(ka, va, kb, vb, n, shift, nbits, hist, nb);
    else
      rs_scatter_k<K, 16><<<nb, RS_THREADS, 0, s>>>(ka, va, kb, vb, n, shift, nbits, hist, nb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    K* tk = ka; ka = kb; kb = tk;
    uint32_t* tv = va; va = vb; vb = tv;
    *in_alt ^= 1;
  }
  return hipSuccess;
}

hipError_t radix_sort_u32(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt,
                          int64_t n, int bits, void* temp, hipStream_t s, int* in_alt) {
  return radix_sort_t<uint32_t>(keys, vals, keys_alt, vals_alt, n, bits, temp, s, in_alt);
}
hipError_t radix_sort_u64(u64* keys, uint32_t* vals, u64* keys_alt, uint32_t* vals_alt, int64_t n,
                          int bits, void* temp, hipStream_t s, int* in_alt) {
  return radix_sort_t<u64>(keys, vals, keys_alt, vals_alt, n, bits, temp, s, in_alt);
}

// ============================================================ small helpers
__global__ void iota_k(uint32_t* out, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = (uint32_t)i;
}
hipError_t iota_u32(uint32_t* out, int64_t n, hipStream_t s) {
  iota_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(out, n);
  return hipGetLastError();
}

__global__ void gather_k(const uint32_t* src, const uint32_t* perm, uint32_t* dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[perm[i]];
}
hipError_t gather_u32(const uint32_t* src, const uint32_t* perm, uint32_t* dst, int64_t n,
                      hipStream_t s) {
  gather_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(src, perm, dst, n);
  return hipGetLastError();
}

// Byte fill with 16-byte stores (large clears of bitmaps and value arrays):
// n16 aligned quads, then the ntail bytes after them.
__global__ void fill_k(uint4* p, int64_t n16, uint32_t v, uint8_t* tail, int ntail) {
  const uint4 q = make_uint4(v, v, v, v);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = q;
  if (blockIdx.x == 0 && (int)threadIdx.x < ntail) tail[threadIdx.x] = (uint8_t)v;
}
hipError_t fill_bytes(void* p, int byte, size_t bytes, hipStream_t s) {
  if (bytes < ((size_t)1 << 20) || ((uintptr_t)p & 15u)) return hipMemsetAsync(p, byte, bytes, s);
  const int64_t n16 = (int64_t)(bytes / 16);
  const uint32_t v = (uint32_t)(byte & 0xff) * 0x01010101u;
  fill_k<<<grid_for(n16, 256, 8192), 256, 0, s>>>((uint4*)p, n16, v, (uint8_t*)p + n16 * 16, (int)(bytes % 16));
  return hipGetLastError();
}

struct ColPtrsIn { const uint32_t* c[MAXC]; };
struct ColPtrsOut { uint32_t* c[MAXC]; };

// dst.c[j][i] = src.c[j][perm[i]] for every column j < ncols, one launch.
__global__ void gather_cols_k(ColPtrsIn src, ColPtrsOut dst, int ncols, const uint32_t* perm, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t p = perm[i];
    for (int j = 0; j < ncols; ++j) dst.c[j][i] = src.c[j][p];
  }
}
hipError_t gather_cols(const uint32_t* const* src, uint32_t* const* dst, int ncols, const uint32_t* perm, int64_t n,
                       hipStream_t s) {
  if (n <= 0 || ncols <= 0) return hipSuccess;
  if (ncols > MAXC) return hipErrorInvalidValue;
  ColPtrsIn a{};
  ColPtrsOut b{};
  for (int j = 0; j < ncols; ++j) {
    a.c[j] = src[j];
    b.c[j] = dst[j];
  }
  gather_cols_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(a, b, ncols, perm, n);
  return hipGetLastError();
}

// key[i] = col[i] - lo (unsigned) and perm[i] = i, one launch.
__global__ void keys_perm_k(const uint32_t* col, int32_t lo, int64_t n, uint32_t* key, uint32_t* perm) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    key[i] = col[i] - (uint32_t)lo;
    perm[i] = (uint32_t)i;
  }
}
hipError_t keys_perm(const uint32_t* col, int32_t lo, int64_t n, uint32_t* key, uint32_t* perm, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  keys_perm_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(col, lo, n, key, perm);
  return hipGetLastError();
}

__device__ __forceinline__ uint32_t order_bits(uint32_t x, int type) {
  if (type == T_F32) return x ^ ((x >> 31) ? 0xffffffffu : 0x80000000u);  // totalOrder
  return x ^ 0x80000000u;                                                  // signed int
}

__global__ void ordered_key_k(const uint32_t* col, int type, const uint32_t* perm,
                              uint32_t* out, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = order_bits(col[perm ? perm[i] : i], type);
}
hipError_t ordered_key(const uint32_t* col, int type, const uint32_t* perm, uint32_t* out,
                       int64_t n, hipStream_t s) {
  ordered_key_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(col, type, perm, out, n);
  return hipGetLastError();
}

__global__ void minmax_k(const int32_t* col, int64_t n, int32_t* out) {
  int32_t lo = INT32_MAX, hi = INT32_MIN;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    lo = min(lo, col[i]);
    hi = max(hi, col[i]);
  }
  for (int d = 32; d > 0; d >>= 1) {
    lo = min(lo, __shfl_xor(lo, d, 64));
    hi = max(hi, __shfl_xor(hi, d, 64));
  }
  // one atomic pair per workgroup: same-address atomics serialize
  __shared__ int32_t s_lo[4], s_hi[4];
  if (lane_id() == 0) {
    s_lo[threadIdx.x >> 6] = lo;
    s_hi[threadIdx.x >> 6] = hi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) {
      lo = min(lo, s_lo[w]);
      hi = max(hi, s_hi[w]);
    }
    atomicMin(&out[0], lo);
    atomicMax(&out[1], hi);
  }
}
hipError_t minmax_i32(const int32_t* col, int64_t n, int32_t* out, hipStream_t s) {
  minmax_k<<<grid_for(n, 256, 2048), 256, 0, s>>>(col, n, out);
  return hipGetLastError();
}

// out = {min, max} of col[0, m), m = *count (at most cap) or cap when count
// is null; {INT32_MAX, INT32_MIN} for no rows.  One workgroup, no
// initialized output: for short columns (a few tens of thousands of rows).
__global__ __launch_bounds__(1024) void bounds_one_k(const int32_t* col, const uint32_t* count, int64_t cap,
                                                     int32_t* out) {
  const int64_t m = count ? min((int64_t)*count, cap) : cap;
  int32_t lo = INT32_MAX, hi = INT32_MIN;
  for (int64_t i = threadIdx.x; i < m; i += 1024) {
    lo = min(lo, col[i]);
    hi = max(hi, col[i]);
  }
  for (int d = 32; d > 0; d >>= 1) {
    lo = min(lo, __shfl_xor(lo, d, 64));
    hi = max(hi, __shfl_xor(hi, d, 64));
  }
  __shared__ int32_t s_lo[16], s_hi[16];
  if (lane_id() == 0) {
    s_lo[threadIdx.x >> 6] = lo;
    s_hi[threadIdx.x >> 6] = hi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < 16; ++k) {
      lo = min(lo, s_lo[k]);
      hi = max(hi, s_hi[k]);
    }
    out[0] = lo;
    out[1] = hi;
  }
}
hipError_t bounds_one(const int32_t* col, const uint32_t* count, int64_t cap, int32_t* out, hipStream_t s) {
  bounds_one_k<<<1, 1024, 0, s>>>(col, count, cap, out);
  return hipGetLastError();
}

__global__ void sub_lo_k(const uint32_t* col, int32_t lo, uint32_t* out, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = col[i] - (uint32_t)lo;
}
hipError_t sub_lo(const uint32_t* col, int32_t lo, uint32_t* out, int64_t n, hipStream_t s) {
  sub_lo_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(col, lo, out, n);
  return hipGetLastError();
}

template <typename K>
__global__ void csr_offsets_k(const K* sorted, int shift, int64_t n, uint32_t range, uint32_t* off) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k <= (int64_t)range;
       k += (int64_t)gridDim.x * blockDim.x) {
    int64_t lo = 0, hi = n;  // first i with sorted[i] >> shift >= k
    while (lo < hi) {
      int64_t mid = (lo + hi) >> 1;
      if ((int64_t)(sorted[mid] >> shift) < k) lo = mid + 1; else hi = mid;
    }
    off[k] = (uint32_t)lo;
  }
}
hipError_t csr_offsets(const uint32_t* sorted, int64_t n, uint32_t range, uint32_t* off,
                       hipStream_t s) {
  csr_offsets_k<uint32_t><<<grid_for((int64_t)range + 1, 256, 65536), 256, 0, s>>>(sorted, 0, n, range, off);
  return hipGetLastError();
}
hipError_t csr_offsets_high(const void* sorted, bool wide, int shift, int64_t n, uint32_t range, uint32_t* off,
                            hipStream_t s) {
  if (wide)
    csr_offsets_k<u64><<<grid_for((int64_t)range + 1, 256, 65536), 256, 0, s>>>((const u64*)sorted, shift, n, range,
                                                                                 off);
  else
    csr_offsets_k<uint32_t><<<grid_for((int64_t)range + 1, 256, 65536), 256, 0, s>>>((const uint32_t*)sorted, shift,
                                                                                      n, range, off);
  return hipGetLastError();
}

// Compacted offsets: row i starts a segment when flag[i] (its key differs
// from row i - 1's); the segment's number is pos[i] (the exclusive scan of
// the flags), its key sorted[i] and its first row i; the last row closes the
// array with off[number of segments] = n.
__global__ void segment_keys_k(const uint32_t* sorted, const uint32_t* flag, const uint32_t* pos, int64_t n,
                               uint32_t* keys, uint32_t* off) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t f = flag[i], p = pos[i];
    if (f) {
      keys[p] = sorted[i];
      off[p] = (uint32_t)i;
    }
    if (i == n - 1) off[p + f] = (uint32_t)n;
  }
}
size_t compact_offsets_temp_bytes(int64_t n) { return ((size_t)n * 8 + 255) / 256 * 256 + scan_temp_bytes(n); }
hipError_t compact_offsets(const uint32_t* sorted, int64_t n, uint32_t* keys, uint32_t* off, uint32_t* count,
                           void* temp, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  uint32_t* flag = (uint32_t*)temp;
  uint32_t* pos = flag + n;
  void* scan_tmp = (char*)temp + ((size_t)n * 8 + 255) / 256 * 256;
  const uint32_t* cols[1] = {sorted};
  hipError_t e = row_change_flags(cols, 1, n, flag, s);
  if (e != hipSuccess) return e;
  e = scan_exclusive_u32(flag, pos, n, count, scan_tmp, s);
  if (e != hipSuccess) return e;
  segment_keys_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(sorted, flag, pos, n, keys, off);
  return hipGetLastError();
}

// Composite sort key of row i of an ordered index and perm[i] = i, one
// launch: the key column's image kcol[i] - klo in the high bits, below it
// (obits bits) the order part -- degree order: 3 - min(3, bitlen(deg(z)) / 3)
// with z = ocol[i] and deg(z) = doff[z - olo + 1] - doff[z - olo] (0 outside
// [olo, olo + drange)), so the rows whose z has the most rows come first, by
// base-8 class (2 bits: at least 256 rows, 32 to 255, 4 to 31, fewer; rows
// of one class keep their order); value
// order: ocol[i] - olo.  Sorting by it keeps the key order.
template <typename K>
__global__ void order_keys_k(const uint32_t* kcol, int32_t klo, const uint32_t* ocol, int32_t olo, int obits,
                             const uint32_t* doff, uint32_t drange, int64_t n, K* key, uint32_t* perm) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t o = ocol[i] - (uint32_t)olo;
    uint32_t part = o;
    if (doff) {
      const uint32_t deg = o < drange ? doff[o + 1] - doff[o] : 0u;
      part = 3u - min(3u, (deg ? 32u - (uint32_t)__clz(deg) : 0u) / 3u);
    }
    key[i] = ((K)(kcol[i] - (uint32_t)klo) << obits) | (K)part;
    perm[i] = (uint32_t)i;
  }
}
hipError_t order_keys(const uint32_t* kcol, int32_t klo, const uint32_t* ocol, int32_t olo, int obits,
                      const uint32_t* doff, uint32_t drange, int64_t n, void* key, bool wide, uint32_t* perm,
                      hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (wide)
    order_keys_k<u64><<<grid_for(n, 256, 65536), 256, 0, s>>>(kcol, klo, ocol, olo, obits, doff, drange, n, (u64*)key,
                                                              perm);
  else
    order_keys_k<uint32_t><<<grid_for(n, 256, 65536), 256, 0, s>>>(kcol, klo, ocol, olo, obits, doff, drange, n,
                                                                   (uint32_t*)key, perm);
  return hipGetLastError();
}

// out[k] = col[off[k]] (the first row of key k's segment), or 0xffffffff
// for an empty segment.
__global__ void segment_first_k(const uint32_t* off, const uint32_t* col, uint32_t range, uint32_t* out) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < (int64_t)range;
       k += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t b = off[k];
    out[k] = b < off[k + 1] ? col[b] : 0xffffffffu;
  }
}
hipError_t segment_first(const uint32_t* off, const uint32_t* col, uint32_t range, uint32_t* out, hipStream_t s) {
  if (range == 0) return hipSuccess;
  segment_first_k<<<grid_for(range, 256, 65536), 256, 0, s>>>(off, col, range, out);
  return hipGetLastError();
}

// key[i] = c0[i] (c1 null) or (c0[i] << 32) | c1[i], as unsigned.
__global__ void neg_keys_k(const uint32_t* c0, const uint32_t* c1, int64_t n, u64* key) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    key[i] = c1 ? ((u64)c0[i] << 32) | c1[i] : (u64)c0[i];
}
hipError_t neg_keys(const uint32_t* c0, const uint32_t* c1, int64_t n, u64* key, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  neg_keys_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(c0, c1, n, key);
  return hipGetLastError();
}

// out[i] = key[i] >> shift
template <typename K>
__global__ void high_bits_k(const K* key, int shift, int64_t n, uint32_t* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = (uint32_t)(key[i] >> shift);
}
hipError_t high_bits(const void* key, bool wide, int shift, int64_t n, uint32_t* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (wide)
    high_bits_k<u64><<<grid_for(n, 256, 65536), 256, 0, s>>>((const u64*)key, shift, n, out);
  else
    high_bits_k<uint32_t><<<grid_for(n, 256, 65536), 256, 0, s>>>((const uint32_t*)key, shift, n, out);
  return hipGetLastError();
}

struct ColPtrs { const uint32_t* c[MAXC]; };

__global__ void row_change_k(ColPtrs cols, int ncols, int64_t n, uint32_t* flag) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    uint32_t f = (i == 0);
    if (i > 0)
      for (int c = 0; c < ncols; ++c) f |= cols.c[c][i] != cols.c[c][i - 1];
    flag[i] = f;
  }
}
hipError_t row_change_flags(const uint32_t* const* cols, int ncols, int64_t n, uint32_t* flag,
                            hipStream_t s) {
  ColPtrs p{};
  for (int c = 0; c < ncols; ++c) p.c[c] = cols[c];
  row_change_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(p, ncols, n, flag);
  return hipGetLastError();
}

__global__ void compact_k(const uint32_t* src, const uint32_t* flag, const uint32_t* pos,
                          uint32_t* dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    if (flag[i]) dst[pos[i]] = src[i];
}
hipError_t compact_u32(const uint32_t* src, const uint32_t* flag, const uint32_t* pos,
                       uint32_t* dst, int64_t n, hipStream_t s) {
  compact_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(src, flag, pos, dst, n);
  return hipGetLastError();
}

// ============================================================ hash tables
// Open addressing over a power-of-two array with linear probing, so a probe
// sequence walks consecutive 8- or 16-byte slots of the same 128-byte line.
// A slot only ever changes from EMPTY to a key, so a plain (possibly stale)
// read is a safe filter: a stale EMPTY is resolved by the compare-and-swap.
__device__ __forceinline__ int set_insert(u64* table, u64 mask, u64 key, u64* counters) {
  u64 i = mix64(key) & mask;
  for (u64 probe = 0; probe <= mask; ++probe) {
    const u64 cur = table[i];
    if (cur == key) return 0;
    if (cur == EMPTY_KEY) {
      const u64 prev = atomicCAS(&table[i], EMPTY_KEY, key);
      if (prev == EMPTY_KEY) return 1;
      if (prev == key) return 0;
    }
    i = (i + 1) & mask;
  }
  atomicOr(&counters[CNT_FATAL], 1ull);
  return 0;
}

// Returns the slot index of key (inserting it if absent); *ins = newly inserted.
__device__ __forceinline__ u64 slot_find_or_insert(Slot16* t, u64 mask, u64 key, bool* ins,
                                                   u64* counters) {
  u64 i = mix64(key) & mask;
  *ins = false;
  for (u64 probe = 0; probe <= mask; ++probe) {
    const u64 cur = t[i].key;
    if (cur == key) return i;
    if (cur == EMPTY_KEY) {
      const u64 prev = atomicCAS(&t[i].key, EMPTY_KEY, key);
      if (prev == EMPTY_KEY) {
        *ins = true;
        return i;
      }
      if (prev == key) return i;
    }
    i = (i + 1) & mask;
  }
  atomicOr(&counters[CNT_FATAL], 1ull);
  return ~0ull;
}

template <typename KP>
__device__ __forceinline__ u64 pack_key(KP& kp, uint32_t a, uint32_t b) {
  u64 k = (uint32_t)(a - (uint32_t)kp.lo[0]);
  if (kp.nkey == 2) k = (k << kp.shift) | (uint32_t)(b - (uint32_t)kp.lo[1]);
  return k;
}
__device__ __forceinline__ void unpack_key(const KeyPack& kp, u64 key, uint32_t* a, uint32_t* b) {
  if (kp.nkey == 2) {
    *a = (uint32_t)(key >> kp.shift) + (uint32_t)kp.lo[0];
    *b = (uint32_t)(key & ((1ull << kp.shift) - 1ull)) + (uint32_t)kp.lo[1];
  } else {
    *a = (uint32_t)key + (uint32_t)kp.lo[0];
    *b = 0;
  }
}

// Min/max are kept as an order-preserving unsigned image so a single
// atomicMin implements both (max stores the complement).
__device__ __forceinline__ uint32_t fold_encode(uint32_t x, int type, int is_max) {
  const uint32_t o = order_bits(x, type);
  return is_max ? ~o : o;
}
__device__ __forceinline__ uint32_t fold_decode(uint32_t e, int type, int is_max) {
  const uint32_t o = is_max ? ~e : e;
  if (type == T_F32) return (o & 0x80000000u) ? (o ^ 0x80000000u) : ~o;
  return o ^ 0x80000000u;
}

// One atomic per workgroup for a per-thread count (every thread must call).
__device__ __forceinline__ void block_count_add(u64* counter, uint32_t mine) {
  __shared__ uint32_t s_bc[4];
  uint32_t v = mine;
  for (int d = 32; d > 0; d >>= 1) v += __shfl_xor(v, d, 64);
  if (lane_id() == 0) s_bc[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += s_bc[i];
    if (t) atomicAdd(counter, (u64)t);
  }
}

__global__ void set_insert_rows_k(u64* table, u64 mask, const uint32_t* c0, const uint32_t* c1,
                                  int64_t n, KeyPack kp, u64* counters) {
  uint32_t mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    mine += set_insert(table, mask, pack_key(kp, c0[i], c1 ? c1[i] : 0u), counters);
  block_count_add(&counters[CNT_INSERTED], mine);
}
hipError_t set_insert_rows(u64* table, u64 mask, const uint32_t* c0, const uint32_t* c1, int64_t n,
                           KeyPack kp, unsigned long long* counters, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  set_insert_rows_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(table, mask, c0, c1, n, kp, counters);
  return hipGetLastError();
}

__global__ void table16_insert_rows_k(Slot16* t, u64 mask, const uint32_t* c0, const uint32_t* c1,
                                      const uint32_t* v, int64_t n, KeyPack kp, int type,
                                      int is_max, u64* counters) {
  uint32_t mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    bool ins;
    const u64 s = slot_find_or_insert(t, mask, pack_key(kp, c0[i], c1 ? c1[i] : 0u), &ins,
                                      counters);
    if (s != ~0ull) atomicMin(&t[s].val, fold_encode(v[i], type, is_max));
    mine += ins;
  }
  block_count_add(&counters[CNT_INSERTED], mine);
}
hipError_t table16_insert_rows(Slot16* t, u64 mask, const uint32_t* c0, const uint32_t* c1,
                               const uint32_t* v, int64_t n, KeyPack kp, int type, int is_max,
                               unsigned long long* counters, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  table16_insert_rows_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(t, mask, c0, c1, v, n, kp, type,
                                                               is_max, counters);
  return hipGetLastError();
}

__global__ void table16_rehash_k(const Slot16* old, int64_t old_cap, Slot16* nt, u64 mask,
                                 u64* counters) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < old_cap;
       i += (int64_t)gridDim.x * blockDim.x) {
    const Slot16 s = old[i];
    if (s.key == EMPTY_KEY) continue;
    bool ins;
    const u64 j = slot_find_or_insert(nt, mask, s.key, &ins, counters);
    if (j != ~0ull) {
      nt[j].val = s.val;
      nt[j].stamp = s.stamp;
    }
  }
}
hipError_t table16_rehash(const Slot16* old, int64_t old_cap, Slot16* nt, u64 mask,
                          unsigned long long* counters, hipStream_t s) {
  table16_rehash_k<<<grid_for(old_cap, 256, 8192), 256, 0, s>>>(old, old_cap, nt, mask, counters);
  return hipGetLastError();
}

__device__ __forceinline__ uint32_t stored_value(uint32_t e, int type, int fold_kind) {
  if (fold_kind == FOLD_MIN) return fold_decode(e, type, 0);
  if (fold_kind == FOLD_MAX) return fold_decode(e, type, 1);
  return e;
}

__global__ void table16_rows_from_idx_k(const Slot16* t, const uint32_t* idx, int64_t n,
                                        KeyPack kp, int type, int fold_kind, uint32_t* k0,
                                        uint32_t* k1, uint32_t* v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const Slot16 s = t[idx[i]];
    uint32_t a, b;
    unpack_key(kp, s.key, &a, &b);
    k0[i] = a;
    if (k1) k1[i] = b;
    v[i] = stored_value(s.val, type, fold_kind);
  }
}
hipError_t table16_rows_from_idx(const Slot16* t, const uint32_t* idx, int64_t n, KeyPack kp,
                                 int type, int fold_kind, uint32_t* k0, uint32_t* k1, uint32_t* v,
                                 hipStream_t s) {
  if (n <= 0) return hipSuccess;
  table16_rows_from_idx_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(t, idx, n, kp, type, fold_kind,
                                                                 k0, k1, v);
  return hipGetLastError();
}

// ---- ordered compaction of table slots / counters ----------------------------
// Two passes over the same contiguous ranges (CP_RANGE items per workgroup):
// count the kept items, scan the per-range counts, then write each kept item
// at its range offset plus its rank inside the range.  No shared counter, and
// the output order is the slot order.
constexpr int CP_THREADS = 256;
constexpr int CP_RANGE = CP_THREADS * 32;
// Items per workgroup: CP_RANGE for large inputs, fewer for small ones so
// that about 256 workgroups share the passes (a few long ranges would each
// walk dozens of scan steps one after another).
static int64_t cp_range(int64_t n) {
  const int64_t r = (n / 256 + CP_THREADS - 1) / CP_THREADS * CP_THREADS;
  return std::min<int64_t>(CP_RANGE, std::max<int64_t>(CP_THREADS, r));
}

enum CompactKind { CK_NONEMPTY = 0, CK_STAMP = 1, CK_COUNTER = 2, CK_DENSE = 3 };

struct CompactArgs {
  int kind;
  const Slot16* t;        // CK_NONEMPTY / CK_STAMP
  const uint32_t* counts; // CK_COUNTER; CK_DENSE: value array
  const uint32_t* pres;   // CK_DENSE: presence bits
  const uint32_t* dict;   // CK_DENSE: first-key dictionary
  int64_t n;
  uint32_t round;         // CK_STAMP
  KeyPack kp;
  int type, fold_kind;
  int64_t range1;         // CK_COUNTER: second-key range
  int64_t nrank;          // CK_DENSE: 0 = slot rank * range1 + y, else slot y * nrank + rank
  uint32_t* k0;           // CK_NONEMPTY / CK_COUNTER rows; CK_STAMP: slot indices
  uint32_t* k1;
  uint32_t* v;
  uint32_t* range_cnt;    // [nranges]
  const uint32_t* range_off;
  int64_t out_cap;
  int64_t rlen;           // items per workgroup (cp_range(n), a multiple of CP_THREADS)
};

__device__ __forceinline__ bool cp_keep(const CompactArgs& a, int64_t i) {
  if (i >= a.n) return false;
  if (a.kind == CK_COUNTER) return a.counts[i] != 0;
  if (a.kind == CK_DENSE) return (a.pres[i >> 5] >> (i & 31)) & 1u;
  const Slot16 s = a.t[i];
  if (s.key == EMPTY_KEY) return false;
  return a.kind == CK_NONEMPTY || s.stamp == a.round;
}

__global__ __launch_bounds__(CP_THREADS) void compact_count_k(CompactArgs a) {
  const int64_t base = (int64_t)blockIdx.x * a.rlen;
  uint32_t c = 0;
  for (int64_t k = 0; k < a.rlen / CP_THREADS; ++k) c += cp_keep(a, base + k * CP_THREADS + threadIdx.x);
  uint32_t tot;
  block_excl_scan<uint32_t>(c, &tot);
  if (threadIdx.x == 0) a.range_cnt[blockIdx.x] = tot;
}

// Each step ranks its 256 items by wavefront ballots and one exchange of
// the four wavefront totals: one barrier per step, the exchange words
// alternating between steps so that a step's writes never meet the previous
// step's reads.
__global__ __launch_bounds__(CP_THREADS) void compact_write_k(CompactArgs a) {
  __shared__ uint32_t s_wc[2][CP_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * a.rlen;
  const int w = threadIdx.x >> 6;
  // dense slots below 2^32 (the dense forms' limit) split with 32-bit division
  const bool narrow = a.n <= (int64_t)0xffffffffll && a.nrank <= (int64_t)0xffffffffll &&
                      a.range1 <= (int64_t)0xffffffffll;
  uint32_t out = a.range_off[blockIdx.x];
  for (int64_t k = 0; k < a.rlen / CP_THREADS; ++k) {
    const int64_t i = base + k * CP_THREADS + threadIdx.x;
    const bool keep = cp_keep(a, i);
    const u64 m = __ballot(keep);
    uint32_t* wc = s_wc[k & 1];
    if (lane_id() == 0) wc[w] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int j = 0; j < CP_THREADS / 64; ++j) {
      const uint32_t c = wc[j];
      pre += j < w ? c : 0u;
      tot += c;
    }
    const uint32_t p = out + pre + (uint32_t)__popcll(m & lanemask_lt());
    if (keep && p < (u64)a.out_cap) {
      if (a.kind == CK_STAMP) {
        a.k0[p] = (uint32_t)i;
      } else if (a.kind == CK_DENSE) {
        int64_t rk, yb;
        if (narrow) {
          const uint32_t i32 = (uint32_t)i, d = (uint32_t)(a.nrank ? a.nrank : a.range1);
          const uint32_t q = i32 / d, r = i32 - q * d;
          rk = a.nrank ? r : q;
          yb = a.nrank ? q : r;
        } else {
          rk = a.nrank ? i % a.nrank : i / a.range1;
          yb = a.nrank ? i / a.nrank : i % a.range1;
        }
        a.k0[p] = a.dict[rk];
        if (a.k1) a.k1[p] = (uint32_t)yb + (uint32_t)a.kp.lo[1];
        a.v[p] = stored_value(a.counts[i], a.type, a.fold_kind);
      } else if (a.kind == CK_COUNTER) {
        if (a.kp.nkey == 2) {
          const uint32_t q = narrow ? (uint32_t)i / (uint32_t)a.range1 : (uint32_t)(i / a.range1);
          a.k0[p] = q + (uint32_t)a.kp.lo[0];
          a.k1[p] = (uint32_t)(i - (int64_t)q * a.range1) + (uint32_t)a.kp.lo[1];
        } else {
          a.k0[p] = (uint32_t)i + (uint32_t)a.kp.lo[0];
        }
        a.v[p] = a.counts[i];
      } else {
        const Slot16 s = a.t[i];
        uint32_t x0, x1;
        unpack_key(a.kp, s.key, &x0, &x1);
        a.k0[p] = x0;
        if (a.k1) a.k1[p] = x1;
        a.v[p] = stored_value(s.val, a.type, a.fold_kind);
      }
    }
    out += tot;
  }
}

static hipError_t compact_run(CompactArgs a, uint32_t* total, void* temp, hipStream_t s) {
  a.rlen = cp_range(a.n);
  const int64_t nr = (a.n + a.rlen - 1) / a.rlen;
  if (nr == 0) return hipMemsetAsync(total, 0, 4, s);
  uint32_t* cnt = (uint32_t*)temp;
  uint32_t* off = cnt + ((nr + 63) & ~63ll);
  char* stemp = (char*)(off + ((nr + 63) & ~63ll));
  a.range_cnt = cnt;
  compact_count_k<<<(unsigned)nr, CP_THREADS, 0, s>>>(a);
  hipError_t e = scan_exclusive_u32(cnt, off, nr, total, stemp, s);
  if (e != hipSuccess) return e;
  if (!a.k0) return hipSuccess;  // count only
  a.range_off = off;
  compact_write_k<<<(unsigned)nr, CP_THREADS, 0, s>>>(a);
  return hipGetLastError();
}

size_t compact_temp_bytes(int64_t n) {
  const int64_t nr = (n + cp_range(n) - 1) / cp_range(n);
  return (size_t)((nr + 63) & ~63ll) * 8 + scan_temp_bytes(nr) + 256;
}

hipError_t table16_stamped(const Slot16* t, int64_t cap, uint32_t round, uint32_t* delta_idx,
                           int64_t out_cap, uint32_t* total, void* temp, hipStream_t s) {
  CompactArgs a{};
  a.kind = CK_STAMP;
  a.t = t;
  a.n = cap;
  a.round = round;
  a.k0 = delta_idx;
  a.out_cap = out_cap;
  return compact_run(a, total, temp, s);
}

hipError_t table16_compact(const Slot16* t, int64_t cap, KeyPack kp, int type, int fold_kind,
                           uint32_t* k0, uint32_t* k1, uint32_t* v, int64_t out_cap, uint32_t* total,
                           void* temp, hipStream_t s) {
  CompactArgs a{};
  a.kind = CK_NONEMPTY;
  a.t = t;
  a.n = cap;
  a.kp = kp;
  a.type = type;
  a.fold_kind = fold_kind;
  a.k0 = k0;
  a.k1 = k1;
  a.v = v;
  a.out_cap = out_cap;
  return compact_run(a, total, temp, s);
}

hipError_t dcount_rows(const uint32_t* counts, int64_t n, int64_t range1, KeyPack kp, uint32_t* k0,
                       uint32_t* k1, uint32_t* v, int64_t out_cap, uint32_t* total, void* temp,
                       hipStream_t s) {
  CompactArgs a{};
  a.kind = CK_COUNTER;
  a.counts = counts;
  a.n = n;
  a.kp = kp;
  a.range1 = range1;
  a.k0 = k0;
  a.k1 = k1;
  a.v = v;
  a.out_cap = out_cap;
  return compact_run(a, total, temp, s);
}

hipError_t dense_rows(const uint32_t* vals, const uint32_t* pres, const uint32_t* dict, int64_t n,
                      int64_t range1, int64_t nrank, KeyPack kp, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                      uint32_t* v, int64_t out_cap, uint32_t* total, void* temp, hipStream_t s) {
  CompactArgs a{};
  a.kind = CK_DENSE;
  a.nrank = nrank;
  a.counts = vals;
  a.pres = pres;
  a.dict = dict;
  a.n = n;
  a.kp = kp;
  a.type = type;
  a.fold_kind = fold_kind;
  a.range1 = range1;
  a.k0 = k0;
  a.k1 = k1;
  a.v = v;
  a.out_cap = out_cap;
  return compact_run(a, total, temp, s);
}

// ---- first-key dictionaries ---------------------------------------------------
// mark[v - lo] = 1 for every value of a column that falls in [lo, lo + range).
__global__ void dict_mark_k(const uint32_t* col, int64_t n, int32_t lo, uint32_t range, uint32_t* mark) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t k = col[i] - (uint32_t)lo;
    if (k < range) mark[k] = 1u;
  }
}
hipError_t dict_mark(const uint32_t* col, int64_t n, int32_t lo, uint32_t range, uint32_t* mark, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  dict_mark_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(col, n, lo, range, mark);
  return hipGetLastError();
}

// Marked values get consecutive ranks in value order: map[k] = rank (or
// ~0 when unmarked; map may be the mark array itself), dict[rank] = lo + k.
__global__ void dict_finish_k(uint32_t* map, const uint32_t* pos, uint32_t range, int32_t lo, uint32_t* dict) {
  for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < range; k += gridDim.x * blockDim.x) {
    const bool m = map[k] != 0;
    if (m) dict[pos[k]] = (uint32_t)lo + k;
    map[k] = m ? pos[k] : 0xffffffffu;
  }
}
hipError_t dict_finish(uint32_t* map, const uint32_t* pos, uint32_t range, int32_t lo, uint32_t* dict,
                       hipStream_t s) {
  if (range == 0) return hipSuccess;
  dict_finish_k<<<grid_for(range, 256, 65536), 256, 0, s>>>(map, pos, range, lo, dict);
  return hipGetLastError();
}

// Preloaded rows into a dense value head: improve the value, set presence,
// count keys that were absent.
__global__ void dense_insert_rows_k(uint32_t* vals, uint32_t* pres, const uint32_t* map, uint32_t map_n,
                                    uint32_t range1, const uint32_t* c0, const uint32_t* c1, const uint32_t* v,
                                    int64_t n, KeyPack kp, int type, int is_max, u64* counters) {
  uint32_t mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t k0 = c0[i] - (uint32_t)kp.lo[0];
    const uint32_t k1 = c1 ? c1[i] - (uint32_t)kp.lo[1] : 0u;
    const uint32_t r0 = k0 < map_n ? map[k0] : 0xffffffffu;
    if (r0 == 0xffffffffu || k1 >= range1) {
      atomicOr(&counters[CNT_FATAL], 4ull);
      continue;
    }
    const uint32_t slot = r0 * range1 + k1;
    atomicMin(&vals[slot], fold_encode(v[i], type, is_max));
    const uint32_t bit = 1u << (slot & 31);
    mine += (atomicOr(&pres[slot >> 5], bit) & bit) == 0;
  }
  block_count_add(&counters[CNT_INSERTED], mine);
}
hipError_t dense_insert_rows(uint32_t* vals, uint32_t* pres, const uint32_t* map, uint32_t map_n, uint32_t range1,
                             const uint32_t* c0, const uint32_t* c1, const uint32_t* v, int64_t n, KeyPack kp,
                             int type, int is_max, u64* counters, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  dense_insert_rows_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(vals, pres, map, map_n, range1, c0, c1, v, n, kp,
                                                             type, is_max, counters);
  return hipGetLastError();
}

// Delta rows of the listed slots (values read after the round, i.e. the
// round's best), clearing each slot's listed bit for the next round.
__global__ void dense_delta_rows_k(const uint32_t* idx, int64_t n, const uint32_t* vals, uint32_t* chg,
                                   const uint32_t* dict, uint32_t range1, int32_t lo1, int type, int fold_kind,
                                   uint32_t* k0, uint32_t* k1, uint32_t* v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t slot = idx[i];
    k0[i] = dict[slot / range1];
    if (k1) k1[i] = slot % range1 + (uint32_t)lo1;
    v[i] = stored_value(vals[slot], type, fold_kind);
    atomicAnd(&chg[slot >> 5], ~(1u << (slot & 31)));
  }
}
hipError_t dense_delta_rows(const uint32_t* idx, int64_t n, const uint32_t* vals, uint32_t* chg, const uint32_t* dict,
                            uint32_t range1, int32_t lo1, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                            uint32_t* v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  dense_delta_rows_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(idx, n, vals, chg, dict, range1, lo1, type, fold_kind,
                                                             k0, k1, v);
  return hipGetLastError();
}

// "value is P1 + / - W" of a carried-value rule: one correctly rounded
// binary32 operation (or int32 wrap-around), as the micro-op list would do.
__device__ __forceinline__ uint32_t fast_value(int fast, int type, uint32_t p1, uint32_t w) {
  if (type == T_F32) {
    const float x = __uint_as_float(p1), y = __uint_as_float(w);
    return __float_as_uint(fast == 1 ? __fadd_rn(x, y) : __fsub_rn(x, y));
  }
  return fast == 1 ? p1 + w : p1 - w;
}

// ============================================================ stage kernel
// One launch evaluates one join step of a rule plan for a batch of source
// rows: bind the source row's columns, expand it through an index (all rows
// of the indexed relation whose key column equals a bound variable), bind
// the matched row's columns, run comparisons and arithmetic, and emit.
//
// Load balance: a wavefront takes 64 consecutive source rows, scans their
// index degrees across its lanes, and then walks the concatenated match
// lists 64 entries at a time, each lane finding its owning source row by a
// six-step binary search over the wave's scan in LDS.  Consecutive lanes
// therefore read consecutive rows of the indexed relation (coalesced), and a
// high-degree key occupies one wavefront for as many iterations as it needs
// instead of one thread.

// The descriptor is read in place from the kernel-argument segment (constant
// address space 4, scalar loads) rather than copied into private memory.  The
// address-space qualifier only exists in the device compilation pass.
#if defined(__HIP_DEVICE_COMPILE__)
#define XL_KARG __attribute__((address_space(4)))
#else
#define XL_KARG
#endif
typedef XL_KARG const StageArgs KernArgs;

// Variable slots live in one 8-wide register vector; an access at a uniform
// runtime slot index lowers to register-indexed moves, never to private
// (scratch) memory.
typedef uint32_t Regs __attribute__((ext_vector_type(8)));
__device__ __forceinline__ uint32_t getv(const Regs& u, int i) { return u[i & 7]; }
__device__ __forceinline__ void setv(Regs& u, int i, uint32_t x) { u[i & 7] = x; }
__device__ __forceinline__ bool eqv(uint32_t x, uint32_t y, int type) {
  if (type == T_F32) return __uint_as_float(x) == __uint_as_float(y);
  return x == y;
}

template <typename SRC>
__device__ __forceinline__ bool bind_cols(SRC& src, int64_t row, Regs& u) {
  const int ncols = src.ncols;
  constexpr int NC = sizeof(src.col) / sizeof(src.col[0]);
  bool ok = true;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (c < ncols && src.act[c].kind != CA_NONE) {
      const uint32_t x = src.col[c][row];
      const int kind = src.act[c].kind;
      if (kind == CA_BIND) setv(u, src.act[c].slot, x);
      else if (kind == CA_CHECK_SLOT) ok = ok && eqv(x, getv(u, src.act[c].slot), src.act[c].type);
      else ok = ok && eqv(x, src.act[c].cval, src.act[c].type);
    }
  }
  return ok;
}

template <class A>
__device__ __forceinline__ uint32_t operand(A& a, const Regs& u, int o) {
  if (o >= 0) return getv(u, o);
  uint32_t r = a.consts[0];
#pragma unroll
  for (int k = 1; k < MAXK; ++k)
    if (-1 - o == k) r = a.consts[k];
  return r;
}

__device__ __forceinline__ bool compare(int cmp, int type, uint32_t x, uint32_t y) {
  if (type == T_F32) {
    const float fx = __uint_as_float(x), fy = __uint_as_float(y);
    switch (cmp) {
      case CMP_NE: return fx != fy;
      case CMP_EQ: return fx == fy;
      case CMP_LT: return fx < fy;
      case CMP_LE: return fx <= fy;
      case CMP_GT: return fx > fy;
      default: return fx >= fy;
    }
  }
  const int32_t ix = (int32_t)x, iy = (int32_t)y;
  switch (cmp) {
    case CMP_NE: return ix != iy;
    case CMP_EQ: return ix == iy;
    case CMP_LT: return ix < iy;
    case CMP_LE: return ix <= iy;
    case CMP_GT: return ix > iy;
    default: return ix >= iy;
  }
}

// Stratified negation: does the negated relation have a row whose
// constrained columns equal (x[, y])?  Binary search of the sorted keys.
__device__ __forceinline__ bool neg_member(const NegTable t, int ncols, uint32_t x, uint32_t y) {
  if (ncols == 0) return t.n > 0;
  const u64 k = ncols == 1 ? (u64)x : ((u64)x << 32) | y;
  int64_t lo = 0, hi = t.n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (t.keys[mid] < k) lo = mid + 1;
    else hi = mid;
  }
  return lo < t.n && t.keys[lo] == k;
}

template <class A>
__device__ __forceinline__ bool run_ops(A& a, Regs& u) {
  bool ok = true;
#pragma unroll
  for (int i = 0; i < MAXOPS; ++i) {
    if (i >= a.nops) continue;
    const MicroOp op = a.ops[i];
    const uint32_t x = operand(a, u, op.a);
    if (op.kind == OP_CMP) {
      ok = ok && compare(op.cmp, op.type, x, operand(a, u, op.b));
    } else if (op.kind == OP_NOTIN) {
      const NegTable t = {a.neg[op.cmp].keys, a.neg[op.cmp].n};
      ok = ok && !neg_member(t, op.type, x, op.type > 1 ? operand(a, u, op.b) : 0u);
    } else if (op.kind == OP_MOV) {
      setv(u, op.dst, x);
    } else {
      const uint32_t y = operand(a, u, op.b);
      uint32_t r;
      if (op.type == T_F32) {
        const float fx = __uint_as_float(x), fy = __uint_as_float(y);
        // one correctly rounded binary32 operation, never contracted
        r = __float_as_uint(op.kind == OP_ADD ? __fadd_rn(fx, fy) : __fsub_rn(fx, fy));
      } else {
        r = op.kind == OP_ADD ? x + y : x - y;
      }
      setv(u, op.dst, r);
    }
  }
  return ok;
}

// Micro-op evaluation, specialized at launch: OPS 0 = no ops, 2 = the
// affine pattern "v is x + / - y" (a move then an add or subtract of two
// slots), 1 = the general interpreter.
template <int OPS>
__device__ __forceinline__ bool eval_ops(KernArgs& a, Regs& u) {
  if (OPS == 0) return true;
  if (OPS == 2) {
    setv(u, a.ops[0].dst, fast_value(a.ops[1].kind == OP_ADD ? 1 : 2, a.ops[1].type, getv(u, a.ops[0].a),
                                     getv(u, a.ops[1].b)));
    return true;
  }
  return run_ops(a, u);
}

// Accumulators of hashed sum/logsumexp folds (EM_HAGG), one 64-bit word per
// table slot.  Integer sums add modulo 2^32 in the low word (the result of
// any order); f32 sums add in f64 and logsumexp folds in f64 with
// max + log1p(exp(-|a - b|)), so the order in which a round's contributions
// arrive moves the f64 result by a few units of its last place, far below
// the f32 rounding applied when the round ends.
__device__ __forceinline__ double lse2d(double a, double b) {
  if (a == -HUGE_VAL) return b;
  if (b == -HUGE_VAL) return a;
  return fmax(a, b) + log1p(exp(-fabs(a - b)));
}
__device__ __forceinline__ u64 acc_identity(int type, int fold_kind) {
  if (fold_kind == FOLD_LSE) return (u64)__double_as_longlong(-HUGE_VAL);
  (void)type;
  return 0ull;  // integer 0 in the low word, or f64 +0.0
}
__device__ __forceinline__ void acc_add(u64* acc, uint32_t x, int type, int fold_kind) {
  if (fold_kind == FOLD_LSE) {
    const double v = (double)__uint_as_float(x);
    if (v == -HUGE_VAL) return;
    u64 old = *acc;
    for (;;) {
      const u64 nv = (u64)__double_as_longlong(lse2d(__longlong_as_double((long long)old), v));
      const u64 prev = atomicCAS(acc, old, nv);
      if (prev == old) break;
      old = prev;
    }
  } else if (type == T_F32) {
    atomicAdd(reinterpret_cast<double*>(acc), (double)__uint_as_float(x));
  } else {
    atomicAdd(reinterpret_cast<uint32_t*>(acc), x);
  }
}
// The round's fold of one key, as the value type's bits.
__device__ __forceinline__ uint32_t acc_value(u64 a, int type, int fold_kind) {
  if (fold_kind == FOLD_LSE || type == T_F32) return __float_as_uint((float)__longlong_as_double((long long)a));
  return (uint32_t)a;
}

// Rows produced by EM_SET / EM_BITSET / EM_MINMAX are staged in a per-wave
// LDS buffer and written out with one counter reservation per flush, so a
// launch issues one global atomic per OUTB rows instead of one per 64.
constexpr int OUTB = 512;

struct EmitState {
  u64 out_base;     // EM_MAT: first output position of this chunk
  uint32_t running; // rows emitted so far in this chunk
  u64 cands;        // candidates seen by this wave (flushed once at the end)
  bool stop;        // overflow observed: no further inserts in this launch
  uint32_t pend_idx, pend_cnt;  // EM_DCOUNT: open run carried to the next batch
  uint32_t buf_n;   // staged rows in this wave's buffer
  uint32_t ins_pend;  // EM_MINMAX: keys inserted since the last flush
  uint32_t* buf0;   // this wave's LDS staging columns
  uint32_t* buf1;
};

__device__ __forceinline__ u64 shfl_u64(u64 v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src, 64), hi = __shfl((uint32_t)(v >> 32), src, 64);
  return ((u64)hi << 32) | lo;
}

// Write the wave's staged rows with one reservation; the reservation also
// tells the wave whether the launch has passed its load limit.
template <int MODE>
__device__ __forceinline__ void flush_rows(KernArgs& a, EmitState& st) {
  typedef XL_KARG const EmitSpec KEmit;
  KEmit& e = a.emit;
  const int lane = lane_id();
  if ((MODE == EM_MINMAX || MODE == EM_DMIN || MODE == EM_HAGG) && st.ins_pend) {
    u64 b = 0;
    if (lane == 0) {
      b = atomicAdd(&e.counters[CNT_INSERTED], (u64)st.ins_pend);
      if (b + st.ins_pend > e.limit) atomicOr(&e.counters[CNT_OVERFLOW], 1ull);
    }
    b = shfl_u64(b, 0);
    if (b + st.ins_pend > e.limit) st.stop = true;
    st.ins_pend = 0;
  }
  if (st.buf_n == 0) return;
  wave_lds_sync();
  u64 base = 0;
  constexpr bool SLOTS = MODE == EM_MINMAX || MODE == EM_DMIN || MODE == EM_HAGG;
  if (lane == 0) {
    base = atomicAdd(&e.counters[CNT_APPENDED], (u64)st.buf_n);
    if (SLOTS ? e.delta_lim && base + st.buf_n > e.delta_lim : base + st.buf_n > e.limit)
      atomicOr(&e.counters[CNT_OVERFLOW], 1ull);
  }
  base = shfl_u64(base, 0);
  if (SLOTS ? e.delta_lim && base + st.buf_n > e.delta_lim : base + st.buf_n > e.limit) st.stop = true;
  for (uint32_t i = lane; i < st.buf_n; i += 64) {
    if (SLOTS) {
      if (!e.delta_lim || base + i < e.delta_lim) e.delta_idx[base + i] = st.buf0[i];
    } else {
      const u64 p = (u64)e.row_base + base + i;
      if (p < (u64)e.row_cap) {
        e.row_col[0][p] = st.buf0[i];
        if (e.key.nkey == 2) e.row_col[1][p] = st.buf1[i];
      } else {
        atomicOr(&e.counters[CNT_FATAL], 2ull);
      }
    }
  }
  wave_lds_sync();
  st.buf_n = 0;
}

template <int MODE>
__device__ __forceinline__ void emit(KernArgs& a, const Regs& u, bool act,
                                     EmitState& st) {
  typedef XL_KARG const EmitSpec KEmit;
  KEmit& e = a.emit;
  const u64 lt = lanemask_lt();
  if (MODE == EM_COUNT) {
    st.running += (uint32_t)__popcll(__ballot(act));
    return;
  }
  if (MODE == EM_MAT) {
    const u64 m = __ballot(act);
    if (act) {
      const u64 pos = st.out_base + st.running + __popcll(m & lt);
      if (e.mat_packed) {
        const u64 key = pack_key(e.key, getv(u, e.key.slot[0]), getv(u, e.key.slot[1]));
        if (e.key32) ((uint32_t*)e.out_key)[pos] = (uint32_t)key;
        else e.out_key[pos] = key;
        if (e.val_slot >= 0) e.out_val[pos] = getv(u, e.val_slot);
      } else {
#pragma unroll
        for (int i = 0; i < MAXV; ++i)
          if (i < e.nout) e.out_col[i][pos] = getv(u, e.out_slot[i]);
      }
    }
    st.running += (uint32_t)__popcll(m);
    return;
  }
  // EM_SET / EM_BITSET / EM_MINMAX: stop early once the load limit is passed.
  st.cands += (u64)__popcll(__ballot(act));
  if (MODE != EM_DCOUNT && st.stop) return;
  if (MODE == EM_SET || MODE == EM_BITSET) {
    int ins = 0;
    if (MODE == EM_SET) {
      if (act) ins = set_insert(e.table, e.mask, pack_key(e.key, getv(u, e.key.slot[0]), getv(u, e.key.slot[1])),
                                e.counters);
    } else {
      // Dense domain: the packed key's two components index row and column.
      // Consecutive lanes that hit the same bitmap word (neighbouring second
      // keys of one first key) form a run; the run's bits are OR-combined
      // and its first lane does a single test-and-set for all of them.  The
      // bits that were off are this round's new tuples: they are set in the
      // delta bitmap (dchg), which is turned into rows after the round.
      u64 wi = ~0ull;
      uint32_t bit = 0;
      if (act) {
        const u64 key = pack_key(e.key, getv(u, e.key.slot[0]), getv(u, e.key.slot[1]));
        const u64 b = e.key.nkey == 2
                          ? (key >> e.key.shift) * e.row_bits + (key & ((1ull << e.key.shift) - 1ull))
                          : key;
        wi = b >> 5;
        bit = 1u << (b & 31);
      }
      const int lane = lane_id();
      const u64 prev = shfl_u64(wi, lane > 0 ? lane - 1 : 0);
      const u64 am = __ballot(act);
      const bool head = act && (lane == 0 || !((am >> (lane - 1)) & 1ull) || prev != wi);
      const u64 heads = __ballot(head) | ~am;
      const int h0 = 63 - __clzll((long long)(heads & ((2ull << lane) - 1ull)));
      const u64 ahead = heads & ~((2ull << lane) - 1ull);
      const int tail = (ahead ? __ffsll((long long)ahead) - 1 : 64) - 1;
      // inclusive OR of the run's bits from its first lane
      uint32_t incl = bit;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t t = __shfl_up(incl, d, 64);
        if (lane - d >= h0) incl |= t;
      }
      const uint32_t total = __shfl(incl, tail, 64);
      if (head) {
        uint32_t* wp = e.bits + wi;
        const uint32_t cur = *wp;
        if ((cur & total) != total) {
          // the bits this run turned on are new tuples: they go to the delta bitmap
          const uint32_t fresh = total & ~atomicOr(wp, total);
          if (fresh) {
            atomicOr(&e.dchg[wi], fresh);
            st.ins_pend += (uint32_t)__popc(fresh);
          }
        }
      }
      return;
    }
    const u64 m = __ballot(ins);
    if (m) {
      if (st.buf_n + 64 > OUTB) flush_rows<MODE>(a, st);
      if (ins) {
        const uint32_t pos = st.buf_n + (uint32_t)__popcll(m & lt);
        st.buf0[pos] = getv(u, e.key.slot[0]);
        st.buf1[pos] = getv(u, e.key.slot[1]);
      }
      st.buf_n += (uint32_t)__popcll(m);
    }
    return;
  }
  if (MODE == EM_DCOUNT) {
    // lanes holding the same key consecutively form a run; one atomic per run
    uint32_t idx = 0;
    if (act) {
      const u64 key = pack_key(e.key, getv(u, e.key.slot[0]), getv(u, e.key.slot[1]));
      idx = (uint32_t)(e.key.nkey == 2
                           ? (key >> e.key.shift) * e.row_bits + (key & ((1ull << e.key.shift) - 1ull))
                           : key);
    }
    const int lane = lane_id();
    const uint32_t prev = __shfl_up(idx, 1, 64);
    const u64 am = __ballot(act);
    const bool prev_act = lane > 0 && ((am >> (lane - 1)) & 1ull);
    const bool start = act && !(prev_act && prev == idx);
    const u64 sm = __ballot(start);
    if (!sm) return;
    const u64 bnd = sm | ~am;
    uint32_t len = 0;
    if (start) {
      const u64 above = bnd & ~((2ull << lane) - 1ull);
      const int nxt = above ? __ffsll((long long)above) - 1 : 64;
      len = (uint32_t)(nxt - lane);
    }
    // The wave walks its rows in order: the batch's last run stays open and
    // absorbs the next batch's first run when the key repeats (sums commute,
    // so merging equal keys is always exact).
    const int f = __ffsll((long long)sm) - 1;
    const int l = 63 - __clzll((long long)sm);
    const uint32_t idx_f = __shfl(idx, f, 64), len_f = __shfl(len, f, 64);
    const uint32_t idx_l = __shfl(idx, l, 64), len_l = __shfl(len, l, 64);
    const bool merged = st.pend_cnt && st.pend_idx == idx_f;
    if (start && lane != l && !(lane == f && merged)) atomicAdd(&e.bits[idx], len);
    if (merged) st.pend_cnt += len_f;
    if (!(merged && f == l)) {
      if (st.pend_cnt && lane == 0) atomicAdd(&e.bits[st.pend_idx], st.pend_cnt);
      st.pend_idx = idx_l;
      st.pend_cnt = len_l;
    }
    return;
  }
  if (MODE == EM_DMIN) {
    // Dense slots: a plain read first (most candidates do not improve), then
    // one atomicMin.  A slot holds a key once its presence bit is set; the
    // lane that sets it counts the key.  The first lane to improve a slot in
    // this round lists it in the delta.
    bool ins = false, app = false;
    uint32_t slot = 0;
    if (act) {
      const uint32_t k0 = getv(u, e.key.slot[0]) - (uint32_t)e.key.lo[0];
      const uint32_t k1 = e.key.nkey == 2 ? getv(u, e.key.slot[1]) - (uint32_t)e.key.lo[1] : 0u;
      const uint32_t r0 = k0 < e.dmap_n ? e.dmap[k0] : 0xffffffffu;
      if (r0 == 0xffffffffu || (u64)k1 >= e.row_bits) {
        atomicOr(&e.counters[CNT_FATAL], 4ull);  // key outside the planned domain
      } else {
        slot = r0 * (uint32_t)e.row_bits + k1;
        const uint32_t enc = fold_encode(getv(u, e.val_slot), e.val_type, e.is_max);
        const uint32_t cur = e.bits[slot];
        bool better = false;
        uint32_t old = cur;
        if (enc < cur) {
          old = atomicMin(&e.bits[slot], enc);
          better = enc < old;
        }
        const uint32_t bit = 1u << (slot & 31);
        if ((better && old == 0xffffffffu) || (enc == 0xffffffffu && cur == 0xffffffffu))
          ins = (atomicOr(&e.dpres[slot >> 5], bit) & bit) == 0;
        if (better || ins) app = (atomicOr(&e.dchg[slot >> 5], bit) & bit) == 0;
      }
    }
    st.ins_pend += (uint32_t)__popcll(__ballot(ins));
    const u64 ma = __ballot(app);
    if (ma || st.ins_pend + 64 > OUTB) {
      if (st.buf_n + 64 > OUTB || st.ins_pend + 64 > OUTB) flush_rows<MODE>(a, st);
      if (app) st.buf0[st.buf_n + (uint32_t)__popcll(ma & lt)] = slot;
      st.buf_n += (uint32_t)__popcll(ma);
    }
    return;
  }
  if (MODE == EM_MARK) {
    if (act) {
      const uint32_t k0 = getv(u, e.key.slot[0]) - (uint32_t)e.key.lo[0];
      const uint32_t k1 = getv(u, e.key.slot[1]) - (uint32_t)e.key.lo[1];
      const uint32_t r0 = k0 < e.dmap_n ? e.dmap[k0] : 0xffffffffu;
      if (r0 == 0xffffffffu || (u64)k1 >= e.row_bits) {
        atomicOr(&e.counters[CNT_FATAL], 4ull);
      } else {
        const uint32_t slot = k1 * e.nrank + r0, bit = 1u << (slot & 31);
        if (!(e.dchg[slot >> 5] & bit)) atomicOr(&e.dchg[slot >> 5], bit);
      }
    }
    return;
  }
  if (MODE == EM_MINMAX || MODE == EM_HAGG) {
    bool ins = false, app = false;
    u64 slot = ~0ull;
    if (act) {
      slot = slot_find_or_insert(e.table16, e.mask, pack_key(e.key, getv(u, e.key.slot[0]),
                                                             getv(u, e.key.slot[1])),
                                 &ins, e.counters);
      if (slot != ~0ull) {
        if (MODE == EM_MINMAX) {
          const uint32_t enc = fold_encode(getv(u, e.val_slot), e.val_type, e.is_max);
          const uint32_t old = atomicMin(&e.table16[slot].val, enc);
          if (ins || enc < old) app = atomicExch(&e.table16[slot].stamp, e.round) != e.round;
        } else {
          // the full-relation value is only read by the round's merge
          if (ins) e.table16[slot].val = e.agg_identity;
          acc_add(e.acc + slot, getv(u, e.val_slot), e.val_type, e.fold_kind);
          app = atomicExch(&e.table16[slot].stamp, e.round) != e.round;
        }
      }
    }
    st.ins_pend += (uint32_t)__popcll(__ballot(ins));
    const u64 ma = __ballot(app);
    if (ma || st.ins_pend + 64 > OUTB) {
      if (st.buf_n + 64 > OUTB || st.ins_pend + 64 > OUTB) flush_rows<MODE>(a, st);
      if (app) st.buf0[st.buf_n + (uint32_t)__popcll(ma & lt)] = (uint32_t)slot;
      st.buf_n += (uint32_t)__popcll(ma);
    }
  }
}

constexpr int ST_THREADS = 256;
constexpr int ST_WAVES = ST_THREADS / 64;

template <int MODE, bool HAS_INDEX, int OPS>
__global__ __launch_bounds__(ST_THREADS) void stage_k(StageArgs by_value) {
  (void)by_value;
  KernArgs& a = *(KernArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ uint32_t s_excl[ST_WAVES][64];
  __shared__ uint32_t s_beg[ST_WAVES][64];
  __shared__ uint32_t s_beg2[ST_WAVES][64], s_deg2[ST_WAVES][64];
  __shared__ uint32_t s_v[ST_WAVES][MAXV][64];
  constexpr bool STAGED = MODE == EM_SET || MODE == EM_BITSET || MODE == EM_MINMAX || MODE == EM_DMIN ||
                         MODE == EM_HAGG;
  __shared__ uint32_t s_out[STAGED ? ST_WAVES : 1][2][STAGED ? OUTB : 1];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  int64_t src_n = a.src.n, src_base = 0;
  if (a.src_range) {  // batched rounds: the round's delta range lives on the device
    src_base = (int64_t)a.src_range[0];
    src_n = a.emit.counters[CNT_OVERFLOW] ? 0 : (int64_t)a.src_range[1] - src_base;
  }
  const int64_t nchunks = (src_n + 63) / 64;
  const int64_t nwaves = (int64_t)gridDim.x * ST_WAVES;
  EmitState st;
  st.stop = false;
  st.cands = 0;
  st.pend_idx = st.pend_cnt = 0;
  st.buf_n = st.ins_pend = 0;
  st.buf0 = s_out[STAGED ? w : 0][0];
  st.buf1 = s_out[STAGED ? w : 0][1];
  // EM_DCOUNT walks one contiguous range of chunks per wave (runs of equal
  // keys stay in one wave); every other mode interleaves chunks.
  const int64_t wave_id = (int64_t)blockIdx.x * ST_WAVES + w;
  const int64_t per = (nchunks + nwaves - 1) / nwaves;
  const int64_t c_first = MODE == EM_DCOUNT ? wave_id * per : wave_id;
  const int64_t c_end = MODE == EM_DCOUNT ? min(nchunks, c_first + per) : nchunks;
  const int64_t c_step = MODE == EM_DCOUNT ? 1 : nwaves;
  for (int64_t chunk = c_first; chunk < c_end; chunk += c_step) {
    st.running = 0;
    st.out_base = (MODE == EM_MAT) ? a.emit.chunk_off[chunk] + (u64)a.emit.mat_base : 0;
    const int64_t row = chunk * 64 + lane;
    Regs v = (Regs)(0u);
    bool ok = row < src_n;
    if (ok) ok = bind_cols(a.src, src_base + row, v);
    if (HAS_INDEX) {
      uint32_t beg = 0, deg = 0, beg2 = 0, deg2 = 1;
      if (ok) {
        uint32_t kk;
        if (index_segment(a.idx, getv(v, a.idx.key_slot), &kk)) {
          beg = a.idx.off[kk];
          deg = a.idx.off[kk + 1] - beg;
          // the wave's match count must stay below 2^32: a key with 2^26 or
          // more rows is refused (the host reports it as unsupported)
          if (deg >= (1u << 26)) {
            atomicOr(&a.emit.counters[CNT_FATAL], 32ull);
            deg = 0;
          }
        }
        if (a.has_idx2) {
          uint32_t k2;
          deg2 = 0;
          if (index_segment(a.idx2, getv(v, a.idx2.key_slot), &k2)) {
            beg2 = a.idx2.off[k2];
            deg2 = a.idx2.off[k2 + 1] - beg2;
          }
          // the wave's product count must stay below 2^32: a row beyond
          // 2^24 products is refused (the host then runs the two steps apart)
          if ((u64)deg * deg2 >= (1u << 24)) {
            atomicOr(&a.emit.counters[CNT_FATAL], 16ull);
            // batched rounds stop here, so the host re-runs this round apart
            if (a.src_range) atomicOr(&a.emit.counters[CNT_OVERFLOW], 1ull);
            deg = 0;
          } else {
            deg *= deg2;
          }
        }
      }
      const uint32_t incl = wave_incl_scan(deg);
      const uint32_t total = __shfl(incl, 63, 64);
      s_excl[w][lane] = incl - deg;
      s_beg[w][lane] = beg;
      s_beg2[w][lane] = beg2;
      s_deg2[w][lane] = deg2;
#pragma unroll
      for (int s = 0; s < MAXV; ++s) s_v[w][s][lane] = v[s];
      wave_lds_sync();
      for (uint32_t base = 0; base < total; base += 64) {
        const uint32_t j = base + lane;
        bool act = j < total;
        int r = 0;
#pragma unroll
        for (int step = 32; step > 0; step >>= 1)
          if (s_excl[w][r + step] <= j) r += step;
        Regs u;
#pragma unroll
        for (int s = 0; s < MAXV; ++s) u[s] = s_v[w][s][r];
        if (act) {
          const uint32_t k = j - s_excl[w][r];
          if (a.has_idx2) {
            const uint32_t d2 = s_deg2[w][r];
            act = bind_cols(a.idx, s_beg[w][r] + k / d2, u) && bind_cols(a.idx2, s_beg2[w][r] + k % d2, u);
          } else {
            act = bind_cols(a.idx, s_beg[w][r] + k, u);
          }
        }
        if (act) act = eval_ops<OPS>(a, u);
        emit<MODE>(a, u, act, st);
      }
      wave_lds_sync();
    } else {
      bool act = ok;
      if (act) act = eval_ops<OPS>(a, v);
      emit<MODE>(a, v, act, st);
    }
    if (MODE == EM_COUNT && lane == 0) a.emit.chunk_cnt[chunk] = st.running;
  }
  if (MODE == EM_SET || MODE == EM_BITSET || MODE == EM_MINMAX || MODE == EM_DCOUNT || MODE == EM_DMIN ||
      MODE == EM_MARK || MODE == EM_HAGG) {
    // one atomic per workgroup: a shared counter hit by every wave serializes
    __shared__ u64 s_cands[ST_WAVES], s_new[ST_WAVES];
    u64 nw = 0;
    if (MODE == EM_BITSET) {  // new tuples: per-lane counts summed over the wave
      nw = st.ins_pend;
      for (int k = 32; k > 0; k >>= 1) nw += __shfl_xor(nw, k, 64);
    }
    if (lane == 0) {
      s_cands[w] = st.cands;
      s_new[w] = nw;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      u64 t = 0, tn = 0;
      for (int i = 0; i < ST_WAVES; ++i) {
        t += s_cands[i];
        tn += s_new[i];
      }
      if (t) atomicAdd(&a.emit.counters[CNT_CANDIDATES], t);
      if (tn) atomicAdd(&a.emit.counters[CNT_APPENDED], tn);
    }
  }
  if (MODE == EM_DCOUNT && st.pend_cnt && lane == 0) atomicAdd(&a.emit.bits[st.pend_idx], st.pend_cnt);
  if (STAGED) flush_rows<MODE>(a, st);  // rows already inserted are always written
}

static int ops_kind(const StageArgs& a) {
  if (a.nops == 0) return 0;
  const MicroOp& m = a.ops[0];
  const MicroOp& o = a.ops[1];
  if (a.nops == 2 && m.kind == OP_MOV && m.a >= 0 && (o.kind == OP_ADD || o.kind == OP_SUB) && o.dst == m.dst &&
      o.a == m.dst && o.b >= 0 && o.type == m.type)
    return 2;
  return 1;
}

template <int MODE, int OPS>
static void launch_ops(const StageArgs& a, unsigned grid, hipStream_t s) {
  if (a.has_index) stage_k<MODE, true, OPS><<<grid, ST_THREADS, 0, s>>>(a);
  else stage_k<MODE, false, OPS><<<grid, ST_THREADS, 0, s>>>(a);
}

template <int MODE>
static void launch_mode(const StageArgs& a, unsigned grid, hipStream_t s) {
  switch (ops_kind(a)) {
    case 0: launch_ops<MODE, 0>(a, grid, s); break;
    case 2: launch_ops<MODE, 2>(a, grid, s); break;
    default: launch_ops<MODE, 1>(a, grid, s); break;
  }
}

// Batched rounds of a set head over its append-only row list: bnd[j] is the
// row count after round j - 1 of the batch (bnd[0], bnd[1] bound the first
// round's delta, later entries start as ~0).  After round j's launches,
// bnd[j + 1] = base + rows appended in the batch so far, unless a launch of
// the batch overflowed (the entry then stays ~0 and the host re-runs round j).
__global__ void batch_init_k(u64* bnd, int n, u64 b0, u64 b1) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) bnd[i] = i == 0 ? b0 : i == 1 ? b1 : ~0ull;
}
__global__ void batch_mark_k(u64* bnd, int j, const u64* counters, u64 base) {
  if (threadIdx.x == 0 && !counters[CNT_OVERFLOW]) bnd[j + 1] = base + counters[CNT_APPENDED];
}
hipError_t batch_init(u64* bnd, int n, u64 b0, u64 b1, hipStream_t s) {
  batch_init_k<<<1, 256, 0, s>>>(bnd, n, b0, b1);
  return hipGetLastError();
}
hipError_t batch_mark(u64* bnd, int j, const u64* counters, u64 base, hipStream_t s) {
  batch_mark_k<<<1, 64, 0, s>>>(bnd, j, counters, base);
  return hipGetLastError();
}
__global__ void batch_mark_heads_k(BatchMarks m, int j) {
  if (threadIdx.x != 0) return;
  u64 any = 0;
  for (int h = 0; h < m.n; ++h) any |= m.cnt[h][CNT_OVERFLOW];
  for (int h = 0; h < m.n; ++h) {
    if (any) m.cnt[h][CNT_OVERFLOW] = 1ull;
    else m.bnd[h][j + 1] = m.base[h] + m.cnt[h][CNT_APPENDED];
  }
}
hipError_t batch_mark_heads(const BatchMarks& m, int j, hipStream_t s) {
  if (m.n <= 0 || m.n > MAX_BATCH_HEADS) return hipErrorInvalidValue;
  batch_mark_heads_k<<<1, 64, 0, s>>>(m, j);
  return hipGetLastError();
}

hipError_t stage_launch(const StageArgs& a, hipStream_t s, int grid_cap) {
  if (a.src.n <= 0) return hipSuccess;
  const int64_t nchunks = (a.src.n + 63) / 64;
  const unsigned grid = grid_for(nchunks, ST_WAVES, grid_cap);
  switch (a.emit.mode) {
    case EM_DCOUNT: launch_mode<EM_DCOUNT>(a, std::min(grid, 4096u), s); return hipGetLastError();
    case EM_COUNT: launch_mode<EM_COUNT>(a, grid, s); break;
    case EM_MAT: launch_mode<EM_MAT>(a, grid, s); break;
    case EM_SET: launch_mode<EM_SET>(a, grid, s); break;
    case EM_BITSET: launch_mode<EM_BITSET>(a, grid, s); break;
    case EM_DMIN: launch_mode<EM_DMIN>(a, grid, s); break;
    case EM_MARK: launch_mode<EM_MARK>(a, grid, s); break;
    case EM_HAGG: launch_mode<EM_HAGG>(a, grid, s); break;
    default: launch_mode<EM_MINMAX>(a, grid, s); break;
  }
  return hipGetLastError();
}

// ============================================================ dense sum / logsumexp heads
// Marked slots -> ascending slot list, clearing the marks.  Each workgroup
// owns MK_THREADS * wpt consecutive bitmap words: count pass, scan of the per-group
// counts, write pass.
constexpr int MK_THREADS = 256, MK_WPT = 4;

// Words per thread of a bitmap pass over nw words: the most (at most MK_WPT)
// that still gives about 512 workgroups, so a small bitmap spreads over the
// chip.  The count and write passes of one bitmap take the same value.
static int mk_wpt(int64_t nw) {
  return nw >= (int64_t)MK_THREADS * 4 * 512 ? 4 : nw >= (int64_t)MK_THREADS * 2 * 512 ? 2 : 1;
}
static int64_t mk_blocks(int64_t nw, int wpt) {
  const int64_t words = (int64_t)MK_THREADS * wpt;
  return (nw + words - 1) / words;
}

__global__ __launch_bounds__(MK_THREADS) void bits_count_k(const uint32_t* bits, int64_t nw, int wpt, uint32_t* cnt) {
  const int64_t w0 = (int64_t)blockIdx.x * MK_THREADS * wpt + (int64_t)threadIdx.x * wpt;
  uint32_t c = 0;
  for (int k = 0; k < wpt; ++k)
    if (w0 + k < nw) c += __popc(bits[w0 + k]);
  uint32_t tot;
  block_excl_scan<uint32_t>(c, &tot);
  if (threadIdx.x == 0) cnt[blockIdx.x] = tot;
}

__global__ __launch_bounds__(MK_THREADS) void bits_list_k(uint32_t* bits, int64_t nw, int wpt, const uint32_t* off,
                                                          uint32_t* list) {
  const int64_t w0 = (int64_t)blockIdx.x * MK_THREADS * wpt + (int64_t)threadIdx.x * wpt;
  uint32_t d[MK_WPT], c = 0;
#pragma unroll
  for (int k = 0; k < MK_WPT; ++k) {
    d[k] = k < wpt && w0 + k < nw ? bits[w0 + k] : 0u;
    c += __popc(d[k]);
  }
  uint32_t tot;
  uint32_t p = off[blockIdx.x] + block_excl_scan<uint32_t>(c, &tot);
#pragma unroll
  for (int k = 0; k < MK_WPT; ++k) {
    if (!d[k]) continue;
    bits[w0 + k] = 0u;
    for (uint32_t b = d[k]; b; b &= b - 1) list[p++] = (uint32_t)(w0 + k) * 32u + (uint32_t)(__ffs(b) - 1);
  }
}

// Marked slots -> slot list in one pass, clearing the marks: each wavefront
// takes 128 consecutive words (two per lane, lane-major, so the loads
// coalesce; a wavefront's word columns go out one after another, so short
// wavefronts finish sooner); the four wavefronts of a workgroup reserve
// their entries with one atomic on *total (one per wavefront put thousands
// of same-address atomics in line) and each writes its entries in word
// order.  The list is ascending within each wavefront's range and
// the ranges land in any order: for consumers that take each listed key on
// its own (the dense pull folds every key's in-edges itself).  Each word
// column's entries are staged in LDS (entry o at o + o / 32, so the lanes of
// a nearly full column write different banks) and go out with consecutive
// lanes on consecutive entries.  *total must be zero before the launch.
constexpr int LW_WORDS = 2;
constexpr int LW_STAGE = 64 * 32 + 64;  // one column's entries, padded
__global__ __launch_bounds__(256) void bits_list_waves_k(uint32_t* bits, int64_t nw, uint32_t* list, uint32_t* total) {
  __shared__ uint32_t stage_all[4][LW_STAGE];
  __shared__ uint32_t s_all[4], s_base[4];
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  uint32_t* stage = stage_all[wv];
  // workgroup-uniform steps (the reservation takes two barriers)
  for (int64_t g0 = (int64_t)blockIdx.x * 4 * 64 * LW_WORDS; g0 < nw; g0 += (int64_t)gridDim.x * 4 * 64 * LW_WORDS) {
    const int64_t w0 = g0 + (int64_t)wv * 64 * LW_WORDS;
    uint32_t d[LW_WORDS], run[LW_WORDS], cnt[LW_WORDS], all = 0;
#pragma unroll
    for (int k = 0; k < LW_WORDS; ++k) {
      const int64_t wi = w0 + k * 64 + lane;
      d[k] = wi < nw ? bits[wi] : 0u;
      const uint32_t c = (uint32_t)__popc(d[k]);
      const uint32_t incl = wave_incl_scan(c);
      run[k] = incl - c;
      cnt[k] = __shfl(incl, 63, 64);
      all += cnt[k];
    }
    if (lane == 0) s_all[wv] = all;
    __syncthreads();
    if (threadIdx.x == 0) {
      const uint32_t a0 = s_all[0], a1 = s_all[1], a2 = s_all[2], a3 = s_all[3];
      const uint32_t sum = a0 + a1 + a2 + a3;
      const uint32_t b = sum ? atomicAdd(total, sum) : 0u;
      s_base[0] = b;
      s_base[1] = b + a0;
      s_base[2] = b + a0 + a1;
      s_base[3] = b + a0 + a1 + a2;
    }
    __syncthreads();
    if (all == 0) continue;  // (wave-uniform; the next step's barriers come after s_base is read)
    uint32_t base = s_base[wv];
#pragma unroll
    for (int k = 0; k < LW_WORDS; ++k) {
      if (cnt[k] == 0) continue;  // (wave-uniform)
      const int64_t wi = w0 + k * 64 + lane;
      if (d[k]) {
        bits[wi] = 0u;
        uint32_t o = run[k];
        for (uint32_t b = d[k]; b; b &= b - 1, ++o) stage[o + (o >> 5)] = (uint32_t)wi * 32u + (uint32_t)(__ffs(b) - 1);
      }
      wave_lds_sync();
      for (uint32_t o = (uint32_t)lane; o < cnt[k]; o += 64) list[base + o] = stage[o + (o >> 5)];
      base += cnt[k];
      wave_lds_sync();
    }
  }
}
hipError_t bits_list_waves(uint32_t* bits, int64_t nbits, uint32_t* list, uint32_t* total, hipStream_t s) {
  const int64_t nw = (nbits + 31) / 32;
  if (nw <= 0) return hipSuccess;
  const int64_t waves = (nw + 64 * LW_WORDS - 1) / (64 * LW_WORDS);
  bits_list_waves_k<<<(unsigned)std::min<int64_t>((waves + 3) / 4, 2048), 256, 0, s>>>(bits, nw, list, total);
  return hipGetLastError();
}

// Rows (k0, k1) of the set bits of a dense key bitmap, in bit order: bit b
// is k0 = lo0 + b / row_bits, k1 = lo1 + b % row_bits (one key: k0 = lo0 + b).
// Optionally clears the words it read (a delta bitmap).  A workgroup owns
// MK_THREADS * wpt consecutive words (the same ranges as bits_count_k) and walks them
// in steps of one word per thread: the step's set bits are ranked by a block
// scan and staged in LDS, then written out with consecutive threads on
// consecutive rows.
__global__ __launch_bounds__(MK_THREADS) void bits_keys_k(uint32_t* bits, int64_t nw, int wpt, const uint32_t* off,
                                                          u64 row_bits, int32_t lo0, int32_t lo1, int nkey,
                                                          bool clear, uint32_t* c0, uint32_t* c1) {
  __shared__ uint32_t stage[MK_THREADS * 32];
  uint32_t p = off[blockIdx.x];
  const u64 base = (u64)blockIdx.x * MK_THREADS * wpt * 32u;
  for (int k = 0; k < wpt; ++k) {
    const int64_t wi = (int64_t)blockIdx.x * MK_THREADS * wpt + (int64_t)k * MK_THREADS + threadIdx.x;
    const uint32_t d = wi < nw ? bits[wi] : 0u;
    uint32_t tot;
    uint32_t q = block_excl_scan<uint32_t>((uint32_t)__popc(d), &tot);
    if (d) {
      if (clear) bits[wi] = 0u;
      for (uint32_t b = d; b; b &= b - 1) stage[q++] = (uint32_t)(k * MK_THREADS + threadIdx.x) * 32u + (uint32_t)(__ffs(b) - 1);
    }
    __syncthreads();
    for (uint32_t r = threadIdx.x; r < tot; r += MK_THREADS) {
      const u64 bi = base + stage[r];
      if (nkey == 2) {
        if (nw <= (int64_t)(0xffffffffu / 32u) && row_bits <= 0xffffffffu) {  // 32-bit division
          const uint32_t q = (uint32_t)bi / (uint32_t)row_bits;
          c0[p + r] = (uint32_t)lo0 + q;
          c1[p + r] = (uint32_t)lo1 + ((uint32_t)bi - q * (uint32_t)row_bits);
        } else {
          c0[p + r] = (uint32_t)lo0 + (uint32_t)(bi / row_bits);
          c1[p + r] = (uint32_t)lo1 + (uint32_t)(bi % row_bits);
        }
      } else {
        c0[p + r] = (uint32_t)lo0 + (uint32_t)bi;
      }
    }
    p += tot;
    __syncthreads();
  }
}

hipError_t bits_keys(uint32_t* bits, int64_t nbits, u64 row_bits, int32_t lo0, int32_t lo1, int nkey, bool clear,
                     uint32_t* c0, uint32_t* c1, uint32_t* total, void* temp, bool write, hipStream_t s) {
  const int64_t nw = (nbits + 31) / 32;
  const int wpt = mk_wpt(nw);
  const int64_t nb = mk_blocks(nw, wpt);
  if (nb == 0) return hipMemsetAsync(total, 0, 4, s);
  uint32_t* cnt = (uint32_t*)temp;
  uint32_t* off = cnt + ((nb + 63) & ~63ll);
  char* stemp = (char*)(off + ((nb + 63) & ~63ll));
  if (!write) {
    bits_count_k<<<(unsigned)nb, MK_THREADS, 0, s>>>(bits, nw, wpt, cnt);
    return scan_exclusive_u32(cnt, off, nb, total, stemp, s);
  }
  bits_keys_k<<<(unsigned)nb, MK_THREADS, 0, s>>>(bits, nw, wpt, off, row_bits, lo0, lo1, nkey, clear, c0, c1);
  return hipGetLastError();
}

size_t bits_list_temp_bytes(int64_t nbits) {
  const int64_t nw = (nbits + 31) / 32, nb = mk_blocks(nw, mk_wpt(nw));
  return (size_t)((nb + 63) & ~63ll) * 8 + scan_temp_bytes(nb) + 256;
}

hipError_t bits_list(uint32_t* bits, int64_t nbits, uint32_t* list, uint32_t* total, void* temp, bool write,
                     hipStream_t s) {
  const int64_t nw = (nbits + 31) / 32;
  const int wpt = mk_wpt(nw);
  const int64_t nb = mk_blocks(nw, wpt);
  if (nb == 0) return hipMemsetAsync(total, 0, 4, s);
  uint32_t* cnt = (uint32_t*)temp;
  uint32_t* off = cnt + ((nb + 63) & ~63ll);
  char* stemp = (char*)(off + ((nb + 63) & ~63ll));
  if (!write) {
    bits_count_k<<<(unsigned)nb, MK_THREADS, 0, s>>>(bits, nw, wpt, cnt);
    return scan_exclusive_u32(cnt, off, nb, total, stemp, s);
  }
  bits_list_k<<<(unsigned)nb, MK_THREADS, 0, s>>>(bits, nw, wpt, off, list);
  return hipGetLastError();
}

__device__ __forceinline__ float lse2(float a, float b) {
  if (a == -INFINITY) return b;
  if (b == -INFINITY) return a;
  const float m = fmaxf(a, b);
  return m + log1pf(expf(-fabsf(a - b)));
}

// Delta rows of batched keyed-table rounds: list positions [bnd[j], bnd[j + 1])
// (read on the device; ~0 as the end: the round overflowed, nothing to do)
// hold the slots the round touched; row i is written for position i.  With
// acc (hashed sum/logsumexp), each slot's accumulator is the round's fold of
// its key: it becomes the row's value, is merged into the slot's full-relation
// value and is reset to the identity; otherwise (min/max) the row takes the
// slot's value.  Each slot appears once in a round's list, so no two threads
// touch one slot.
__global__ void table16_rows_range_k(Slot16* t, u64* acc, const uint32_t* idx, const u64* bnd, int j,
                                     KeyPack kp, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                                     uint32_t* v) {
  const u64 lo = bnd[j], hi = bnd[j + 1];
  if (hi == ~0ull) return;
  const u64 ident = acc ? acc_identity(type, fold_kind) : 0ull;
  for (u64 i = lo + (u64)blockIdx.x * blockDim.x + threadIdx.x; i < hi; i += (u64)gridDim.x * blockDim.x) {
    const uint32_t slot = idx[i];
    const Slot16 s = t[slot];
    uint32_t a, b;
    unpack_key(kp, s.key, &a, &b);
    k0[i] = a;
    if (k1) k1[i] = b;
    if (acc) {
      const uint32_t d = acc_value(acc[slot], type, fold_kind);
      acc[slot] = ident;
      uint32_t r;
      if (fold_kind == FOLD_LSE) r = __float_as_uint(lse2(__uint_as_float(s.val), __uint_as_float(d)));
      else if (type == T_F32) r = __float_as_uint(__fadd_rn(__uint_as_float(s.val), __uint_as_float(d)));
      else r = s.val + d;
      t[slot].val = r;
      v[i] = d;
    } else {
      v[i] = stored_value(s.val, type, fold_kind);
    }
  }
}
hipError_t table16_rows_range(Slot16* t, unsigned long long* acc, const uint32_t* idx, const unsigned long long* bnd,
                              int j, int64_t max_n, KeyPack kp, int type, int fold_kind, uint32_t* k0,
                              uint32_t* k1, uint32_t* v, hipStream_t s) {
  if (max_n <= 0) return hipSuccess;
  table16_rows_range_k<<<grid_for(max_n, 256, 4096), 256, 0, s>>>(t, acc, idx, bnd, j, kp, type, fold_kind, k0,
                                                                 k1, v);
  return hipGetLastError();
}

__global__ void acc_fill_k(u64* acc, int64_t n, int type, int fold_kind) {
  const u64 ident = acc_identity(type, fold_kind);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    acc[i] = ident;
}
hipError_t acc_fill(unsigned long long* acc, int64_t n, int type, int fold_kind, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  acc_fill_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(acc, n, type, fold_kind);
  return hipGetLastError();
}

// Fold a contribution into a full-relation slot this thread owns; returns
// whether the key is new to the relation.
__device__ __forceinline__ bool dense_merge(uint32_t* fval, uint32_t* fpres, uint32_t t, uint32_t x,
                                            int fold_kind, int type) {
  const uint32_t bit = 1u << (t & 31);
  const bool had = atomicOr(&fpres[t >> 5], bit) & bit;
  uint32_t r = x;
  if (had) {
    const uint32_t cur = fval[t];
    if (fold_kind == FOLD_LSE) r = __float_as_uint(lse2(__uint_as_float(cur), __uint_as_float(x)));
    else if (type == T_F32) r = __float_as_uint(__fadd_rn(__uint_as_float(cur), __uint_as_float(x)));
    else r = cur + x;
  }
  fval[t] = r;
  return !had;
}

typedef XL_KARG const DensePullArgs PullArgs;

// Binds S, Z, Y and P1, then e's row e_row; false when the row does not
// derive anything for this key.  FAST: the value is one add/subtract (a.fast).
template <bool FAST>
__device__ __forceinline__ bool pull_bind(PullArgs& a, uint32_t r, uint32_t s, uint32_t y, uint32_t e_row,
                                          Regs& u) {
  const uint32_t z = a.rev.col[a.zcol][e_row];
  const uint32_t zb = z - (uint32_t)a.lo1;
  if (zb >= a.range1) return false;
  const uint32_t zs = zb * a.nrank + r;
  if (!((a.cpres[zs >> 5] >> (zs & 31)) & 1u)) return false;
  if constexpr (FAST) {
    setv(u, a.val_slot, fast_value(a.fast, a.val_type, a.cval[zs], a.rev.col[a.fcol][e_row]));
    return true;
  }
  u = (Regs)(0u);
  setv(u, a.slot_s, s);
  setv(u, a.slot_z, z);
  setv(u, a.slot_y, y);
  if (a.slot_p >= 0) setv(u, a.slot_p, a.cval[zs]);
  if (!bind_cols(a.rev, e_row, u)) return false;
  return run_ops(a, u);
}

// Wave-balanced pull: a wavefront takes 64 listed keys, scans their row
// counts in rev and walks the concatenated row lists 64 rows per step (owner
// found by a six-step search), so consecutive lanes read consecutive rows
// of e.  Per step, the lanes of one key form a run; its contributions are
// folded across the run (segmented shuffles) and merged by the run's last
// lane into the key's running state in LDS: (max m, sum of exp(x - m)) for
// logsumexp, the sum otherwise.  The order is fixed, so the result is
// deterministic.
constexpr int DP_WAVES = 4;
constexpr uint32_t DP_LANE_MAX = 32;  // wavefronts whose keys have at most this many rows: one lane per key

__device__ __forceinline__ float seg_max_scan(float v, int lane, int head) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float t = __shfl_up(v, d, 64);
    if (lane - d >= head) v = fmaxf(v, t);
  }
  return v;
}
template <typename T>
__device__ __forceinline__ T seg_sum_scan(T v, int lane, int head) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const T t = __shfl_up(v, d, 64);
    if (lane - d >= head) v = v + t;
  }
  return v;
}

template <bool FAST>
__global__ __launch_bounds__(DP_WAVES * 64) void dense_pull_k(DensePullArgs by_value) {
  (void)by_value;
  PullArgs& a = *(PullArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ uint32_t s_excl[DP_WAVES][64], s_beg[DP_WAVES][64], s_key[DP_WAVES][64];
  __shared__ uint32_t s_m[DP_WAVES][64], s_acc[DP_WAVES][64], s_any[DP_WAVES][64];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const bool lse = a.fold_kind == FOLD_LSE, f32 = a.val_type == T_F32;
  const int64_t nkeys = a.n_dev ? (int64_t)*a.n_dev : a.n;
  const int64_t nchunks = (nkeys + 63) / 64;
  uint32_t mine = 0, examined = 0;
  for (int64_t chunk = (int64_t)blockIdx.x * DP_WAVES + w; chunk < nchunks; chunk += (int64_t)gridDim.x * DP_WAVES) {
    const int64_t i = chunk * 64 + lane;
    uint32_t t = 0, e0 = 0, deg = 0;
    if (i < nkeys) {
      t = a.list[i];
      const uint32_t kk = t / a.nrank + (uint32_t)a.lo1 - (uint32_t)a.rev.key_lo;
      if (kk < a.rev.key_range) {
        e0 = a.rev.off[kk];
        deg = a.rev.off[kk + 1] - e0;
      }
    }
    const uint32_t incl = wave_incl_scan(deg);
    const uint32_t total = __shfl(incl, 63, 64);
    if (lane == 0) examined += total;
    s_excl[w][lane] = incl - deg;
    s_beg[w][lane] = e0;
    s_key[w][lane] = t;
    s_m[w][lane] = __float_as_uint(-INFINITY);
    s_acc[w][lane] = 0u;
    s_any[w][lane] = 0u;
    wave_lds_sync();
    uint32_t maxdeg = deg;
    for (int k = 32; k > 0; k >>= 1) maxdeg = max(maxdeg, (uint32_t)__shfl_xor(maxdeg, k, 64));
    if (maxdeg <= DP_LANE_MAX) {
      // Short lists: one lane per key, every key's j-th in-edge in step j.
      // Listed keys are ordered by y, so the keys of one y read the delta
      // values of one z at consecutive slots.  Sequential fold per key in
      // index order (online max shift for logsumexp).
      const uint32_t r = t % a.nrank, y = t / a.nrank + (uint32_t)a.lo1;
      float m = -INFINITY, facc = 0.0f;
      uint32_t uacc = 0;
      bool any = false;
      auto fold = [&](uint32_t x) {
        any = true;
        if (lse) {
          const float xv = __uint_as_float(x);
          if (xv > m) {
            facc = (m == -INFINITY ? 0.0f : facc * expf(m - xv)) + 1.0f;
            m = xv;
          } else if (xv != -INFINITY) {
            facc += expf(xv - m);
          }
        } else if (f32) {
          facc = __fadd_rn(facc, __uint_as_float(x));
        } else {
          uacc += x;
        }
      };
      if constexpr (FAST) {
        // the value is one add/subtract of the delta value and a column of
        // e: eight in-edges at a time, each level of loads issued together
        const uint32_t* zc = a.rev.col[a.zcol];
        const uint32_t* wc = a.rev.col[a.fcol];
        for (uint32_t jb = 0; jb < maxdeg; jb += 8) {
          uint32_t zs[8], wv[8], pw[8], cv[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const uint32_t jj = jb + (uint32_t)q;
            const uint32_t zb = jj < deg ? zc[e0 + jj] - (uint32_t)a.lo1 : 0xffffffffu;
            zs[q] = zb < a.range1 ? zb * a.nrank + r : 0xffffffffu;
            wv[q] = jj < deg ? wc[e0 + jj] : 0u;
          }
#pragma unroll
          for (int q = 0; q < 8; ++q) pw[q] = zs[q] != 0xffffffffu ? a.cpres[zs[q] >> 5] : 0u;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const bool pres = zs[q] != 0xffffffffu && ((pw[q] >> (zs[q] & 31)) & 1u);
            cv[q] = pres ? a.cval[zs[q]] : 0u;
            pw[q] = pres;
          }
#pragma unroll
          for (int q = 0; q < 8; ++q)
            if (pw[q]) fold(fast_value(a.fast, a.val_type, cv[q], wv[q]));
        }
      }
      for (uint32_t jj = 0; !FAST && jj < maxdeg; ++jj) {
        if (jj >= deg) continue;
        Regs u;
        if (!pull_bind<FAST>(a, r, a.dict[r], y, e0 + jj, u)) continue;
        const uint32_t x = getv(u, a.val_slot);
        any = true;
        if (lse) {
          const float xv = __uint_as_float(x);
          if (xv > m) {
            facc = (m == -INFINITY ? 0.0f : facc * expf(m - xv)) + 1.0f;
            m = xv;
          } else if (xv != -INFINITY) {
            facc += expf(xv - m);
          }
        } else if (f32) {
          facc = __fadd_rn(facc, __uint_as_float(x));
        } else {
          uacc += x;
        }
      }
      s_m[w][lane] = __float_as_uint(m);
      s_acc[w][lane] = (lse || f32) ? __float_as_uint(facc) : uacc;
      s_any[w][lane] = any ? 1u : 0u;
    }
    for (uint32_t base = 0; maxdeg > DP_LANE_MAX && base < total; base += 64) {
      const uint32_t j = base + (uint32_t)lane;
      const bool act = j < total;
      int q = 0;
#pragma unroll
      for (int step = 32; step > 0; step >>= 1)
        if (s_excl[w][q + step] <= j) q += step;
      bool ok = false;
      uint32_t x = 0;
      if (act) {
        const uint32_t tq = s_key[w][q], r = tq % a.nrank;
        Regs u;
        ok = pull_bind<FAST>(a, r, a.dict[r], tq / a.nrank + (uint32_t)a.lo1, s_beg[w][q] + (j - s_excl[w][q]), u);
        if (ok) x = getv(u, a.val_slot);
      }
      // runs of equal owners among the active lanes
      const int qp = __shfl_up(q, 1, 64);
      const u64 am = __ballot(act);
      const u64 heads = __ballot(act && (lane == 0 || qp != q)) | ~am;
      const int head = 63 - __clzll((long long)(heads & ((2ull << lane) - 1ull)));
      const u64 above = heads & ~((2ull << lane) - 1ull);
      const int tail = above ? __ffsll((long long)above) - 2 : 63;
      const bool is_tail = act && tail == lane;
      const int oks = seg_sum_scan<int>(ok ? 1 : 0, lane, head);
      if (lse) {
        const float xv = ok ? __uint_as_float(x) : -INFINITY;
        const float mrun = __shfl(seg_max_scan(xv, lane, head), tail, 64);
        const float ev = (ok && mrun != -INFINITY) ? expf(xv - mrun) : 0.0f;
        const float srun = seg_sum_scan<float>(ev, lane, head);
        if (is_tail && oks > 0) {
          const float m = __uint_as_float(s_m[w][q]), acc = __uint_as_float(s_acc[w][q]);
          float nm = m, nacc = acc;
          if (mrun != -INFINITY) {
            if (mrun > m) {
              nacc = (m == -INFINITY ? 0.0f : acc * expf(m - mrun)) + srun;
              nm = mrun;
            } else {
              nacc = acc + srun * expf(mrun - m);
            }
          }
          s_m[w][q] = __float_as_uint(nm);
          s_acc[w][q] = __float_as_uint(nacc);
          s_any[w][q] = 1u;
        }
      } else if (f32) {
        const float srun = seg_sum_scan<float>(ok ? __uint_as_float(x) : 0.0f, lane, head);
        if (is_tail && oks > 0) {
          s_acc[w][q] = __float_as_uint(__fadd_rn(__uint_as_float(s_acc[w][q]), srun));
          s_any[w][q] = 1u;
        }
      } else {
        const uint32_t srun = seg_sum_scan<uint32_t>(ok ? x : 0u, lane, head);
        if (is_tail && oks > 0) {
          s_acc[w][q] += srun;
          s_any[w][q] = 1u;
        }
      }
      wave_lds_sync();
    }
    uint32_t out = 0;
    if (i < nkeys) {
      if (lse) {
        const float m = __uint_as_float(s_m[w][lane]);
        out = __float_as_uint(m == -INFINITY ? -INFINITY : m + logf(__uint_as_float(s_acc[w][lane])));
      } else {
        out = s_acc[w][lane];
      }
      if (!s_any[w][lane]) atomicOr(&a.counters[CNT_FATAL], 8ull);  // a marked key always has a contribution
      if (a.k0) {
        const uint32_t r = t % a.nrank, yb = t / a.nrank;
        a.k0[i] = a.dict[r];
        a.k1[i] = yb + (uint32_t)a.lo1;
        a.v[i] = out;
      }
      a.nval[t] = out;
    }
    // Presence bits of the next delta and of the full relation (both laid out
    // like the slots): the listed slots ascend, so the lanes of one presence
    // word are a run; the run ORs its bits together and its last lane sets
    // them with one atomic, whose old word tells every lane of the run
    // whether its slot was present.  The full relation's value is then read
    // and written by its own lane (each slot is listed once).
    {
      const bool act = i < nkeys;
      const uint32_t wd = act ? t >> 5 : 0xffffffffu;
      const uint32_t bit = act ? 1u << (t & 31) : 0u;
      const uint32_t wprev = __shfl_up(wd, 1, 64);
      const u64 heads = __ballot(lane == 0 || wprev != wd);
      const int head = 63 - __clzll((long long)(heads & ((2ull << lane) - 1ull)));
      const u64 above = heads & ~((2ull << lane) - 1ull);
      const int tail = above ? __ffsll((long long)above) - 2 : 63;
      uint32_t run = bit;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(run, d, 64);
        if (lane - d >= head) run |= o;
      }
      uint32_t old = 0;
      if (act && lane == tail) {
        atomicOr(&a.npres[wd], run);
        old = atomicOr(&a.fpres[wd], run);
      }
      old = __shfl(old, tail, 64);
      if (act) {
        const bool had = old & bit;
        uint32_t nv = out;
        if (had) {
          const uint32_t cur = a.fval[t];
          if (lse) nv = __float_as_uint(lse2(__uint_as_float(cur), __uint_as_float(out)));
          else if (f32) nv = __float_as_uint(__fadd_rn(__uint_as_float(cur), __uint_as_float(out)));
          else nv = cur + out;
        }
        a.fval[t] = nv;
        mine += had ? 0u : 1u;
      }
    }
    wave_lds_sync();
  }
  block_count_add(&a.counters[CNT_INSERTED], mine);
  __syncthreads();  // the helper's LDS words are reused by the second call
  block_count_add(&a.counters[CNT_CANDIDATES], examined);
}

// At most as many workgroups as the device keeps resident: each wavefront
// then loops over several chunks of 64 keys, which costs far less than
// launching a short-lived wavefront per chunk.
template <bool FAST>
static hipError_t dense_pull_launch(const DensePullArgs& a, hipStream_t s) {
  int cap = 0;
  hipError_t e = resident_blocks(dense_pull_k<FAST>, DP_WAVES * 64, 0, &cap);
  if (e != hipSuccess) return e;
  dense_pull_k<FAST><<<grid_for((a.n + 63) / 64, DP_WAVES, cap), DP_WAVES * 64, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t dense_pull(const DensePullArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  return a.fast ? dense_pull_launch<true>(a, s) : dense_pull_launch<false>(a, s);
}

// Rows with distinct keys (a folded seed round) into a dense sum/logsumexp
// head: each becomes the current delta value of its slot and is folded into
// the full relation.
__global__ void dense_apply_rows_k(const uint32_t* c0, const uint32_t* c1, const uint32_t* v, int64_t n,
                                   const uint32_t* map, uint32_t map_n, uint32_t range1, uint32_t nrank, KeyPack kp,
                                   int fold_kind, int type, uint32_t* cval, uint32_t* cpres, uint32_t* fval,
                                   uint32_t* fpres, u64* counters) {
  uint32_t mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t k0 = c0[i] - (uint32_t)kp.lo[0], k1 = c1[i] - (uint32_t)kp.lo[1];
    const uint32_t r0 = k0 < map_n ? map[k0] : 0xffffffffu;
    if (r0 == 0xffffffffu || k1 >= range1) {
      atomicOr(&counters[CNT_FATAL], 4ull);
      continue;
    }
    const uint32_t t = k1 * nrank + r0;  // delta and full relation: second-key-major
    cval[t] = v[i];
    atomicOr(&cpres[t >> 5], 1u << (t & 31));
    mine += dense_merge(fval, fpres, t, v[i], fold_kind, type);
  }
  block_count_add(&counters[CNT_INSERTED], mine);
}
hipError_t dense_apply_rows(const uint32_t* c0, const uint32_t* c1, const uint32_t* v, int64_t n, const uint32_t* map,
                            uint32_t map_n, uint32_t range1, uint32_t nrank, KeyPack kp, int fold_kind, int type,
                            uint32_t* cval, uint32_t* cpres, uint32_t* fval, uint32_t* fpres, u64* counters,
                            hipStream_t s) {
  if (n <= 0) return hipSuccess;
  dense_apply_rows_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(c0, c1, v, n, map, map_n, range1, nrank, kp, fold_kind,
                                                            type, cval, cpres, fval, fpres, counters);
  return hipGetLastError();
}

// Marks of a carried-value round whose value is one add or subtract (every
// candidate then yields a value), both rows target-major with wpr words:
// every nonzero word w of z's delta presence row is ORed into word w of the
// mark row of each out-neighbour y of z (mark all zero on entry).  Only the
// delta's words cost more than one load; reading every target's in-edges
// instead took three times as long on the layered DAG.  Word i of clear, an
// array of the same shape (the presence bits the coming pull writes), is
// zeroed by the thread that reads word i of pres.
__global__ void dense_mark_out_k(IndexProbe fwd, int ycol, int32_t lo1, uint32_t range1, uint32_t wpr,
                                 const uint32_t* pres, uint32_t* mark, uint32_t* clear) {
  const int64_t n = (int64_t)range1 * wpr;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t p = pres[i];
    if (clear) clear[i] = 0u;
    if (!p) continue;
    uint32_t zb, wd;
    if (n <= (int64_t)0xffffffffll) {  // 32-bit division
      zb = (uint32_t)i / wpr;
      wd = (uint32_t)i - zb * wpr;
    } else {
      zb = (uint32_t)(i / wpr);
      wd = (uint32_t)(i % wpr);
    }
    const uint32_t kk = zb + (uint32_t)lo1 - (uint32_t)fwd.key_lo;
    if (kk >= fwd.key_range) continue;
    const uint32_t e1 = fwd.off[kk + 1];
    for (uint32_t e = fwd.off[kk]; e < e1; ++e) {
      const uint32_t yb = fwd.col[ycol][e] - (uint32_t)lo1;
      if (yb < range1) atomicOr(&mark[(u64)yb * wpr + wd], p);
    }
  }
}
hipError_t dense_mark_out(const IndexProbe& fwd, int ycol, int32_t lo1, uint32_t range1, uint32_t nrank,
                          const uint32_t* pres, uint32_t* mark, uint32_t* clear, hipStream_t s) {
  const uint32_t wpr = nrank / 32;
  if (range1 == 0 || wpr == 0 || nrank % 32 != 0) return hipErrorInvalidValue;
  if (clear && (clear == pres || clear == mark)) return hipErrorInvalidValue;
  dense_mark_out_k<<<grid_for((int64_t)range1 * wpr, 256, 65536), 256, 0, s>>>(fwd, ycol, lo1, range1, wpr, pres,
                                                                              mark, clear);
  return hipGetLastError();
}


// ============================================================ dense min/max heads, tiled rounds
// Delta rows of a dense min/max head from its delta bits, in slot order
// (rank-major, so grouped by rank and ascending in the second key), clearing
// the bits.  Same word ranges and count pass as bits_keys; the write pass
// stages each step's set bits in LDS so the row writes are coalesced.  With
// roff, it also writes each rank's first row (the rows before the rank's
// first word of wpr words) and, after the last rank, the row total.
__global__ __launch_bounds__(MK_THREADS) void dense_delta_bits_k(uint32_t* chg, int64_t nw, int wpt, const uint32_t* off,
                                                                 uint32_t range1, const uint32_t* vals,
                                                                 const uint32_t* dict, int32_t lo1, int type,
                                                                 int fold_kind, uint32_t* k0, uint32_t* k1,
                                                                 uint32_t* v, uint32_t* roff, uint32_t wpr) {
  __shared__ uint32_t stage[MK_THREADS * 32];
  uint32_t p = off[blockIdx.x];
  const u64 base = (u64)blockIdx.x * MK_THREADS * wpt * 32u;
  for (int k = 0; k < wpt; ++k) {
    const int64_t wi = (int64_t)blockIdx.x * MK_THREADS * wpt + (int64_t)k * MK_THREADS + threadIdx.x;
    const uint32_t d = wi < nw ? chg[wi] : 0u;
    uint32_t tot;
    uint32_t q = block_excl_scan<uint32_t>((uint32_t)__popc(d), &tot);
    if (roff && wi < nw && (uint32_t)wi % wpr == 0u) roff[(uint32_t)wi / wpr] = p + q;
    if (d) {
      chg[wi] = 0u;
      for (uint32_t b = d; b; b &= b - 1)
        stage[q++] = (uint32_t)(k * MK_THREADS + threadIdx.x) * 32u + (uint32_t)(__ffs(b) - 1);
    }
    __syncthreads();
    for (uint32_t r = threadIdx.x; r < tot; r += MK_THREADS) {
      const u64 slot = base + stage[r];
      uint32_t rk, y;
      if (nw <= (int64_t)(0xffffffffu / 32u)) {  // slots below 2^32: 32-bit division
        rk = (uint32_t)slot / range1;
        y = (uint32_t)slot - rk * range1;
      } else {
        rk = (uint32_t)(slot / range1);
        y = (uint32_t)(slot % range1);
      }
      k0[p + r] = dict[rk];
      k1[p + r] = (uint32_t)lo1 + y;
      v[p + r] = stored_value(vals[slot], type, fold_kind);
    }
    p += tot;
    __syncthreads();
  }
  if (roff && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) roff[(uint32_t)(nw / wpr)] = p;
}
hipError_t dense_delta_from_bits(uint32_t* chg, int64_t nslots, uint32_t range1, const uint32_t* vals, const uint32_t* dict,
                            int32_t lo1, int type, int fold_kind, uint32_t* k0, uint32_t* k1, uint32_t* v,
                            uint32_t* roff, uint32_t* total, void* temp, bool write, hipStream_t s) {
  const int64_t nw = (nslots + 31) / 32;
  const uint32_t wpr = range1 / 32;
  if (roff && (range1 % 32 != 0 || wpr == 0)) return hipErrorInvalidValue;
  const int wpt = mk_wpt(nw);
  const int64_t nb = mk_blocks(nw, wpt);
  if (nb == 0) return hipMemsetAsync(total, 0, 4, s);
  uint32_t* cnt = (uint32_t*)temp;
  uint32_t* off = cnt + ((nb + 63) & ~63ll);
  char* stemp = (char*)(off + ((nb + 63) & ~63ll));
  if (!write) {
    bits_count_k<<<(unsigned)nb, MK_THREADS, 0, s>>>(chg, nw, wpt, cnt);
    return scan_exclusive_u32(cnt, off, nb, total, stemp, s);
  }
  dense_delta_bits_k<<<(unsigned)nb, MK_THREADS, 0, s>>>(chg, nw, wpt, off, range1, vals, dict, lo1, type, fold_kind, k0,
                                                         k1, v, roff, wpr);
  return hipGetLastError();
}

typedef XL_KARG const DenseTileArgs TileArgs;
constexpr int DT_THREADS = 1024, DT_WAVES = DT_THREADS / 64;

__global__ __launch_bounds__(DT_THREADS) void dense_min_tile_k(DenseTileArgs by_value) {
  (void)by_value;
  TileArgs& a = *(TileArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  extern __shared__ uint32_t lds[];
  uint32_t* tv = lds;                    // tile values
  uint32_t* tchg = lds + a.tile;         // improved in this round
  uint32_t* tpres = tchg + a.tile / 32;  // presence before the round
  __shared__ uint32_t s_excl[DT_WAVES][64], s_beg[DT_WAVES][64], s_z[DT_WAVES][64], s_d[DT_WAVES][64];
  __shared__ uint32_t s_tc[DT_WAVES];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const uint32_t* ycol = a.idx.col[a.ycol];
  u64 cands = 0;
  uint32_t ins = 0, imp = 0;
  const uint32_t nwork = a.n0 * a.ntiles;
  for (uint32_t b = blockIdx.x; b < nwork; b += gridDim.x) {
    const uint32_t r = b / a.ntiles, t = b % a.ntiles;
    const uint32_t rb = a.roff[r], re = a.roff[r + 1];
    if (rb == re) {  // (uniform) no delta row of this rank: the tile cannot change
      if (a.tcnt && threadIdx.x == 0) a.tcnt[b] = 0u;
      continue;
    }
    const uint32_t y0 = t * a.tile;
    const uint32_t tw = min(a.tile, a.range1 - y0);
    const u64 base = (u64)r * a.range1 + y0;  // first slot (a multiple of 32)
    for (uint32_t i = threadIdx.x; i < tw; i += DT_THREADS) tv[i] = a.vals[base + i];
    for (uint32_t i = threadIdx.x; i < tw / 32; i += DT_THREADS) {
      tchg[i] = 0u;
      tpres[i] = a.pres[base / 32 + i];
    }
    __syncthreads();
    const uint32_t s = a.dict[r];
    for (uint32_t r0 = rb + (uint32_t)w * 64; r0 < re; r0 += DT_WAVES * 64) {
      const uint32_t j = r0 + (uint32_t)lane;
      uint32_t beg = 0, deg = 0, z = 0, d1 = 0;
      if (j < re) {
        z = a.dk1[j];
        d1 = a.dval[j];
        const uint32_t kk = z - (uint32_t)a.idx.key_lo;
        if (kk < a.idx.key_range) {  // only the rows of z whose Y is in this tile
          const u64 o = (u64)t * a.idx.key_range + kk;
          beg = a.toff[o];
          deg = a.toff[o + 1] - beg;
        }
      }
      const uint32_t incl = wave_incl_scan(deg);
      const uint32_t total = __shfl(incl, 63, 64);
      s_excl[w][lane] = incl - deg;
      s_beg[w][lane] = beg;
      s_z[w][lane] = z;
      s_d[w][lane] = d1;
      wave_lds_sync();
      for (uint32_t k0 = 0; k0 < total; k0 += 64) {
        const uint32_t jj = k0 + (uint32_t)lane;
        if (jj < total) {
          int q = 0;
#pragma unroll
          for (int step = 32; step > 0; step >>= 1)
            if (s_excl[w][q + step] <= jj) q += step;
          const uint32_t erow = s_beg[w][q] + (jj - s_excl[w][q]);
          const uint32_t y = ycol[erow];
          const uint32_t yl = y - (uint32_t)a.lo1 - y0;
          if (yl < tw) {  // the tiled index only lists rows of this tile
            ++cands;
            bool ok;
            uint32_t val;
            if (a.fast) {
              val = fast_value(a.fast, a.val_type, s_d[w][q], a.idx.col[a.fcol][erow]);
              ok = true;
            } else {
              Regs u = (Regs)(0u);
              setv(u, a.slot_s, s);
              setv(u, a.slot_z, s_z[w][q]);
              if (a.slot_p >= 0) setv(u, a.slot_p, s_d[w][q]);
              setv(u, a.slot_y, y);
              ok = bind_cols(a.idx, erow, u) && run_ops(a, u);
              val = getv(u, a.val_slot);
            }
            if (ok) {
              const uint32_t enc = fold_encode(val, a.val_type, a.is_max);
              const uint32_t bit = 1u << (yl & 31);
              if (enc < tv[yl]) {
                if (enc < atomicMin(&tv[yl], enc) && !(tchg[yl >> 5] & bit)) atomicOr(&tchg[yl >> 5], bit);
              } else if (enc == 0xffffffffu && !(tpres[yl >> 5] & bit) && !(tchg[yl >> 5] & bit)) {
                atomicOr(&tchg[yl >> 5], bit);  // a first value equal to the empty encoding
              }
            }
          }
        }
      }
      wave_lds_sync();
    }
    __syncthreads();
    // write back the improved slots; new keys get their presence bit
    for (uint32_t i = threadIdx.x; i < tw; i += DT_THREADS)
      if ((tchg[i >> 5] >> (i & 31)) & 1u) a.vals[base + i] = tv[i];
    uint32_t item = 0;
    for (uint32_t i = threadIdx.x; i < tw / 32; i += DT_THREADS) {
      const uint32_t c = tchg[i];
      if (!c) continue;
      a.chg[base / 32 + i] = c;  // the delta bits were cleared when this round's rows were made
      const uint32_t fresh = c & ~tpres[i];
      if (fresh) a.pres[base / 32 + i] = tpres[i] | fresh;
      ins += (uint32_t)__popc(fresh);
      item += (uint32_t)__popc(c);
    }
    imp += item;
    if (a.tcnt) {
      for (int k = 32; k > 0; k >>= 1) item += __shfl_xor(item, k, 64);
      if (lane == 0) s_tc[w] = item;
    }
    __syncthreads();
    if (a.tcnt && threadIdx.x == 0) {  // s_tc is next written after this item's tile loads and barrier
      uint32_t tc = 0;
      for (int i = 0; i < DT_WAVES; ++i) tc += s_tc[i];
      a.tcnt[b] = tc;
    }
  }
  // one atomic per workgroup for each count
  __shared__ u64 s_c[DT_WAVES], s_i[DT_WAVES], s_m[DT_WAVES];
  u64 ci = ins, cm = imp;
  for (int k = 32; k > 0; k >>= 1) {
    cands += __shfl_xor(cands, k, 64);
    ci += __shfl_xor(ci, k, 64);
    cm += __shfl_xor(cm, k, 64);
  }
  if (lane == 0) {
    s_c[w] = cands;
    s_i[w] = ci;
    s_m[w] = cm;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    u64 tc = 0, ti = 0, tm = 0;
    for (int i = 0; i < DT_WAVES; ++i) {
      tc += s_c[i];
      ti += s_i[i];
      tm += s_m[i];
    }
    if (tc) atomicAdd(&a.counters[CNT_CANDIDATES], tc);
    if (ti) atomicAdd(&a.counters[CNT_INSERTED], ti);
    if (tm) atomicAdd(&a.counters[CNT_APPENDED], tm);
  }
}

// Composite sort key of e's rows for the tiled index: (z - zlo) * (ntiles + 1)
// + the tile of y (ntiles for a y outside the head's second-key slots).
// Key of an edge row in the tiled index: tile of Y (ntiles for a Y outside
// the head's range) major, Z minor; or the tile alone (tile_only).
__global__ void tile_keys_k(const uint32_t* zc, const uint32_t* yc, int64_t n, int32_t zlo, int32_t lo1,
                            uint32_t tile, uint32_t ntiles, uint32_t zr, bool tile_only, uint32_t* key) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t tt = min((yc[i] - (uint32_t)lo1) / tile, ntiles);
    key[i] = tile_only ? tt : tt * zr + (zc[i] - (uint32_t)zlo);
  }
}
hipError_t tile_keys(const uint32_t* zc, const uint32_t* yc, int64_t n, int32_t zlo, int32_t lo1, uint32_t tile,
                     uint32_t ntiles, uint32_t zr, bool tile_only, uint32_t* key, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  tile_keys_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(zc, yc, n, zlo, lo1, tile, ntiles, zr, tile_only, key);
  return hipGetLastError();
}

size_t dense_tile_lds_bytes(uint32_t tile) { return ((size_t)tile + 2 * (size_t)(tile / 32)) * 4; }

hipError_t dense_min_tiles(const DenseTileArgs& a, hipStream_t s) {
  const uint32_t nwork = a.n0 * a.ntiles;
  if (nwork == 0) return hipSuccess;
  dense_min_tile_k<<<std::min<uint32_t>(nwork, 65536), DT_THREADS, dense_tile_lds_bytes(a.tile), s>>>(a);
  return hipGetLastError();
}

// Delta rows of a tiled round in one launch, from the per-(rank, tile)
// counts of improved slots that the round's tile kernel wrote: workgroup b
// lists tile b (one delta bit word per thread, the tile's words in one step)
// after summing the counts of the tiles before it itself, so no count pass
// or scan launch precedes it.  Rows come out in slot order (rank-major, as
// the two-pass form writes them) and the delta bits are cleared; workgroup
// b also writes its rank's first row when it holds the rank's first tile,
// and the last one writes roff[n0] and the total.
constexpr int TL_THREADS = 1024;
__global__ __launch_bounds__(TL_THREADS) void tile_delta_rows_k(uint32_t* chg, const uint32_t* tcnt, uint32_t nwork,
                                                                uint32_t ntiles, uint32_t tile, uint32_t range1,
                                                                const uint32_t* vals, const uint32_t* dict,
                                                                int32_t lo1, int type, int fold_kind, uint32_t* k0,
                                                                uint32_t* k1, uint32_t* v, uint32_t* roff,
                                                                uint32_t* total) {
  extern __shared__ uint32_t stage[];  // tile entries: slot offsets within the tile
  __shared__ uint32_t s_w[TL_THREADS / 64];
  const uint32_t b = blockIdx.x, r = b / ntiles, t = b - r * ntiles;
  uint32_t acc = 0;
  for (uint32_t i = threadIdx.x; i < b; i += TL_THREADS) acc += tcnt[i];
  uint32_t p;
  block_excl_scan_u32(acc, &p, s_w);
  const uint32_t own = tcnt[b];
  if (threadIdx.x == 0) {
    if (t == 0) roff[r] = p;
    if (b == nwork - 1) {
      roff[r + 1] = p + own;
      *total = p + own;
    }
  }
  if (own == 0) return;  // the tile kernel wrote no delta bit in this tile
  const uint32_t y0 = t * tile;
  const uint32_t tw = min(tile, range1 - y0);
  const u64 base = (u64)r * range1 + y0;  // a multiple of 32
  const uint32_t nwt = tw / 32;
  const uint32_t key0 = dict[r];
  for (uint32_t w0 = 0; w0 < nwt; w0 += TL_THREADS) {
    const uint32_t wi = w0 + threadIdx.x;
    const uint32_t d = wi < nwt ? chg[base / 32 + wi] : 0u;
    uint32_t tot;
    uint32_t q = block_excl_scan_u32((uint32_t)__popc(d), &tot, s_w);
    if (d) {
      chg[base / 32 + wi] = 0u;
      for (uint32_t bb = d; bb; bb &= bb - 1) stage[q++] = (wi - w0) * 32u + (uint32_t)(__ffs(bb) - 1);
    }
    __syncthreads();
    for (uint32_t e = threadIdx.x; e < tot; e += TL_THREADS) {
      const uint32_t y = w0 * 32u + stage[e];
      k0[p + e] = key0;
      k1[p + e] = (uint32_t)lo1 + y0 + y;
      v[p + e] = stored_value(vals[base + y], type, fold_kind);
    }
    p += tot;
    __syncthreads();
  }
}
hipError_t tile_delta_rows(uint32_t* chg, const uint32_t* tcnt, uint32_t n0, uint32_t ntiles, uint32_t tile,
                           uint32_t range1, const uint32_t* vals, const uint32_t* dict, int32_t lo1, int type,
                           int fold_kind, uint32_t* k0, uint32_t* k1, uint32_t* v, uint32_t* roff, uint32_t* total,
                           hipStream_t s) {
  const uint32_t nwork = n0 * ntiles;
  if (nwork == 0 || nwork > TL_MAX_WORK || tile % 32 != 0 || range1 % 32 != 0 || tile > TL_MAX_TILE)
    return hipErrorInvalidValue;
  const uint32_t stage = std::min<uint32_t>(tile, (uint32_t)TL_THREADS * 32u);
  tile_delta_rows_k<<<nwork, TL_THREADS, (size_t)stage * 4, s>>>(chg, tcnt, nwork, ntiles, tile, range1, vals, dict,
                                                                 lo1, type, fold_kind, k0, k1, v, roff, total);
  return hipGetLastError();
}

// ============================================================ segmented aggregation
template <typename K>
__global__ void seg_heads_k(const K* keys, int64_t n, uint32_t* flag) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    flag[i] = (i == 0) || keys[i] != keys[i - 1];
}
hipError_t seg_heads(const void* keys, int key_bytes, int64_t n, uint32_t* flag, hipStream_t s) {
  if (key_bytes == 4) seg_heads_k<uint32_t><<<grid_for(n, 256, 65536), 256, 0, s>>>((const uint32_t*)keys, n, flag);
  else seg_heads_k<u64><<<grid_for(n, 256, 65536), 256, 0, s>>>((const u64*)keys, n, flag);
  return hipGetLastError();
}

__global__ void seg_starts_k(const uint32_t* flag, const uint32_t* pos, int64_t n,
                             uint32_t* start) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    if (flag[i]) start[pos[i]] = (uint32_t)i;
}
hipError_t seg_starts(const uint32_t* flag, const uint32_t* pos, int64_t n, uint32_t* start,
                      hipStream_t s) {
  seg_starts_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(flag, pos, n, start);
  return hipGetLastError();
}

// One thread folds one key group of the sorted candidates, in sorted order.
// logsumexp is the two-pass max-shifted form: m = max, then m + log(sum exp(x - m)).
template <typename K>
__global__ void seg_reduce_k(const K* keys, const uint32_t* vals, const uint32_t* start,
                             int64_t nseg, int64_t n, KeyPack kp, int type, int fold_kind,
                             uint32_t* k0, uint32_t* k1, uint32_t* v) {
  for (int64_t sg = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; sg < nseg;
       sg += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t b = start[sg];
    const uint32_t e = sg + 1 < nseg ? start[sg + 1] : (uint32_t)n;
    uint32_t out;
    if (fold_kind == FOLD_COUNT) {
      out = e - b;
    } else if (fold_kind == FOLD_LSE) {
      float m = -INFINITY;
      for (uint32_t i = b; i < e; ++i) m = fmaxf(m, __uint_as_float(vals[i]));
      if (m == -INFINITY) {
        out = __float_as_uint(-INFINITY);
      } else {
        float acc = 0.0f;
        for (uint32_t i = b; i < e; ++i) acc += expf(__uint_as_float(vals[i]) - m);
        out = __float_as_uint(m + logf(acc));
      }
    } else if (fold_kind == FOLD_SUM) {
      if (type == T_F32) {
        float acc = 0.0f;
        for (uint32_t i = b; i < e; ++i) acc += __uint_as_float(vals[i]);
        out = __float_as_uint(acc);
      } else {
        uint32_t acc = 0;
        for (uint32_t i = b; i < e; ++i) acc += vals[i];
        out = acc;
      }
    } else {  // FOLD_MIN / FOLD_MAX
      const int is_max = fold_kind == FOLD_MAX;
      uint32_t best = fold_encode(vals[b], type, is_max);
      for (uint32_t i = b + 1; i < e; ++i) best = min(best, fold_encode(vals[i], type, is_max));
      out = fold_decode(best, type, is_max);
    }
    uint32_t a0, a1;
    unpack_key(kp, keys[b], &a0, &a1);
    k0[sg] = a0;
    if (k1) k1[sg] = a1;
    v[sg] = out;
  }
}
hipError_t seg_reduce(const void* keys, int key_bytes, const uint32_t* vals, const uint32_t* start, int64_t nseg,
                      int64_t n, KeyPack kp, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                      uint32_t* v, hipStream_t s) {
  if (nseg <= 0) return hipSuccess;
  if (key_bytes == 4)
    seg_reduce_k<uint32_t><<<grid_for(nseg, 256, 65536), 256, 0, s>>>((const uint32_t*)keys, vals, start, nseg, n,
                                                                      kp, type, fold_kind, k0, k1, v);
  else
    seg_reduce_k<u64><<<grid_for(nseg, 256, 65536), 256, 0, s>>>((const u64*)keys, vals, start, nseg, n, kp, type,
                                                                 fold_kind, k0, k1, v);
  return hipGetLastError();
}

__global__ void agg_merge_k(Slot16* t, u64 mask, const uint32_t* k0, const uint32_t* k1,
                            const uint32_t* v, int64_t n, KeyPack kp, int type, int fold_kind,
                            u64* counters) {
  uint32_t mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    bool ins;
    const u64 s = slot_find_or_insert(t, mask, pack_key(kp, k0[i], k1 ? k1[i] : 0u), &ins,
                                      counters);
    if (s != ~0ull) {
      const uint32_t d = v[i];
      uint32_t r = d;
      if (!ins) {
        const uint32_t cur = t[s].val;
        if (fold_kind == FOLD_LSE) {
          r = __float_as_uint(lse2(__uint_as_float(cur), __uint_as_float(d)));
        } else if (fold_kind == FOLD_SUM) {
          r = type == T_F32 ? __float_as_uint(__fadd_rn(__uint_as_float(cur), __uint_as_float(d)))
                            : cur + d;
        } else if (fold_kind == FOLD_COUNT) {
          r = cur + d;
        }
      }
      t[s].val = r;
    }
    mine += ins;
  }
  block_count_add(&counters[CNT_INSERTED], mine);
}
hipError_t agg_merge(Slot16* t, u64 mask, const uint32_t* k0, const uint32_t* k1,
                     const uint32_t* v, int64_t n, KeyPack kp, int type, int fold_kind,
                     unsigned long long* counters, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  agg_merge_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(t, mask, k0, k1, v, n, kp, type, fold_kind,
                                                     counters);
  return hipGetLastError();
}

// ============================================================ dense set heads
__global__ void bits_set_rows_k(uint32_t* bits, u64 row_bits, const uint32_t* c0,
                                const uint32_t* c1, int64_t n, KeyPack kp) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const u64 key = pack_key(kp, c0[i], c1 ? c1[i] : 0u);
    const u64 b = kp.nkey == 2 ? (key >> kp.shift) * row_bits + (key & ((1ull << kp.shift) - 1ull))
                               : key;
    atomicOr(&bits[b >> 5], 1u << (b & 31));
  }
}
hipError_t bits_set_rows(uint32_t* bits, u64 row_bits, const uint32_t* c0, const uint32_t* c1,
                         int64_t n, KeyPack kp, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  bits_set_rows_k<<<grid_for(n, 256, 8192), 256, 0, s>>>(bits, row_bits, c0, c1, n, kp);
  return hipGetLastError();
}


__global__ void add_u32_k(const uint32_t* in, uint32_t add, uint32_t* out, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = in[i] + add;
}
hipError_t add_u32(const uint32_t* in, uint32_t add, uint32_t* out, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  add_u32_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(in, add, out, n);
  return hipGetLastError();
}

// Count fold of a one-atom body grouped by an indexed column: key x = key_lo + i
// has off[i + 1] - off[i] rows, added to counts[x - head_lo].  One thread per
// key, so no two threads touch one counter; a key with rows outside the head's
// domain raises the fatal counter.
__global__ void index_degree_add_k(const uint32_t* off, uint32_t key_range, int32_t key_lo, int32_t head_lo,
                                   uint32_t head_range, uint32_t* counts, u64* check) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < key_range; i += gridDim.x * blockDim.x) {
    const uint32_t d = off[i + 1] - off[i];
    if (!d) continue;
    const uint32_t hk = (uint32_t)key_lo + i - (uint32_t)head_lo;
    if (hk < head_range)
      counts[hk] += d;
    else
      atomicOr(check, (u64)CHECK_COUNT_DOMAIN);
  }
}
hipError_t index_degree_add(const uint32_t* off, uint32_t key_range, int32_t key_lo, int32_t head_lo,
                            uint32_t head_range, uint32_t* counts, u64* check, hipStream_t s) {
  if (key_range == 0) return hipSuccess;
  index_degree_add_k<<<grid_for(key_range, 256, 65536), 256, 0, s>>>(off, key_range, key_lo, head_lo,
                                                                      head_range, counts, check);
  return hipGetLastError();
}

// *check |= bit when *v differs from expected (one thread).
__global__ void check_eq_k(const uint32_t* v, uint32_t expected, u64* check, u64 bit) {
  if (threadIdx.x == 0 && *v != expected) atomicOr(check, bit);
}
hipError_t check_eq(const uint32_t* v, uint32_t expected, u64* check, u64 bit, hipStream_t s) {
  check_eq_k<<<1, 64, 0, s>>>(v, expected, check, bit);
  return hipGetLastError();
}

}  // namespace k
}  // namespace xlh
