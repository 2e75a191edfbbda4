// Frontier form of closure-shaped strata on gfx950: one workgroup per first
// key per round, its bitmap row staged in LDS (see FrontierArgs), and the
// kernels that move between row lists and bitmap rows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_util.h"
#include "kernels.h"

namespace xlh {
namespace k {

// Frontier round (see FrontierArgs).  LDS holds bitmap row x before and after
// the round plus a piece of the delta row decoded into a list of Z values;
// each step decodes up to 512 words, cut so the list holds at most FR_ZCAP
// values (a sparse row takes one step).  The wave-balanced expansion of the
// Z list is the same as in the generic stage kernel.  A plain LDS test
// precedes each LDS atomic because most produced tuples are already known.
constexpr int FR_THREADS = 256;
constexpr int FR_WAVES = FR_THREADS / 64;
constexpr uint32_t FR_ZCAP = 4096;  // Z (or Y) values decoded per step
constexpr int FR_PROBE = 4;         // in-edges a pulling lane loads at once


// Workgroup totals of two per-thread counts (one barrier pair).
__device__ __forceinline__ void block_sum2(uint32_t x, uint32_t y, uint32_t* tx, uint32_t* ty, uint32_t* s_w,
                                           uint32_t* s_w2) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  for (int k = 32; k > 0; k >>= 1) {
    x += __shfl_xor(x, k, 64);
    y += __shfl_xor(y, k, 64);
  }
  if (lane == 0) {
    s_w[w] = x;
    s_w2[w] = y;
  }
  __syncthreads();
  uint32_t a = 0, b = 0;
  for (int k = 0; k < (int)(blockDim.x >> 6); ++k) {
    a += s_w[k];
    b += s_w2[k];
  }
  __syncthreads();
  *tx = a;
  *ty = b;
}

__global__ __launch_bounds__(FR_THREADS) void frontier_round_k(FrontierArgs a) {
  extern __shared__ uint32_t lds[];
  uint32_t* old_row = lds;
  uint32_t* new_row = lds + a.row_words;
  uint32_t* f_row = lds + 2 * a.row_words;  // this round's delta row of x
  __shared__ uint32_t zlist[FR_ZCAP];
  __shared__ uint32_t s_excl[FR_WAVES][64];
  __shared__ uint32_t s_beg[FR_WAVES][64];
  __shared__ uint32_t s_w[FR_WAVES], s_w2[FR_WAVES], s_cut[2];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const uint32_t W = a.row_words;
  const uint32_t* ycol = a.idx.col[a.ybind_col];
  const uint32_t* zcol = a.rev.col[a.rev_zcol];
  u64 cands = 0, news = 0;  // cands: this lane's share; news: workgroup total
  for (int64_t sg = blockIdx.x; sg < a.nseg; sg += gridDim.x) {
    if (a.in_cnt[sg] == 0) {  // x gained nothing last round: its delta row is empty
      if (threadIdx.x == 0) a.out_cnt[sg] = 0;
      continue;
    }
    const uint32_t x = a.x[sg];
    uint32_t* grow = a.bits + (u64)(x - (uint32_t)a.lo0) * W;
    const uint32_t* drow = a.in_diff + (u64)sg * W;
    uint32_t nd = 0, nu = 0;
    for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) {
      const uint32_t v = grow[i], f = drow[i];
      old_row[i] = v;
      new_row[i] = v;
      f_row[i] = f;
      nd += __popc(f);
      if (a.pull_ratio) nu += __popc(~v & a.hasin[i]);
    }
    uint32_t tnd, tnu;
    block_sum2(nd, nu, &tnd, &tnu, s_w, s_w2);
    const bool pull = a.pull_ratio && (u64)a.pull_ratio * tnd >= (u64)tnu;
    for (uint32_t cb = 0; cb < W;) {
      // Decode words [cb, cb + 512), two per thread, cut after the last
      // thread whose values still fit the list: push takes the delta's Z
      // values, pull the unreached Y values that have an in-edge.
      const uint32_t w0 = cb + 2u * threadIdx.x;
      uint32_t d0 = 0, d1 = 0;
      if (w0 < W) d0 = pull ? (~old_row[w0] & a.hasin[w0]) : f_row[w0];
      if (w0 + 1 < W) d1 = pull ? (~old_row[w0 + 1] & a.hasin[w0 + 1]) : f_row[w0 + 1];
      const uint32_t c = __popc(d0) + __popc(d1);
      uint32_t tot;
      uint32_t pos = block_excl_scan_u32(c, &tot, s_w);
      if (pos + c <= FR_ZCAP) {
        for (uint32_t bits = d0; bits; bits &= bits - 1)
          zlist[pos++] = (uint32_t)a.lo1 + w0 * 32u + (uint32_t)(__ffs(bits) - 1);
        for (uint32_t bits = d1; bits; bits &= bits - 1)
          zlist[pos++] = (uint32_t)a.lo1 + (w0 + 1) * 32u + (uint32_t)(__ffs(bits) - 1);
      } else if (pos <= FR_ZCAP) {  // the first thread that does not fit
        s_cut[0] = pos;
        s_cut[1] = 2u * threadIdx.x;
      }
      __syncthreads();
      const uint32_t nz = tot <= FR_ZCAP ? tot : s_cut[0];
      cb += tot <= FR_ZCAP ? 2u * FR_THREADS : s_cut[1];
      if (pull) {
        // One lane per unreached Y: test its in-edges FR_PROBE at a time
        // (independent loads) until one comes from the delta.
        for (uint32_t r = threadIdx.x; r < nz; r += FR_THREADS) {
          const uint32_t y = zlist[r];
          const uint32_t kk = y - (uint32_t)a.rev.key_lo;
          if (kk >= a.rev.key_range) continue;
          const uint32_t e1 = a.rev.off[kk + 1];
          bool hit = false;
          for (uint32_t e = a.rev.off[kk]; e < e1 && !hit; e += FR_PROBE) {
            uint32_t zz[FR_PROBE];
#pragma unroll
            for (int u = 0; u < FR_PROBE; ++u) zz[u] = e + u < e1 ? zcol[e + u] - (uint32_t)a.lo1 : 0xffffffffu;
            // count the in-edges a scan in order would examine: up to the
            // first one from the delta (the rest of the batch is wasted load)
            const uint32_t nb = e1 - e < (uint32_t)FR_PROBE ? e1 - e : (uint32_t)FR_PROBE;
#pragma unroll
            for (int u = 0; u < FR_PROBE; ++u) {
              if (hit || (uint32_t)u >= nb) continue;
              ++cands;
              hit = zz[u] < W * 32u && ((f_row[zz[u] >> 5] >> (zz[u] & 31)) & 1u);
            }
          }
          if (hit) {
            const uint32_t yb = y - (uint32_t)a.lo1;
            atomicOr(&new_row[yb >> 5], 1u << (yb & 31));
          }
        }
        __syncthreads();
        continue;
      }
      for (uint32_t r0 = (uint32_t)w * 64; r0 < nz; r0 += FR_WAVES * 64) {
        const uint32_t r = r0 + lane;
        uint32_t beg = 0, deg = 0;
        if (r < nz) {
          const uint32_t kk = zlist[r] - (uint32_t)a.idx.key_lo;
          if (kk < a.idx.key_range) {
            beg = a.idx.off[kk];
            deg = a.idx.off[kk + 1] - beg;
          }
        }
        // Rows with at least 64 matches are walked by the whole wavefront, one
        // row at a time, lane = item: no owner search at all.  The remaining
        // small rows share 64-item steps through a scan and a six-step search.
        const bool big = deg >= 64;
        u64 bigm = __ballot(big);
        const uint32_t sdeg = big ? 0u : deg;
        const uint32_t incl = wave_incl_scan(sdeg);
        const uint32_t total = __shfl(incl, 63, 64);
        s_excl[w][lane] = incl - sdeg;
        s_beg[w][lane] = beg;
        wave_lds_sync();
        if (lane == 0) cands += total;
        while (bigm) {
          const int rb = __ffsll((long long)bigm) - 1;
          bigm &= bigm - 1;
          const uint32_t bb = __shfl(beg, rb, 64), bd = __shfl(deg, rb, 64);
          if (lane == 0) cands += bd;
          for (uint32_t k0 = 0; k0 < bd; k0 += 256) {
            uint32_t y[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const uint32_t k = k0 + 64 * u + lane;
              y[u] = k < bd ? ycol[bb + k] - (uint32_t)a.lo1 : 0xffffffffu;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              if (y[u] != 0xffffffffu) {
                const uint32_t bit = 1u << (y[u] & 31);
                if (!(new_row[y[u] >> 5] & bit)) atomicOr(&new_row[y[u] >> 5], bit);
              }
            }
          }
        }
        for (uint32_t b0 = 0; b0 < total; b0 += 64) {
          const uint32_t j = b0 + lane;
          if (j < total) {
            int q = 0;
#pragma unroll
            for (int step = 32; step > 0; step >>= 1)
              if (s_excl[w][q + step] <= j) q += step;
            const uint32_t y = ycol[s_beg[w][q] + (j - s_excl[w][q])] - (uint32_t)a.lo1;
            const uint32_t bit = 1u << (y & 31);
            if (!(new_row[y >> 5] & bit)) atomicOr(&new_row[y >> 5], bit);
          }
        }
        wave_lds_sync();
      }
      __syncthreads();
    }
    // next delta row = new bits; write back the changed words of row x
    uint32_t nnew = 0;
    uint32_t* orow = a.out_diff + (u64)sg * W;
    for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) {
      const uint32_t nv = new_row[i];
      const uint32_t dd = nv & ~old_row[i];
      orow[i] = dd;
      if (dd) {
        grow[i] = nv;
        nnew += __popc(dd);
      }
    }
    uint32_t tnew;
    block_excl_scan_u32(nnew, &tnew, s_w);
    if (threadIdx.x == 0) a.out_cnt[sg] = tnew;
    news += tnew;
  }
  // one atomic per workgroup for each total
  for (int k = 32; k > 0; k >>= 1) cands += __shfl_xor(cands, k, 64);
  __shared__ u64 s_c[FR_WAVES];
  if (lane == 0) s_c[w] = cands;
  __syncthreads();
  if (threadIdx.x == 0) {
    u64 t = 0;
    for (int i = 0; i < FR_WAVES; ++i) t += s_c[i];
    if (t) atomicAdd(&a.counters[CNT_CANDIDATES], t);
    if (news) atomicAdd(&a.counters[CNT_APPENDED], news);
  }
}

hipError_t frontier_round(const FrontierArgs& a, hipStream_t s) {
  if (a.nseg <= 0) return hipSuccess;
  const size_t lds = (size_t)a.row_words * 3 * sizeof(uint32_t);
  const unsigned grid = (unsigned)std::min<int64_t>(a.nseg, 4096);
  frontier_round_k<<<grid, FR_THREADS, lds, s>>>(a);
  return hipGetLastError();
}


// Number of set bits in each bitmap row.
__global__ __launch_bounds__(256) void row_popcount_k(const uint32_t* bits, int64_t nrows,
                                                      uint32_t row_words, uint32_t* cnt) {
  __shared__ uint32_t s_w[4];
  for (int64_t r = blockIdx.x; r < nrows; r += gridDim.x) {
    const uint32_t* row = bits + (u64)r * row_words;
    uint32_t c = 0;
    for (uint32_t i = threadIdx.x; i < row_words; i += 256) c += __popc(row[i]);
    uint32_t tot;
    block_excl_scan_u32(c, &tot, s_w);
    if (threadIdx.x == 0) cnt[r] = tot;
  }
}
hipError_t row_popcount(const uint32_t* bits, int64_t nrows, uint32_t row_words, uint32_t* cnt,
                        hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  row_popcount_k<<<(unsigned)std::min<int64_t>(nrows, 1 << 16), 256, 0, s>>>(bits, nrows, row_words, cnt);
  return hipGetLastError();
}

// Relation rows (x, y) of every set bit, in ascending (x, y) order: bitmap row
// r holds x = lo0 + r and starts at off[r].  Each chunk of 256 words is
// decoded into LDS first so the column writes are coalesced.
__global__ __launch_bounds__(256) void bits_to_rows_k(const uint32_t* bits, int64_t nrows,
                                                      uint32_t row_words, const uint32_t* off,
                                                      int32_t lo0, int32_t lo1, uint32_t* c0,
                                                      uint32_t* c1) {
  __shared__ uint32_t stage[256 * 32];
  __shared__ uint32_t s_w[4];
  for (int64_t r = blockIdx.x; r < nrows; r += gridDim.x) {
    const uint32_t* row = bits + (u64)r * row_words;
    u64 out = off[r];
    const uint32_t x = (uint32_t)lo0 + (uint32_t)r;
    for (uint32_t cb = 0; cb < row_words; cb += 256) {
      const uint32_t wi = cb + threadIdx.x;
      const uint32_t d = wi < row_words ? row[wi] : 0u;
      uint32_t n;
      uint32_t pos = block_excl_scan_u32(__popc(d), &n, s_w);
      for (uint32_t b = d; b; b &= b - 1) stage[pos++] = (uint32_t)lo1 + wi * 32u + (uint32_t)(__ffs(b) - 1);
      __syncthreads();
      for (uint32_t i = threadIdx.x; i < n; i += 256) {
        c0[out + i] = x;
        c1[out + i] = stage[i];
      }
      out += n;
      __syncthreads();
    }
  }
}
hipError_t bits_to_rows(const uint32_t* bits, int64_t nrows, uint32_t row_words, const uint32_t* off,
                        int32_t lo0, int32_t lo1, uint32_t* c0, uint32_t* c1, hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  bits_to_rows_k<<<(unsigned)std::min<int64_t>(nrows, 1 << 16), 256, 0, s>>>(bits, nrows, row_words, off,
                                                                            lo0, lo1, c0, c1);
  return hipGetLastError();
}

// out row sg = bitmap row (x[sg] - lo0), row_words words each.
__global__ void gather_rows_k(const uint32_t* bits, uint32_t row_words, const uint32_t* x, int32_t lo0,
                              int64_t nseg, uint32_t* out) {
  for (int64_t sg = blockIdx.x; sg < nseg; sg += gridDim.x) {
    const uint32_t* src = bits + (u64)(x[sg] - (uint32_t)lo0) * row_words;
    uint32_t* dst = out + (u64)sg * row_words;
    for (uint32_t i = threadIdx.x; i < row_words; i += blockDim.x) dst[i] = src[i];
  }
}
hipError_t gather_rows(const uint32_t* bits, uint32_t row_words, const uint32_t* x, int32_t lo0, int64_t nseg,
                       uint32_t* out, hipStream_t s) {
  if (nseg <= 0) return hipSuccess;
  gather_rows_k<<<(unsigned)std::min<int64_t>(nseg, 1 << 16), 256, 0, s>>>(bits, row_words, x, lo0, nseg, out);
  return hipGetLastError();
}

// hasin bit (y - lo1) for y in [lo1, lo1 + 32 * words): y has an in-edge in
// the index of e by its Y column.
__global__ void hasin_bits_k(IndexProbe rev, int32_t lo1, uint32_t words, uint32_t* out) {
  for (uint32_t wi = blockIdx.x * blockDim.x + threadIdx.x; wi < words; wi += gridDim.x * blockDim.x) {
    uint32_t m = 0;
    for (int b = 0; b < 32; ++b) {
      const uint32_t kk = (uint32_t)lo1 + wi * 32u + (uint32_t)b - (uint32_t)rev.key_lo;
      if (kk < rev.key_range && rev.off[kk + 1] > rev.off[kk]) m |= 1u << b;
    }
    out[wi] = m;
  }
}
hipError_t hasin_bits(const IndexProbe& rev, int32_t lo1, uint32_t words, uint32_t* out, hipStream_t s) {
  hasin_bits_k<<<grid_for(words, 256, 4096), 256, 0, s>>>(rev, lo1, words, out);
  return hipGetLastError();
}

}  // namespace k
}  // namespace xlh
