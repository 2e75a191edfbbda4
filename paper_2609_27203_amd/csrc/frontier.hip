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
constexpr int FR_PROBE = 4;         // in-edges a pulling lane loads at once: one aligned 16-B block
constexpr int FR_UNROLL = 8;        // first in-edges a pulling lane tests together
constexpr uint32_t FR_LONG = 64;    // longer remaining in-edge lists are scanned by the whole wave
// A round pulls only while the delta holds at least 1/FR_PULL_BETA of the
// row's bits (besides pull_ratio * |delta| >= unreached targets): a small
// delta pushes, as in direction-optimizing breadth-first search, since a
// pull would re-test the in-edges of targets it cannot reach.
constexpr uint32_t FR_PULL_BETA = 64;


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

// LDS of one frontier workgroup besides the three bitmap rows.
struct FrontierShared {
  uint32_t zlist[FR_ZCAP];
  uint32_t s_excl[FR_WAVES][64];
  uint32_t s_beg[FR_WAVES][64];
  uint32_t s_w[FR_WAVES], s_w2[FR_WAVES], s_cut[2];
  uint32_t s_sg;
};

// One round of row x in LDS: every Y reachable in one step from the delta
// row f_row (push: expand each delta Z through the index; pull: test each
// unreached Y's in-edges against f_row) is set in new_row, which starts as a
// copy of old_row.  Ends with a workgroup barrier.
__device__ __forceinline__ void frontier_expand(const FrontierArgs& a, const uint32_t* old_row, uint32_t* new_row,
                                                const uint32_t* f_row, bool pull, FrontierShared& L, u64& cands) {
  uint32_t* zlist = L.zlist;
  auto& s_excl = L.s_excl;
  auto& s_beg = L.s_beg;
  uint32_t* s_w = L.s_w;
  uint32_t* s_cut = L.s_cut;
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const uint32_t W = a.row_words;
  const uint32_t* ycol = a.idx.col[a.ybind_col];
  const uint32_t* zcol = a.rev.col[a.rev_zcol];
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
      // Phase A: every lane tests the first in-edge of FR_UNROLL unreached
      // Y values, read from the dense first-row array with the loads issued
      // together.  The Y values whose first in-edge misses the delta are
      // compacted into the list slots this wavefront owns (slot m of wave w
      // is 256 * (m / 64) + 64 * w + m % 64; a miss is never written past
      // the slot its own Y was read from, so no unread value is lost).
      uint32_t nmiss = 0;
      for (uint32_t b = 0; b < nz; b += FR_THREADS * FR_UNROLL) {
        uint32_t yv[FR_UNROLL], zv[FR_UNROLL];
#pragma unroll
        for (int j = 0; j < FR_UNROLL; ++j) {
          const uint32_t pos = b + (uint32_t)j * FR_THREADS + threadIdx.x;
          yv[j] = pos < nz ? zlist[pos] : 0u;
        }
#pragma unroll
        for (int j = 0; j < FR_UNROLL; ++j) {
          const uint32_t pos = b + (uint32_t)j * FR_THREADS + threadIdx.x;
          const uint32_t kk = yv[j] - (uint32_t)a.rev.key_lo;
          zv[j] = pos < nz && kk < a.rev.key_range ? a.rev_first[kk] : 0u;
        }
#pragma unroll
        for (int j = 0; j < FR_UNROLL; ++j) {
          const uint32_t pos = b + (uint32_t)j * FR_THREADS + threadIdx.x;
          const uint32_t kk = yv[j] - (uint32_t)a.rev.key_lo;
          bool miss = false;
          if (pos < nz && kk < a.rev.key_range) {  // every listed Y has an in-edge
            ++cands;
            const uint32_t z0 = zv[j] - (uint32_t)a.lo1;
            if (z0 < W * 32u && ((f_row[z0 >> 5] >> (z0 & 31)) & 1u)) {
              const uint32_t yb = yv[j] - (uint32_t)a.lo1;
              atomicOr(&new_row[yb >> 5], 1u << (yb & 31));
            } else {
              miss = true;
            }
          }
          const u64 bm = __ballot(miss);
          if (miss) {
            const uint32_t m = nmiss + (uint32_t)__popcll(bm & lanemask_lt());
            zlist[(m >> 6) * FR_THREADS + (uint32_t)w * 64 + (m & 63)] = yv[j];
          }
          nmiss += (uint32_t)__popcll(bm);
        }
      }
      wave_lds_sync();
      // Phase B, per wavefront over its misses: one lane per Y tests the
      // remaining in-edges one aligned 16-B block at a time (index columns
      // are 256-B aligned arena blocks rounded up to 256 B, so a block never
      // leaves the column's allocation) until one comes from the delta;
      // lists with more than FR_LONG left are scanned by the whole
      // wavefront, 64 in-edges per step, stopping at the first hit.  The
      // candidates counted are the in-edges a scan in order examines, up to
      // the first hit (the rest of a block or step is wasted load).
      for (uint32_t m0 = 0; m0 < nmiss; m0 += 64) {
        const uint32_t m = m0 + lane;
        uint32_t y = 0, e = 0, e1 = 0;
        if (m < nmiss) {
          y = zlist[(m >> 6) * FR_THREADS + (uint32_t)w * 64 + (m & 63)];
          const uint32_t kk = y - (uint32_t)a.rev.key_lo;
          e = a.rev.off[kk] + 1;
          e1 = a.rev.off[kk + 1];
        }
        const bool longl = e1 > e + FR_LONG;
        u64 lm = __ballot(longl);
        bool hit = false;
        if (!longl) {
          while (e < e1 && !hit) {
            const uint32_t base = e & ~(uint32_t)(FR_PROBE - 1);
            const uint4 q = *reinterpret_cast<const uint4*>(zcol + base);
            const uint32_t zz[FR_PROBE] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int u = 0; u < FR_PROBE; ++u) {
              const uint32_t i = base + (uint32_t)u;
              if (hit || i < e || i >= e1) continue;
              ++cands;
              const uint32_t zb = zz[u] - (uint32_t)a.lo1;
              hit = zb < W * 32u && ((f_row[zb >> 5] >> (zb & 31)) & 1u);
            }
            e = base + FR_PROBE;
          }
        }
        if (hit) {
          const uint32_t yb = y - (uint32_t)a.lo1;
          atomicOr(&new_row[yb >> 5], 1u << (yb & 31));
        }
        while (lm) {
          const int rb = __ffsll((long long)lm) - 1;
          lm &= lm - 1;
          const uint32_t by = __shfl(y, rb, 64), bb = __shfl(e, rb, 64), be = __shfl(e1, rb, 64);
          for (uint32_t k0 = bb; k0 < be; k0 += 64) {
            const uint32_t i = k0 + lane;
            bool h = false;
            if (i < be) {
              const uint32_t zb = zcol[i] - (uint32_t)a.lo1;
              h = zb < W * 32u && ((f_row[zb >> 5] >> (zb & 31)) & 1u);
            }
            const u64 hm = __ballot(h);
            if (hm) {
              if (lane == 0) {
                cands += (u64)__ffsll((long long)hm);
                const uint32_t yb = by - (uint32_t)a.lo1;
                atomicOr(&new_row[yb >> 5], 1u << (yb & 31));
              }
              break;
            }
            if (lane == 0) cands += be - k0 < 64u ? be - k0 : 64u;
          }
        }
      }
      __syncthreads();
      continue;
    }
    // list positions interleaved over the wavefronts (lane l of wavefront w
    // takes j0 + 4 l + w), so a short list still reaches all of them
    for (uint32_t j0 = 0; j0 < nz; j0 += FR_WAVES * 64) {
      const uint32_t r = j0 + (uint32_t)lane * FR_WAVES + (uint32_t)w;
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
}

__global__ __launch_bounds__(FR_THREADS) void frontier_round_k(FrontierArgs a) {
  extern __shared__ uint32_t lds[];
  uint32_t* old_row = lds;
  uint32_t* new_row = lds + a.row_words;
  uint32_t* f_row = lds + 2 * a.row_words;  // this round's delta row of x
  __shared__ FrontierShared L;
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const uint32_t W = a.row_words;
  u64 cands = 0, news = 0;  // cands: this lane's share; news: workgroup total
  uint32_t* s_w = L.s_w;
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
    block_sum2(nd, nu, &tnd, &tnu, L.s_w, L.s_w2);
    const bool pull = a.pull_ratio && (u64)a.pull_ratio * tnd >= (u64)tnu &&
                      (u64)tnd * FR_PULL_BETA >= (u64)W * 32u;
    frontier_expand(a, old_row, new_row, f_row, pull, L, cands);
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

// Resident form (see FrontierArgs): the rounds of one first key x depend only
// on x's own row and the fixed index, so a workgroup runs them back to back
// with the row, the delta and the next row in LDS and no launch, host read or
// HBM round trip in between.
__global__ __launch_bounds__(FR_THREADS) void frontier_resident_k(FrontierArgs a) {
  extern __shared__ uint32_t lds[];
  uint32_t* old_row = lds;
  uint32_t* new_row = lds + a.row_words;
  uint32_t* f_row = lds + 2 * a.row_words;
  __shared__ FrontierShared L;
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const uint32_t W = a.row_words;
  u64 cands = 0, news = 0;
  for (;;) {
    if (threadIdx.x == 0) L.s_sg = atomicAdd(a.queue, 1u);
    __syncthreads();
    const uint32_t sg = L.s_sg;
    if ((int64_t)sg >= a.nseg) break;
    if (a.in_cnt && a.in_cnt[sg] == 0) {  // keeps the barrier above between two reads of s_sg
      __syncthreads();
      continue;
    }
    const uint32_t x = a.x ? a.x[sg] : (uint32_t)a.lo0 + sg;
    uint32_t* grow = a.bits + (u64)(x - (uint32_t)a.lo0) * W;
    const uint32_t* drow = a.in_diff + (u64)sg * W;
    uint32_t nd = 0, nu = 0, tnd, tnu;
    for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) {
      const uint32_t f = drow[i];
      f_row[i] = f;
      nd += __popc(f);
    }
    block_sum2(nd, 0u, &tnd, &tnu, L.s_w, L.s_w2);
    if (tnd == 0) continue;  // no delta: the row stays as it is (block_sum2 ended with a barrier)
    for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) {
      const uint32_t v = grow[i];
      old_row[i] = v;
      new_row[i] = v;
      if (a.pull_ratio) nu += __popc(~v & a.hasin[i]);
    }
    block_sum2(nu, 0u, &tnu, &nd, L.s_w, L.s_w2);
    uint32_t round = 0;
    while (tnd > 0) {
      if (round >= a.max_rounds) {
        if (threadIdx.x == 0) atomicOr(a.overflow, 1u);
        break;
      }
      if (a.pull_ratio && tnu == 0) {  // every target with an in-edge is reached:
        ++round;                       // this round finds nothing and ends x's passes
        break;
      }
      const bool pull = a.pull_ratio && (u64)a.pull_ratio * tnd >= (u64)tnu &&
                        (u64)tnd * FR_PULL_BETA >= (u64)W * 32u;
      frontier_expand(a, old_row, new_row, f_row, pull, L, cands);
      // the new bits become the next delta; the row takes them
      nd = 0;
      nu = 0;
      for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) {
        const uint32_t nv = new_row[i];
        const uint32_t dd = nv & ~old_row[i];
        f_row[i] = dd;
        old_row[i] = nv;
        nd += __popc(dd);
        if (a.pull_ratio) nu += __popc(~nv & a.hasin[i]);
      }
      block_sum2(nd, nu, &tnd, &tnu, L.s_w, L.s_w2);
      if (threadIdx.x == 0 && tnd) atomicAdd(&a.round_new[round < a.round_slots ? round : a.round_slots - 1], (u64)tnd);
      news += tnd;
      ++round;
    }
    if (threadIdx.x == 0 && round) atomicMax(a.max_round, round);
    if (round)
      for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) grow[i] = old_row[i];
    __syncthreads();  // the row is written before LDS takes the next key
  }
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

hipError_t frontier_resident(const FrontierArgs& a, unsigned grid, hipStream_t s) {
  if (a.nseg <= 0) return hipSuccess;
  if (!a.queue || !a.max_round || !a.overflow || !a.round_new || a.round_slots == 0) return hipErrorInvalidValue;
  const size_t lds = (size_t)a.row_words * 3 * sizeof(uint32_t);
  if (grid == 0) {
    int blocks = 0;
    const hipError_t e = resident_blocks(frontier_resident_k, FR_THREADS, lds, &blocks);
    if (e != hipSuccess) return e;
    grid = (unsigned)blocks;
  }
  grid = (unsigned)std::min<int64_t>(grid, a.nseg);
  frontier_resident_k<<<grid, FR_THREADS, lds, s>>>(a);
  return hipGetLastError();
}

// Gathered round (see GatherArgs).  Per head row X with a flagged delta row
// among its A values: X's row is copied into LDS twice (before, after); each
// such delta row is pushed through e2 into the after row by the frontier
// expansion (its B bits decoded into a list, their Y lists walked wave-
// balanced, each Y tested and set in LDS); then the words that differ are
// written to the head row and their new bits to X's next delta row.
__global__ __launch_bounds__(FR_THREADS) void gather_round_k(GatherArgs g) {
  extern __shared__ uint32_t lds[];
  const uint32_t W = g.row_words;
  uint32_t* before = lds;
  uint32_t* after = lds + W;
  __shared__ FrontierShared L;
  __shared__ uint32_t s_any, s_new;
  const int lane = lane_id();
  u64 cands = 0, fresh = 0;
  const uint32_t* acol = g.e1.col[g.e1_acol];
  // rows in a grid-stride loop: most rows have no delta in a given round, and
  // a shared work counter would serialize those cheap visits on one address
  for (int64_t xr64 = blockIdx.x; xr64 < g.range0; xr64 += gridDim.x) {
    const uint32_t xr = (uint32_t)xr64;
    if (threadIdx.x == 0) {
      s_any = 0u;
      s_new = 0u;
    }
    __syncthreads();
    const uint32_t kk = (uint32_t)g.lo0 + xr - (uint32_t)g.e1.key_lo;
    uint32_t b1 = 0, n1 = 0;
    if (kk < g.e1.key_range) {
      b1 = g.e1.off[kk];
      n1 = g.e1.off[kk + 1] - b1;
    }
    // does any A of X have a delta row?
    for (uint32_t q = threadIdx.x; q < n1; q += FR_THREADS) {
      const uint32_t ar = acol[b1 + q] - (uint32_t)g.lo0;
      if ((int64_t)ar < g.range0 && g.in_flag[ar]) s_any = 1u;
    }
    __syncthreads();
    if (!s_any) {
      __syncthreads();  // the shared words are rewritten at the top
      continue;
    }
    uint32_t* hrow = g.bits + (u64)xr * W;
    for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) before[i] = after[i] = hrow[i];
    __syncthreads();
    for (uint32_t q = 0; q < n1; ++q) {
      const uint32_t ar = acol[b1 + q] - (uint32_t)g.lo0;
      if ((int64_t)ar >= g.range0 || !g.in_flag[ar]) continue;  // (uniform)
      frontier_expand(g.push, before, after, g.in_bits + (u64)ar * W, false, L, cands);
    }
    uint32_t* orow = g.out_bits + (u64)xr * W;
    uint32_t nb = 0;
    for (uint32_t i = threadIdx.x; i < W; i += FR_THREADS) {
      const uint32_t nw = after[i] & ~before[i];
      if (nw) {
        hrow[i] = after[i];
        orow[i] = nw;
        nb += (uint32_t)__popc(nw);
      }
    }
    nb = wave_incl_scan(nb);
    if (lane == 63 && nb) atomicAdd(&s_new, nb);
    __syncthreads();
    if (threadIdx.x == 0 && s_new) {
      g.out_flag[xr] = 1u;
      fresh += s_new;
    }
    __syncthreads();  // the LDS rows and shared words are reused by the next row
  }
  const u64 c = wave_incl_scan_t<u64>(cands), fr = wave_incl_scan_t<u64>(fresh);
  if (lane == 63) {
    if (c) atomicAdd(&g.counters[CNT_CANDIDATES], c);
    if (fr) atomicAdd(&g.counters[CNT_APPENDED], fr);
  }
}

// Gathered round by delta row (GatherArgs::by_a).  Every X that e1 pairs
// with A receives the same Y values from A's delta row: the union U(A) of
// e2's Y lists over the B bits of the delta row (words [in_lo, in_hi) only)
// is built once in LDS with the wave-balanced push expansion of the frontier
// kernels, and each nonzero word of U is ORed into the head row of every X
// of A with one device atomic whose old value gives the bits new to X; those
// go to X's next delta row (several A may reach one X, so that is an atomic
// too), raise X's flag and widen its word bounds.  One wavefront per
// workgroup handles one delta row at a time: a row's work is a chain of
// dependent global accesses (flag, word range, delta words, e2 offsets, Y
// lists, X list, atomics), most rows on a forest are small, and rows in
// flight, not threads per row, set the pace.  The wavefront that reads delta
// row A is the only one that touches it in the round, so it also empties it:
// each nonzero word as it is read, then A's flag and bounds, which every
// lane has read before lane 0 resets them.
constexpr uint32_t GA_STEP = 16;             // delta words decoded per step
constexpr uint32_t GA_ZCAP = GA_STEP * 32;   // B values listed per step, at most

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
  for (int k = 32; k > 0; k >>= 1) x = min(x, (uint32_t)__shfl_xor(x, k, 64));
  return x;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  for (int k = 32; k > 0; k >>= 1) x = max(x, (uint32_t)__shfl_xor(x, k, 64));
  return x;
}

__global__ __launch_bounds__(64) void gather_by_a_k(GatherArgs g) {
  extern __shared__ uint32_t U[];  // union of this A's Y values: zero between delta rows
  __shared__ uint32_t zlist[GA_ZCAP];
  __shared__ uint32_t s_excl[64], s_beg[64];
  const uint32_t W = g.row_words;
  const int lane = lane_id();
  u64 cands = 0, fresh = 0;
  const FrontierArgs& a = g.push;
  const uint32_t* ycol = a.idx.col[a.ybind_col];
  const uint32_t* xcol = g.e1a.col[g.e1_xcol];
  for (uint32_t i = lane; i < W; i += 64) U[i] = 0u;
  wave_lds_sync();
  for (int64_t ar64 = blockIdx.x; ar64 < g.range0; ar64 += gridDim.x) {
    const uint32_t ar = (uint32_t)ar64;
    if (!g.in_flag[ar]) continue;  // (uniform: no delta row)
    uint32_t* frow = g.in_bits + (u64)ar * W;
    const uint32_t wb = g.in_lo[ar], we = min(g.in_hi[ar], W);
    const uint32_t kk = (uint32_t)g.lo0 + ar - (uint32_t)g.e1a.key_lo;
    uint32_t b1 = 0, n1 = 0;
    if (kk < g.e1a.key_range) {
      b1 = g.e1a.off[kk];
      n1 = g.e1a.off[kk + 1] - b1;
    }
    if (n1 == 0) {  // (uniform: no X pairs with A) empty the row unread
      for (uint32_t wi = wb + (uint32_t)lane; wi < we; wi += 64) frow[wi] = 0u;
      if (lane == 0) {
        g.in_flag[ar] = 0u;
        g.in_lo[ar] = W;
        g.in_hi[ar] = 0u;
      }
      continue;
    }
    uint32_t umin = 0xffffffffu, umax = 0u;  // this lane's words of U touched
    for (uint32_t cb = wb; cb < we; cb += GA_STEP) {
      // the B values of delta words [cb, cb + GA_STEP), in order
      const uint32_t wi = cb + (uint32_t)lane;
      const uint32_t d = lane < (int)GA_STEP && wi < we ? frow[wi] : 0u;
      if (d) frow[wi] = 0u;
      const uint32_t c = __popc(d);
      const uint32_t incl = wave_incl_scan(c);
      const uint32_t nz = __shfl(incl, 63, 64);
      uint32_t pos = incl - c;
      for (uint32_t bits = d; bits; bits &= bits - 1)
        zlist[pos++] = (uint32_t)a.lo1 + wi * 32u + (uint32_t)(__ffs(bits) - 1);
      wave_lds_sync();
      // each B's Y list: rows of 64 or more by the whole wavefront, smaller
      // ones through a scan and a six-step owner search
      for (uint32_t j0 = 0; j0 < nz; j0 += 64) {
        const uint32_t r = j0 + (uint32_t)lane;
        uint32_t beg = 0, deg = 0;
        if (r < nz) {
          const uint32_t k2 = zlist[r] - (uint32_t)a.idx.key_lo;
          if (k2 < a.idx.key_range) {
            beg = a.idx.off[k2];
            deg = a.idx.off[k2 + 1] - beg;
          }
        }
        const bool big = deg >= 64;
        u64 bigm = __ballot(big);
        const uint32_t sdeg = big ? 0u : deg;
        const uint32_t sincl = wave_incl_scan(sdeg);
        const uint32_t total = __shfl(sincl, 63, 64);
        s_excl[lane] = sincl - sdeg;
        s_beg[lane] = beg;
        wave_lds_sync();
        if (lane == 0) cands += total;
        while (bigm) {
          const int rb = __ffsll((long long)bigm) - 1;
          bigm &= bigm - 1;
          const uint32_t bb = __shfl(beg, rb, 64), bd = __shfl(deg, rb, 64);
          if (lane == 0) cands += bd;
          for (uint32_t k = lane; k < bd; k += 64) {
            const uint32_t y = ycol[bb + k] - (uint32_t)a.lo1;
            const uint32_t bit = 1u << (y & 31);
            umin = min(umin, y >> 5);
            umax = max(umax, y >> 5);
            if (!(U[y >> 5] & bit)) atomicOr(&U[y >> 5], bit);
          }
        }
        for (uint32_t b0 = 0; b0 < total; b0 += 64) {
          const uint32_t j = b0 + lane;
          if (j < total) {
            int q = 0;
#pragma unroll
            for (int step = 32; step > 0; step >>= 1)
              if (s_excl[q + step] <= j) q += step;
            const uint32_t y = ycol[s_beg[q] + (j - s_excl[q])] - (uint32_t)a.lo1;
            const uint32_t bit = 1u << (y & 31);
            umin = min(umin, y >> 5);
            umax = max(umax, y >> 5);
            if (!(U[y >> 5] & bit)) atomicOr(&U[y >> 5], bit);
          }
        }
        wave_lds_sync();
      }
    }
    if (lane == 0) {  // the row is empty now; every lane read wb and we above
      g.in_flag[ar] = 0u;
      g.in_lo[ar] = W;
      g.in_hi[ar] = 0u;
    }
    umin = wave_min_u32(umin);
    umax = wave_max_u32(umax);
    if (umin > umax) continue;  // (uniform: no Y value; U is still zero)
    const uint32_t hi = min(umax + 1u, W);
    uint32_t nb = 0;
    for (uint32_t q = 0; q < n1; ++q) {
      const uint32_t xr = xcol[b1 + q] - (uint32_t)g.lo0;
      if ((int64_t)xr >= g.range0) continue;  // outside the head's rows (not planned)
      if (lane == 0) {  // X's next delta row may get bits in these words
        atomicMin(&g.out_lo[xr], umin);
        atomicMax(&g.out_hi[xr], hi);
      }
      bool any = false;
      for (uint32_t wi = umin + (uint32_t)lane; wi < hi; wi += 64) {
        const uint32_t u = U[wi];
        if (!u) continue;
        const u64 at = (u64)xr * W + wi;
        const uint32_t nw = u & ~atomicOr(g.bits + at, u);
        if (nw) {
          atomicOr(g.out_bits + at, nw);
          nb += (uint32_t)__popc(nw);
          any = true;
        }
      }
      if (__ballot(any) && lane == 0) g.out_flag[xr] = 1u;
    }
    fresh += nb;
    wave_lds_sync();  // every word of U is read before it is cleared
    for (uint32_t wi = umin + (uint32_t)lane; wi < hi; wi += 64) U[wi] = 0u;
    wave_lds_sync();
  }
  const u64 c = wave_incl_scan_t<u64>(cands), fr = wave_incl_scan_t<u64>(fresh);
  if (lane == 63) {
    if (c) atomicAdd(&g.counters[CNT_CANDIDATES], c);
    if (fr) atomicAdd(&g.counters[CNT_APPENDED], fr);
  }
}

hipError_t gather_round(const GatherArgs& a, hipStream_t s) {
  if (a.range0 <= 0) return hipSuccess;
  if (a.by_a) {
    // eight single-wavefront workgroups per compute unit: measured on the
    // 20,000-node forest, 2,048 wavefronts take 0.60 ms per run against 0.71
    // with 1,024, 0.66 with 3,072 and 0.94 with 8,192
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const unsigned grid = (unsigned)std::min<int64_t>(a.range0, 8 * (int64_t)std::max(cus, 1));
    gather_by_a_k<<<grid, 64, (size_t)a.row_words * sizeof(uint32_t), s>>>(a);
  } else {
    const unsigned grid = (unsigned)std::min<int64_t>(a.range0, 2048);
    gather_round_k<<<grid, FR_THREADS, (size_t)a.row_words * 2 * sizeof(uint32_t), s>>>(a);
  }
  return hipGetLastError();
}

// Empty the flagged rows (only their words [lo, hi) when bounds are kept,
// which are then reset to empty) and their flags.
// One wavefront per row: most rows are not flagged, so the rows a wavefront
// visits one after another (a flag load each) are kept few.  Every lane has
// read the flag and the bounds before lane 0 resets them (one wavefront, in
// program order).
__global__ __launch_bounds__(256) void clear_flagged_rows_k(uint32_t* bits, uint32_t* flag, int64_t nrows,
                                                            uint32_t row_words, uint32_t* lo, uint32_t* hi) {
  const uint32_t lane = (uint32_t)lane_id();
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < nrows; r += (int64_t)gridDim.x * 4) {
    if (!flag[r]) continue;  // (uniform within the wavefront)
    uint32_t* row = bits + (u64)r * row_words;
    const uint32_t b = lo ? lo[r] : 0u, e = lo ? min(hi[r], row_words) : row_words;
    for (uint32_t i = b + lane; i < e; i += 64) row[i] = 0u;
    if (lane == 0) {
      flag[r] = 0u;
      if (lo) {
        lo[r] = row_words;
        hi[r] = 0u;
      }
    }
  }
}

hipError_t clear_flagged_rows(uint32_t* bits, uint32_t* flag, int64_t nrows, uint32_t row_words, uint32_t* lo,
                              uint32_t* hi, hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  clear_flagged_rows_k<<<(unsigned)std::min<int64_t>((nrows + 3) / 4, 8192), 256, 0, s>>>(bits, flag, nrows,
                                                                                         row_words, lo, hi);
  return hipGetLastError();
}

// lo[r] = vlo, hi[r] = vhi for every row.
__global__ void fill_bounds_k(uint32_t* lo, uint32_t* hi, int64_t n, uint32_t vlo, uint32_t vhi) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
    lo[r] = vlo;
    hi[r] = vhi;
  }
}
hipError_t fill_bounds(uint32_t* lo, uint32_t* hi, int64_t n, uint32_t vlo, uint32_t vhi, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  fill_bounds_k<<<grid_for(n, 256, 4096), 256, 0, s>>>(lo, hi, n, vlo, vhi);
  return hipGetLastError();
}

// Number of set bits in each bitmap row.
// One wavefront per row: four word loads in flight per lane, then a
// shuffle reduction (no barriers).
__global__ __launch_bounds__(256) void row_popcount_k(const uint32_t* bits, int64_t nrows,
                                                      uint32_t row_words, uint32_t* cnt) {
  const uint32_t lane = (uint32_t)lane_id();
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < nrows; r += (int64_t)gridDim.x * 4) {
    const uint32_t* row = bits + (u64)r * row_words;
    uint32_t c = 0;
    for (uint32_t i = lane; i < row_words; i += 256) {
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) w[k] = i + 64u * k < row_words ? row[i + 64u * k] : 0u;
#pragma unroll
      for (int k = 0; k < 4; ++k) c += (uint32_t)__popc(w[k]);
    }
    for (int k = 32; k > 0; k >>= 1) c += __shfl_xor(c, k, 64);
    if (lane == 0) cnt[r] = c;
  }
}
hipError_t row_popcount(const uint32_t* bits, int64_t nrows, uint32_t row_words, uint32_t* cnt,
                        hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  row_popcount_k<<<(unsigned)std::min<int64_t>((nrows + 3) / 4, 1 << 16), 256, 0, s>>>(bits, nrows, row_words,
                                                                                      cnt);
  return hipGetLastError();
}

// Relation rows (x, y) of every set bit, in ascending (x, y) order: bitmap row
// r holds x = lo0 + r and starts at off[r].  Each chunk of 256 words is
// decoded into LDS first so the column writes are coalesced.  Rows at
// positions cap and beyond are not written (the columns hold cap rows).
__global__ __launch_bounds__(256) void bits_to_rows_k(const uint32_t* bits, int64_t nrows,
                                                      uint32_t row_words, const uint32_t* off,
                                                      int32_t lo0, int32_t lo1, uint32_t* c0,
                                                      uint32_t* c1, u64 cap) {
  __shared__ __align__(16) uint32_t stage[256 * 32 + 4];
  __shared__ uint32_t s_w[4];
  for (int64_t r = blockIdx.x; r < nrows; r += gridDim.x) {
    const uint32_t* row = bits + (u64)r * row_words;
    u64 out = off[r];
    const uint32_t x = (uint32_t)lo0 + (uint32_t)r;
    const uint4 xq = make_uint4(x, x, x, x);
    uint32_t dn = threadIdx.x < row_words ? row[threadIdx.x] : 0u;
    for (uint32_t cb = 0; cb < row_words; cb += 256) {
      const uint32_t wi = cb + threadIdx.x;
      const uint32_t d = dn;
      dn = wi + 256 < row_words ? row[wi + 256] : 0u;  // the next step's word, loaded ahead
      // value i of the chunk goes to stage[sh + i] and to output position
      // out + i, so stage index s and position out - sh + s agree modulo 4:
      // whole quads are one 16-byte LDS read and two 16-byte stores
      const uint32_t sh = (uint32_t)(out & 3u);
      uint32_t n;
      uint32_t pos = sh + block_excl_scan_u32(__popc(d), &n, s_w);
      for (uint32_t b = d; b; b &= b - 1) stage[pos++] = (uint32_t)lo1 + wi * 32u + (uint32_t)(__ffs(b) - 1);
      __syncthreads();
      const uint32_t end = sh + n;
      const u64 base = out - sh;
      for (uint32_t q = threadIdx.x; q < (end + 3u) / 4u; q += 256) {
        const uint32_t s0 = 4u * q;
        const u64 p = base + s0;
        if (s0 >= sh && s0 + 4u <= end && p + 4u <= cap) {
          *reinterpret_cast<uint4*>(c1 + p) = *reinterpret_cast<const uint4*>(stage + s0);
          *reinterpret_cast<uint4*>(c0 + p) = xq;
        } else {
#pragma unroll
          for (uint32_t k = 0; k < 4u; ++k) {
            if (s0 + k >= sh && s0 + k < end && p + k < cap) {
              c0[p + k] = x;
              c1[p + k] = stage[s0 + k];
            }
          }
        }
      }
      out += n;
      __syncthreads();
    }
  }
}
// The same with one wavefront per row (four rows per workgroup, no
// workgroup barriers): for sparse bitmaps, where a row's steps write few
// rows each and the barriers of the workgroup form would set the pace.
__global__ __launch_bounds__(256) void bits_to_rows_wave_k(const uint32_t* bits, int64_t nrows,
                                                           uint32_t row_words, const uint32_t* off,
                                                           int32_t lo0, int32_t lo1, uint32_t* c0,
                                                           uint32_t* c1, u64 cap) {
  __shared__ __align__(16) uint32_t stage_all[4][64 * 32 + 4];
  const uint32_t lane = (uint32_t)lane_id();
  uint32_t* stage = stage_all[threadIdx.x >> 6];
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < nrows; r += (int64_t)gridDim.x * 4) {
    const uint32_t* row = bits + (u64)r * row_words;
    u64 out = off[r];
    const uint32_t x = (uint32_t)lo0 + (uint32_t)r;
    const uint4 xq = make_uint4(x, x, x, x);
    uint32_t dn = lane < row_words ? row[lane] : 0u;
    for (uint32_t cb = 0; cb < row_words; cb += 64) {
      const uint32_t wi = cb + lane;
      const uint32_t d = dn;
      dn = wi + 64 < row_words ? row[wi + 64] : 0u;
      const uint32_t sh = (uint32_t)(out & 3u);
      const uint32_t c = (uint32_t)__popc(d);
      const uint32_t incl = wave_incl_scan(c);
      const uint32_t n = __shfl(incl, 63, 64);
      uint32_t pos = sh + incl - c;
      for (uint32_t b = d; b; b &= b - 1) stage[pos++] = (uint32_t)lo1 + wi * 32u + (uint32_t)(__ffs(b) - 1);
      wave_lds_sync();
      const uint32_t end = sh + n;
      const u64 base = out - sh;
      for (uint32_t q = lane; q < (end + 3u) / 4u; q += 64) {
        const uint32_t s0 = 4u * q;
        const u64 p = base + s0;
        if (s0 >= sh && s0 + 4u <= end && p + 4u <= cap) {
          *reinterpret_cast<uint4*>(c1 + p) = *reinterpret_cast<const uint4*>(stage + s0);
          *reinterpret_cast<uint4*>(c0 + p) = xq;
        } else {
#pragma unroll
          for (uint32_t k = 0; k < 4u; ++k) {
            if (s0 + k >= sh && s0 + k < end && p + k < cap) {
              c0[p + k] = x;
              c1[p + k] = stage[s0 + k];
            }
          }
        }
      }
      out += n;
      wave_lds_sync();
    }
  }
}
hipError_t bits_to_rows(const uint32_t* bits, int64_t nrows, uint32_t row_words, const uint32_t* off,
                        int32_t lo0, int32_t lo1, uint32_t* c0, uint32_t* c1, int64_t cap, hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  // fewer than a quarter of the bits set (cap is the row total): one
  // wavefront per row (same generation's 17%: -3%; the R-MAT closure's
  // 48% takes 3% longer that way)
  if ((double)cap * 4.0 < (double)nrows * row_words * 32.0)
    bits_to_rows_wave_k<<<(unsigned)std::min<int64_t>((nrows + 3) / 4, 1 << 16), 256, 0, s>>>(
        bits, nrows, row_words, off, lo0, lo1, c0, c1, (u64)cap);
  else
    bits_to_rows_k<<<(unsigned)std::min<int64_t>(nrows, 1 << 16), 256, 0, s>>>(bits, nrows, row_words, off, lo0,
                                                                              lo1, c0, c1, (u64)cap);
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
// the index of e by its Y column.  One lane per y and one ballot per 64 y:
// lanes 0 and 32 write the wavefront's two words.
__global__ void hasin_bits_k(IndexProbe rev, int32_t lo1, uint32_t words, uint32_t* out) {
  const uint32_t lane = (uint32_t)lane_id();
  const u64 n = (u64)words * 32u;
  const u64 waves = (u64)gridDim.x * (blockDim.x / 64);
  for (u64 base = ((u64)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6)) * 64; base < n; base += waves * 64) {
    const u64 y = base + lane;
    const uint32_t kk = (uint32_t)lo1 + (uint32_t)y - (uint32_t)rev.key_lo;
    const bool has = y < n && kk < rev.key_range && rev.off[kk + 1] > rev.off[kk];
    const u64 m = __ballot(has);
    const u64 wi = base / 32;
    if (lane == 0) out[wi] = (uint32_t)m;
    if (lane == 32 && wi + 1 < words) out[wi + 1] = (uint32_t)(m >> 32);
  }
}
hipError_t hasin_bits(const IndexProbe& rev, int32_t lo1, uint32_t words, uint32_t* out, hipStream_t s) {
  hasin_bits_k<<<grid_for((int64_t)words * 32, 256, 4096), 256, 0, s>>>(rev, lo1, words, out);
  return hipGetLastError();
}

}  // namespace k
}  // namespace xlh
