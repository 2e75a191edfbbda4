// Host-side launchers for the HIP kernels (all enqueue on the given stream and
// return the launch status; none synchronizes).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "device_types.h"

namespace xlh {
namespace k {

typedef unsigned long long u64;

// ---- device-wide exclusive prefix sum (in place allowed) ----
size_t scan_temp_bytes(int64_t n);
hipError_t scan_exclusive_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total,
                              void* temp, hipStream_t s);
hipError_t scan_exclusive_u64(const u64* in, u64* out, int64_t n, u64* total, void* temp,
                              hipStream_t s);

// ---- LSD radix sort of (key, u32 value) pairs on bits [0, bits) ----
// Ping-pongs between (keys, vals) and (keys_alt, vals_alt); *in_alt tells
// which pair holds the result.  vals may be null (keys only).
size_t radix_temp_bytes(int64_t n);
hipError_t radix_sort_u32(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt,
                          int64_t n, int bits, void* temp, hipStream_t s, int* in_alt);
hipError_t radix_sort_u64(u64* keys, uint32_t* vals, u64* keys_alt, uint32_t* vals_alt,
                          int64_t n, int bits, void* temp, hipStream_t s, int* in_alt);

// ---- small helpers ----
// hipMemsetAsync's result; a kernel of 16-byte stores for 1 MB and more.
hipError_t fill_bytes(void* p, int byte, size_t bytes, hipStream_t s);
hipError_t iota_u32(uint32_t* out, int64_t n, hipStream_t s);
hipError_t gather_u32(const uint32_t* src, const uint32_t* perm, uint32_t* dst, int64_t n,
                      hipStream_t s);
// dst[j][i] = src[j][perm[i]] for the ncols (<= MAXC) columns, one launch.
hipError_t gather_cols(const uint32_t* const* src, uint32_t* const* dst, int ncols, const uint32_t* perm, int64_t n,
                       hipStream_t s);
// key[i] = col[i] - lo (unsigned) and perm[i] = i.
hipError_t keys_perm(const uint32_t* col, int32_t lo, int64_t n, uint32_t* key, uint32_t* perm, hipStream_t s);
// Order-preserving u32 image of a column: i32 signed order, f32 totalOrder.
hipError_t ordered_key(const uint32_t* col, int type, const uint32_t* perm, uint32_t* out,
                       int64_t n, hipStream_t s);
// out[0] = min, out[1] = max over an i32 column (out must be initialised by caller
// to {INT32_MAX, INT32_MIN}).
hipError_t minmax_i32(const int32_t* col, int64_t n, int32_t* out, hipStream_t s);
hipError_t bounds_one(const int32_t* col, const uint32_t* count, int64_t cap, int32_t* out, hipStream_t s);
// key[i] = col[i] - lo as unsigned.
hipError_t sub_lo(const uint32_t* col, int32_t lo, uint32_t* out, int64_t n, hipStream_t s);
// off[k] = first i with sorted[i] >= k, for k in [0, range].
// Compacted index offsets from n ascending keys: keys[0 .. *count) receive
// the distinct keys, off[0 .. *count] the first row of each and n (keys and
// off must hold n and n + 1 values; *count is written on the device).
size_t compact_offsets_temp_bytes(int64_t n);
hipError_t compact_offsets(const uint32_t* sorted, int64_t n, uint32_t* keys, uint32_t* off, uint32_t* count,
                           void* temp, hipStream_t s);
hipError_t csr_offsets(const uint32_t* sorted, int64_t n, uint32_t range, uint32_t* off,
                       hipStream_t s);
// The same over the high bits (key >> shift) of ascending 32-bit (wide
// false) or 64-bit keys.
hipError_t csr_offsets_high(const void* sorted, bool wide, int shift, int64_t n, uint32_t range, uint32_t* off,
                            hipStream_t s);
// Composite keys of an ordered index, 32-bit (wide false) or 64-bit, and
// perm[i] = i: (kcol[i] - klo) << obits | order part, the order part being
// 3 - min(3, bitlen(deg(ocol[i])) / 3) with deg from the CSR offsets doff
// over [olo, olo + drange) (degree order by base-8 class, obits 2), or ocol[i] -
// olo when doff is null (value order, int32 values in [olo, olo + 2^obits)).
hipError_t order_keys(const uint32_t* kcol, int32_t klo, const uint32_t* ocol, int32_t olo, int obits,
                      const uint32_t* doff, uint32_t drange, int64_t n, void* key, bool wide, uint32_t* perm,
                      hipStream_t s);
// out[k] = col[off[k]] for keys k in [0, range) with rows, 0xffffffff otherwise.
hipError_t segment_first(const uint32_t* off, const uint32_t* col, uint32_t range, uint32_t* out, hipStream_t s);
// Packed keys of a negation table: c0[i], or (c0[i] << 32) | c1[i].
hipError_t neg_keys(const uint32_t* c0, const uint32_t* c1, int64_t n, u64* key, hipStream_t s);

// ---- worst-case-optimal triangle join (see WcojArgs) ----
constexpr int WC_CHUNK = 256;  // items per wavefront chunk
hipError_t wcoj_work(const WcojArgs& a, hipStream_t s);
// flag[i] = v[i] != 0
hipError_t nonzero_flags(const uint32_t* v, int64_t n, uint32_t* flag, hipStream_t s);
// crow[pos[i]] = i and cw[pos[i]] = work[i] for rows with work
hipError_t wcoj_compact(const uint32_t* work, const uint32_t* pos, int64_t n, uint32_t* crow,
                        unsigned long long* cw, hipStream_t s);
hipError_t wcoj_probe(const WcojArgs& a, bool materialize, hipStream_t s);
// out[i] = key[i] >> shift, over 32-bit (wide false) or 64-bit keys
hipError_t high_bits(const void* key, bool wide, int shift, int64_t n, uint32_t* out, hipStream_t s);
// flag[i] = 1 if row i differs (bitwise) from row i-1 in any column (or i == 0).
hipError_t row_change_flags(const uint32_t* const* cols, int ncols, int64_t n, uint32_t* flag,
                            hipStream_t s);
// dst[pos[i]] = src[i] where flag[i] != 0.
hipError_t compact_u32(const uint32_t* src, const uint32_t* flag, const uint32_t* pos,
                       uint32_t* dst, int64_t n, hipStream_t s);

// ---- join / project / emit stage ----
// Batched set rounds (see the kernels' comment): bnd holds n entries.
hipError_t batch_init(u64* bnd, int n, u64 b0, u64 b1, hipStream_t s);
hipError_t batch_mark(u64* bnd, int j, const u64* counters, u64 base, hipStream_t s);
// Batched rounds of several set heads: after round j, unless a launch of
// any head overflowed (then every head's overflow flag is raised, so later
// rounds of the batch do nothing for all of them), bnd[h][j + 1] = base[h] +
// rows appended to head h in the batch so far.
constexpr int MAX_BATCH_HEADS = 8;
struct BatchMarks {
  u64* bnd[MAX_BATCH_HEADS];
  u64* cnt[MAX_BATCH_HEADS];
  u64 base[MAX_BATCH_HEADS];
  int n;
};
hipError_t batch_mark_heads(const BatchMarks& m, int j, hipStream_t s);
hipError_t stage_launch(const StageArgs& a, hipStream_t s, int grid_cap);

// ---- hash tables ----
hipError_t set_insert_rows(u64* table, u64 mask, const uint32_t* c0, const uint32_t* c1,
                           int64_t n, KeyPack kp, unsigned long long* counters, hipStream_t s);
hipError_t table16_insert_rows(Slot16* table, u64 mask, const uint32_t* c0, const uint32_t* c1,
                               const uint32_t* v, int64_t n, KeyPack kp, int type, int is_max,
                               unsigned long long* counters, hipStream_t s);
hipError_t table16_rehash(const Slot16* old, int64_t old_cap, Slot16* nt, u64 mask,
                          unsigned long long* counters, hipStream_t s);
// Ordered compactions (count -> scan -> write; *total = items kept; pass null
// outputs to count only).  temp: compact_temp_bytes(n).
size_t compact_temp_bytes(int64_t n);
hipError_t table16_stamped(const Slot16* t, int64_t cap, uint32_t round, uint32_t* delta_idx,
                           int64_t out_cap, uint32_t* total, void* temp, hipStream_t s);
// Rows (k0[, k1], v) of the given slots; folds are decoded (min/max transform).
hipError_t table16_rows_from_idx(const Slot16* t, const uint32_t* idx, int64_t n, KeyPack kp,
                                 int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                                 uint32_t* v, hipStream_t s);
// Delta rows of one batched keyed-table round, from the slot list positions
// [bnd[j], bnd[j + 1]) held on the device (max_n bounds them, for the grid);
// with acc (hashed sum/logsumexp) also the round's merge into the full
// relation and the accumulators' reset.
hipError_t table16_rows_range(Slot16* t, unsigned long long* acc, const uint32_t* idx, const unsigned long long* bnd,
                              int j, int64_t max_n, KeyPack kp, int type, int fold_kind, uint32_t* k0,
                              uint32_t* k1, uint32_t* v, hipStream_t s);
// Set n accumulators of hashed sum/logsumexp folds to the fold's identity.
hipError_t acc_fill(unsigned long long* acc, int64_t n, int type, int fold_kind, hipStream_t s);
hipError_t table16_compact(const Slot16* t, int64_t cap, KeyPack kp, int type, int fold_kind,
                           uint32_t* k0, uint32_t* k1, uint32_t* v, int64_t out_cap, uint32_t* total,
                           void* temp, hipStream_t s);
hipError_t dcount_rows(const uint32_t* counts, int64_t n, int64_t range1, KeyPack kp, uint32_t* k0,
                       uint32_t* k1, uint32_t* v, int64_t out_cap, uint32_t* total, void* temp,
                       hipStream_t s);

// ---- sorted-candidate aggregation (sum / logsumexp / count) ----
hipError_t seg_heads(const void* keys, int key_bytes, int64_t n, uint32_t* flag, hipStream_t s);
hipError_t seg_starts(const uint32_t* flag, const uint32_t* pos, int64_t n, uint32_t* start,
                      hipStream_t s);
// fold_kind: FOLD_SUM / FOLD_LSE / FOLD_COUNT / FOLD_MIN / FOLD_MAX
hipError_t seg_reduce(const void* keys, int key_bytes, const uint32_t* vals, const uint32_t* start, int64_t nseg,
                      int64_t n, KeyPack kp, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                      uint32_t* v, hipStream_t s);
// S(key) = S(key) (+) delta for every delta row (keys unique within the call).
hipError_t agg_merge(Slot16* t, u64 mask, const uint32_t* k0, const uint32_t* k1,
                     const uint32_t* v, int64_t n, KeyPack kp, int type, int fold_kind,
                     unsigned long long* counters, hipStream_t s);

// ---- dense set heads ----
hipError_t bits_set_rows(uint32_t* bits, u64 row_bits, const uint32_t* c0, const uint32_t* c1,
                         int64_t n, KeyPack kp, hipStream_t s);
hipError_t frontier_round(const FrontierArgs& a, hipStream_t s);
// All rounds of every first key in one launch; grid 0 = as many workgroups
// as the device keeps resident.
hipError_t frontier_resident(const FrontierArgs& a, unsigned grid, hipStream_t s);
// One gathered round (see GatherArgs).
hipError_t gather_round(const GatherArgs& a, hipStream_t s);
// Zero the flagged rows of a [nrows][row_words] bitmap and their flags.
hipError_t clear_flagged_rows(uint32_t* bits, uint32_t* flag, int64_t nrows, uint32_t row_words, uint32_t* lo,
                              uint32_t* hi, hipStream_t s);
// lo[r] = vlo, hi[r] = vhi for r < n (word bounds of delta rows).
hipError_t fill_bounds(uint32_t* lo, uint32_t* hi, int64_t n, uint32_t vlo, uint32_t vhi, hipStream_t s);
hipError_t hasin_bits(const IndexProbe& rev, int32_t lo1, uint32_t words, uint32_t* out, hipStream_t s);
hipError_t row_popcount(const uint32_t* bits, int64_t nrows, uint32_t row_words, uint32_t* cnt,
                        hipStream_t s);
hipError_t bits_to_rows(const uint32_t* bits, int64_t nrows, uint32_t row_words, const uint32_t* off,
                        int32_t lo0, int32_t lo1, uint32_t* c0, uint32_t* c1, int64_t cap, hipStream_t s);
// out row sg = bitmap row (x[sg] - lo0)
hipError_t gather_rows(const uint32_t* bits, uint32_t row_words, const uint32_t* x, int32_t lo0, int64_t nseg,
                       uint32_t* out, hipStream_t s);
// Dense value heads (first key through a dictionary, second key direct).
// Rows of every present slot in slot order (= ascending keys).
// nrank = 0: slot rank * range1 + (y - lo1); nrank > 0: slot (y - lo1) * nrank + rank.
hipError_t dense_rows(const uint32_t* vals, const uint32_t* pres, const uint32_t* dict, int64_t n,
                      int64_t range1, int64_t nrank, KeyPack kp, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                      uint32_t* v, int64_t out_cap, uint32_t* total, void* temp, hipStream_t s);
hipError_t dict_mark(const uint32_t* col, int64_t n, int32_t lo, uint32_t range, uint32_t* mark, hipStream_t s);
hipError_t dict_finish(uint32_t* map, const uint32_t* pos, uint32_t range, int32_t lo, uint32_t* dict,
                       hipStream_t s);
hipError_t dense_insert_rows(uint32_t* vals, uint32_t* pres, const uint32_t* map, uint32_t map_n, uint32_t range1,
                             const uint32_t* c0, const uint32_t* c1, const uint32_t* v, int64_t n, KeyPack kp,
                             int type, int is_max, u64* counters, hipStream_t s);
hipError_t dense_delta_rows(const uint32_t* idx, int64_t n, const uint32_t* vals, uint32_t* chg, const uint32_t* dict,
                            uint32_t range1, int32_t lo1, int type, int fold_kind, uint32_t* k0, uint32_t* k1,
                            uint32_t* v, hipStream_t s);
// Dense sum/logsumexp heads.  bits_list: ascending list of the set bits,
// in two calls on the same temp (write=false counts into *total; write=true
// writes the list and clears the bits).
size_t bits_list_temp_bytes(int64_t nbits);
hipError_t bits_list_waves(uint32_t* bits, int64_t nbits, uint32_t* list, uint32_t* total, hipStream_t s);
hipError_t bits_list(uint32_t* bits, int64_t nbits, uint32_t* list, uint32_t* total, void* temp, bool write,
                     hipStream_t s);
hipError_t dense_pull(const DensePullArgs& a, hipStream_t s);
// Marks (target-major, nrank a multiple of 32) of the keys that receive a
// contribution from the delta presence bits pres, pushed through e's index by
// its Z column (fwd; ycol = e's Y column); mark must be all zero on entry.
// clear (optional, the same range1 * nrank / 32 words as pres, not aliasing
// pres or mark) is zeroed in the same launch.
hipError_t dense_mark_out(const IndexProbe& fwd, int ycol, int32_t lo1, uint32_t range1, uint32_t nrank,
                          const uint32_t* pres, uint32_t* mark, uint32_t* clear, hipStream_t s);
// Rows of the set bits of a dense key bitmap in bit order (two calls on the
// same temp as bits_list; temp sized by bits_list_temp_bytes); clear = zero
// the words read.
hipError_t bits_keys(uint32_t* bits, int64_t nbits, u64 row_bits, int32_t lo0, int32_t lo1, int nkey, bool clear,
                     uint32_t* c0, uint32_t* c1, uint32_t* total, void* temp, bool write, hipStream_t s);
hipError_t dense_apply_rows(const uint32_t* c0, const uint32_t* c1, const uint32_t* v, int64_t n, const uint32_t* map,
                            uint32_t map_n, uint32_t range1, uint32_t nrank, KeyPack kp, int fold_kind, int type,
                            uint32_t* cval,
                            uint32_t* cpres, uint32_t* fval, uint32_t* fpres, u64* counters, hipStream_t s);
// Dense min/max heads, tiled rounds (see DenseTileArgs).
// Delta rows from the delta bits in slot order (two calls on the same temp,
// sized by bits_list_temp_bytes: write=false counts, write=true writes the
// rows and clears the bits).  roff (optional, [nslots / range1 + 1], range1 a
// multiple of 32): the write pass also stores each rank's first row and the
// row total.
hipError_t dense_delta_from_bits(uint32_t* chg, int64_t nslots, uint32_t range1, const uint32_t* vals, const uint32_t* dict,
                            int32_t lo1, int type, int fold_kind, uint32_t* k0, uint32_t* k1, uint32_t* v,
                            uint32_t* roff, uint32_t* total, void* temp, bool write, hipStream_t s);
size_t dense_tile_lds_bytes(uint32_t tile);
// key[i] = tile * zr + (z - zlo), where tile = (y - lo1) / tile_slots capped
// at ntiles (a Y outside the head's range); tile_only: key[i] = tile.
hipError_t tile_keys(const uint32_t* zc, const uint32_t* yc, int64_t n, int32_t zlo, int32_t lo1, uint32_t tile,
                     uint32_t ntiles, uint32_t zr, bool tile_only, uint32_t* key, hipStream_t s);
hipError_t dense_min_tiles(const DenseTileArgs& a, hipStream_t s);
// The same delta rows in one launch after a tile round that wrote tcnt
// ([n0 * ntiles] improved slots per (rank, tile), DenseTileArgs::tcnt): one
// workgroup per tile sums the counts of the tiles before it itself.  Fills
// roff[0 .. n0] and *total; clears the delta bits.  Needs n0 * ntiles <=
// TL_MAX_WORK, tile <= TL_MAX_TILE, tile and range1 multiples of 32
// (hipErrorInvalidValue otherwise).
constexpr uint32_t TL_MAX_WORK = 8192;
constexpr uint32_t TL_MAX_TILE = 32768;
hipError_t tile_delta_rows(uint32_t* chg, const uint32_t* tcnt, uint32_t n0, uint32_t ntiles, uint32_t tile,
                           uint32_t range1, const uint32_t* vals, const uint32_t* dict, int32_t lo1, int type,
                           int fold_kind, uint32_t* k0, uint32_t* k1, uint32_t* v, uint32_t* roff, uint32_t* total,
                           hipStream_t s);
// counts[key_lo + i - head_lo] += off[i + 1] - off[i] for every i < key_range
// with rows; a key outside [head_lo, head_lo + head_range) bumps CNT_FATAL.
hipError_t index_degree_add(const uint32_t* off, uint32_t key_range, int32_t key_lo, int32_t head_lo,
                            uint32_t head_range, uint32_t* counts, u64* check, hipStream_t s);
// *check |= bit when the device value *v differs from expected.
hipError_t check_eq(const uint32_t* v, uint32_t expected, u64* check, u64 bit, hipStream_t s);
// out[i] = in[i] + add
hipError_t add_u32(const uint32_t* in, uint32_t add, uint32_t* out, int64_t n, hipStream_t s);

enum FoldKind { FOLD_NONE = 0, FOLD_COUNT, FOLD_SUM, FOLD_MIN, FOLD_MAX, FOLD_LSE };

// ---- column coding of u32, bool, i64, u64 and f64 (coding.hip) ----
// out[i] = int32 image of in[i] (XL_U32: 4-byte values, XL_BOOL: bytes; a
// byte other than 0 or 1 sets *bad).
hipError_t encode_narrow(const void* in, int ltype, int64_t n, uint32_t* out, uint32_t* bad, hipStream_t s);
// out[i] = total-order key of the 8-byte value in[i] (XL_I64, XL_U64, XL_F64).
hipError_t order_keys64(const u64* in, int ltype, int64_t n, u64* out, hipStream_t s);
// flag[i] = sorted[i] differs from sorted[i - 1] (always 1 at i = 0).
hipError_t unique_flags64(const u64* sorted, int64_t n, uint32_t* flag, hipStream_t s);
hipError_t compact64(const u64* src, const uint32_t* flag, const uint32_t* pos, u64* dst, int64_t n,
                     hipStream_t s);
// out[i] = number of keys of the ascending dict[0..nd) below q[i].
hipError_t rank64(const u64* dict, int64_t nd, const u64* q, int64_t n, uint32_t* out, hipStream_t s);
// col[i] = map[col[i]] in place.
hipError_t remap_codes(uint32_t* col, int64_t n, const uint32_t* map, hipStream_t s);
// Values of n int32 images into out (1, 4 or 8 bytes each by ltype); dict
// holds the order keys of the 8-byte types.
hipError_t decode_column(const uint32_t* img, int64_t n, int ltype, const u64* dict, void* out, hipStream_t s);

}  // namespace k
}  // namespace xlh
