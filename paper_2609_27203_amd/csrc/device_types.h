// Plain descriptors passed by value to the HIP kernels.  The host planner
// fills them; the kernels interpret them uniformly across a wavefront (every
// field is the same for all lanes, so the interpretation costs only scalar
// instructions).
#pragma once
#include <stdint.h>

namespace xlh {

constexpr int MAXV = 8;     // variable slots per rule
constexpr int MAXC = 4;     // columns per relation (XL_MAX_ARITY)
constexpr int MAXOPS = 12;  // micro-ops (comparisons / arithmetic) per stage
constexpr int MAXK = 8;     // constants per stage

enum ValType : uint8_t { T_I32 = 1, T_F32 = 2 };

// What to do with one column of a row source or an index relation.
enum ColActKind : int8_t { CA_NONE = 0, CA_BIND = 1, CA_CHECK_SLOT = 2, CA_CHECK_CONST = 3 };
struct ColAct {
  int8_t kind;
  int8_t slot;
  uint8_t type;   // ValType of the column (equality is IEEE for f32)
  int8_t pad;
  uint32_t cval;  // constant bits for CA_CHECK_CONST
};

// Micro-ops run after all columns of a stage are bound.
// OP_NOTIN: stratified negation; cmp = the rule's negation table, type = the
// number of constrained columns (0, 1 or 2), a and b their operands.
enum OpKind : uint8_t { OP_CMP = 1, OP_ADD = 2, OP_SUB = 3, OP_MOV = 4, OP_NOTIN = 5 };
enum CmpKind : uint8_t { CMP_NE = 0, CMP_EQ, CMP_LT, CMP_LE, CMP_GT, CMP_GE };
// Operand encoding: >= 0 is a slot, < 0 is constant index (-1 - k).
struct MicroOp {
  uint8_t kind, cmp, type, pad;
  int8_t dst, a, b, pad2;
};

// A negated literal not q(...) over a complete relation q: the sorted keys
// of q's rows projected onto the literal's constrained columns (variables and
// constants; none, one, or two int32 columns packed (v0 << 32) | v1 as
// unsigned), searched per candidate.  With no constrained column the literal
// only asks whether q has a row (n > 0).
constexpr int MAXNEG = 2;
struct NegTable {
  const unsigned long long* keys;
  int64_t n;
};

// Rows that drive a stage: a relation, a delta, or materialized bindings
// (up to one column per variable slot).
struct RowSource {
  const uint32_t* col[MAXV];
  int64_t n;
  int32_t ncols;
  ColAct act[MAXV];
};

// Index join: the rows of a relation whose key column equals slot key_slot;
// col[] are the relation's columns permuted into key order.
//   direct (keys == nullptr): off[k] .. off[k+1] delimit the rows with key
//     value key_lo + k, for k < key_range (a dense key range);
//   compacted (keys != nullptr): keys[0 .. key_range) are the distinct key
//     values minus key_lo (as unsigned, ascending) and off[i] .. off[i+1]
//     delimit the rows of keys[i] (sparse or wide key ranges, found by
//     binary search).
struct IndexProbe {
  const uint32_t* off;
  const uint32_t* keys;
  const uint32_t* col[MAXC];
  int32_t ncols;
  int32_t key_lo;
  uint32_t key_range;
  int8_t key_slot;
  ColAct act[MAXC];
};

// Head key packing: ((v0 - lo0) << shift) | (v1 - lo1), both as unsigned.
struct KeyPack {
  int32_t nkey;
  int8_t slot[2];
  int32_t lo[2];
  int32_t shift;
};

// Open-addressing slot for keyed values (min/max/sum/logsumexp/count heads).
struct Slot16 {
  unsigned long long key;
  uint32_t val;
  uint32_t stamp;
};

constexpr unsigned long long EMPTY_KEY = ~0ull;

enum EmitMode : int32_t {
  EM_COUNT = 0,   // count the rows each chunk would emit
  EM_MAT = 1,     // write bindings or (packed key, value) at scanned offsets
  EM_SET = 2,     // insert-if-absent into a key set; winners append head rows
  EM_MINMAX = 3,  // atomic improvement in a keyed table; improved keys to delta
  EM_BITSET = 4,  // test-and-set in a dense key-domain bitmap; winners append head rows
  EM_DCOUNT = 5,  // count per key in a dense counter array (runs of equal keys combined)
  EM_DMIN = 6,    // atomic improvement in a dense value array over (dictionary rank of
                  // the first key) x (second key); improved slots to delta
  EM_MARK = 7,    // set the bit of the same dense slot (keys that receive a contribution)
  EM_HAGG = 8,    // sum/logsumexp contributions of a round folded per key in a keyed table's
                  // accumulator array (acc[slot]); the slots touched in the round to delta
};

// Device-side counters of one emission (cleared per round).
enum Counter : int32_t {
  CNT_APPENDED = 0,   // rows appended to the output list
  CNT_INSERTED = 1,   // keys newly inserted into the table
  CNT_OVERFLOW = 2,   // set when inserted keys pass the table's load limit
  CNT_CANDIDATES = 3, // head tuples produced by the join/project step
  CNT_FATAL = 4,      // probe sequence exhausted (must never happen)
  CNT_SEGS = 5,       // delta segments written by the grouped expansion
  CNT_N = 8
};

// Internal consistency flags a run's kernels may set (Context::dcheck); any
// set bit fails the run with XL_DEVICE_ERROR.
enum CheckBit : unsigned long long {
  CHECK_BITMAP_ROWS = 1,    // a dense head's bitmap holds a different row count than its receipt
  CHECK_COUNT_DOMAIN = 2,   // a count key outside the head's planned domain
};

struct EmitSpec {
  int32_t mode;
  KeyPack key;
  int8_t val_slot;
  uint8_t val_type;
  uint8_t is_max;        // EM_MINMAX: fold is max (stored complemented)
  uint8_t mat_packed;    // EM_MAT: write (packed key, value) instead of slots
  int32_t nout;
  int8_t out_slot[MAXV];
  uint32_t* out_col[MAXV];
  unsigned long long* out_key;  // EM_MAT packed: 64-bit keys, or 32-bit when key32
  uint8_t key32;
  uint32_t* out_val;
  const unsigned long long* chunk_off;  // EM_MAT: exclusive offsets per chunk
  int64_t mat_base;                     // EM_MAT: added to every output position
  unsigned long long* chunk_cnt;        // EM_COUNT: rows per chunk
  // EM_SET
  unsigned long long* table;
  unsigned long long mask;   // capacity - 1 (capacity is a power of two)
  uint32_t* row_col[2];      // head row list (key columns), written at row_base + k
  int64_t row_base;
  int64_t row_cap;
  // EM_BITSET: bit (k0 - lo0) * row_bits + (k1 - lo1) of a dense key domain
  // EM_DCOUNT: counter of the same index, with row_bits = the second key's range
  uint32_t* bits;
  unsigned long long row_bits;
  // EM_MINMAX / EM_HAGG
  Slot16* table16;
  uint32_t round;
  uint32_t* delta_idx;       // EM_MINMAX / EM_DMIN: improved slots of this round; EM_HAGG: touched slots
  // EM_MINMAX / EM_DMIN / EM_HAGG: delta_idx positions from delta_lim on are
  // not written and the launch overflows (0: no limit)
  unsigned long long delta_lim;
  // EM_HAGG: one accumulator per table slot, at the fold's identity between
  // rounds (integer sum: the low 32 bits; f32 sum: an f64 sum; logsumexp:
  // an f64 log-sum); a key inserted in the round takes agg_identity as its
  // full-relation value until the round's end merges the accumulator
  unsigned long long* acc;
  int32_t fold_kind;
  uint32_t agg_identity;
  // EM_DMIN: slot = dmap[k0 - lo0] * row_bits + (k1 - lo1) of the value array
  // `bits`; dpres marks slots holding a value, dchg slots already listed in
  // this round's delta.
  const uint32_t* dmap;
  uint32_t dmap_n;
  uint32_t* dpres;
  uint32_t* dchg;
  // EM_MARK: bit (k1 - lo1) * nrank + dmap[k0 - lo0] of dchg (second key
  // major: the keys of one second key lie together)
  uint32_t nrank;
  // shared
  unsigned long long* counters;
  unsigned long long limit;  // overflow threshold on CNT_INSERTED
};

struct StageArgs {
  RowSource src;
  int32_t has_index;
  IndexProbe idx;
  // has_idx2: a second index whose key the driver row binds too; a driver
  // row then yields the product of its two match lists (row k of the
  // product: idx row k / deg2, idx2 row k % deg2)
  int32_t has_idx2;
  IndexProbe idx2;
  int32_t nops;
  MicroOp ops[MAXOPS];
  uint32_t consts[MAXK];
  NegTable neg[MAXNEG];
  EmitSpec emit;
  // batched rounds: the driver rows are [src_range[0], src_range[1]) of the
  // src columns (read on the device; src.n only bounds the grid), and the
  // launch does nothing once an earlier launch of the batch overflowed
  // (emit.counters[CNT_OVERFLOW]); null: rows [0, src.n)
  const unsigned long long* src_range;
};

// One round of a carried-value rule over a dense sum/logsumexp head, for the
// keys marked in the round: key (s, y) folds the contributions of every row
// of e whose Y column is y (rev) and whose Z value z has (s, z) in the
// current delta, evaluating the rule's comparisons and arithmetic per row.
// The delta arrays (cval/cpres, nval/npres) and the marked list use the
// second-key-major slot (y - lo1) * nrank + rank(s): listed keys of one y lie
// together, and the delta values of (s, z) for a fixed z and consecutive s
// are consecutive words, so the wavefront's reads of one in-edge coalesce.
// The full relation (fval/fpres) uses the same slots, so each lane's merge
// reads and writes consecutive words and the presence bits of one word are
// set by one atomic per run of lanes.  A key's contributions are folded in
// index order: the result is deterministic.
struct DensePullArgs {
  const uint32_t* list;   // marked delta slots, ascending
  int64_t n;              // listed keys, or their upper bound when n_dev is set
  const uint32_t* n_dev;  // listed keys in device memory (batched rounds), else null
  const uint32_t* dict;   // rank -> first key value
  uint32_t range1;
  uint32_t nrank;         // ranks (first key values in the dictionary)
  int32_t lo1;
  IndexProbe rev;         // e indexed by its Y column; act[] = the rule's actions on e
  int32_t zcol;
  int8_t slot_s, slot_z, slot_y, slot_p, val_slot;
  uint8_t val_type;
  int8_t fast, fcol;      // as in DenseTileArgs
  int32_t fold_kind;
  int32_t nops;
  MicroOp ops[MAXOPS];
  uint32_t consts[MAXK];
  NegTable neg[MAXNEG];     // unused: rules with negation do not take this form
  const uint32_t* cval;   // current delta: values and presence bits
  const uint32_t* cpres;
  uint32_t* nval;         // next delta: values and presence bits
  uint32_t* npres;
  uint32_t* fval;         // full relation: values and presence bits
  uint32_t* fpres;
  uint32_t* k0;           // next delta rows, row i for list[i] (all null: not written)
  uint32_t* k1;
  uint32_t* v;
  unsigned long long* counters;  // CNT_INSERTED: keys new to the full relation; CNT_FATAL
};

// One round of a carried-value rule over a dense min/max head, tiled: the
// workgroup for (rank r, tile t) keeps value slots [t * tile, t * tile + tile)
// of rank r's row in LDS, walks all delta rows of rank r (grouped by rank,
// roff), expands each through e's index by Z and folds the candidates whose Y
// falls in its tile with LDS atomicMin.  It owns those slots, so the write-back
// of values, presence and delta bits needs no global atomics.
struct DenseTileArgs {
  const uint32_t* dk1;    // delta rows of this round: Z and value, grouped by rank
  const uint32_t* dval;
  const uint32_t* roff;   // [n0 + 1] first delta row of each rank
  const uint32_t* dict;   // rank -> first key value
  uint32_t n0;
  uint32_t range1;        // slots per rank (a multiple of 32)
  int32_t lo1;
  uint32_t tile, ntiles;  // tile width (a multiple of 32) and tiles per rank
  IndexProbe idx;         // e's columns grouped by (tile of Y, Z); act[] = the rule's actions on e
  const uint32_t* toff;   // [t * idx.key_range + (z - idx.key_lo)]: first row of Z value z in tile t
  int32_t ycol;           // column of e bound to Y
  int8_t slot_s, slot_z, slot_p, slot_y, val_slot;
  uint8_t val_type, is_max;
  // 1 / 2: the rule is "value is P1 + / - e.col[fcol]" with nothing else to
  // check, evaluated directly instead of through the micro-op list
  int8_t fast, fcol;
  int32_t nops;
  MicroOp ops[MAXOPS];
  uint32_t consts[MAXK];
  NegTable neg[MAXNEG];   // unused: rules with negation do not take this form
  uint32_t* vals;         // encoded values (fold_encode), presence bits, delta bits
  uint32_t* pres;
  uint32_t* chg;
  unsigned long long* counters;  // CNT_CANDIDATES, CNT_INSERTED (new keys), CNT_APPENDED (improved keys)
  uint32_t* tcnt;         // [n0 * ntiles] or null: improved slots of each (rank, tile) this round
};

// Closure-shaped recursive rule head(X, Y) :- delta head(X, Z), e(Z, Y) over a
// dense set head, run in frontier form: the delta of every first-key value x
// is a bitmap row holding the Z values that became true in the previous
// round.  One workgroup owns one x per round: it stages bitmap row x in LDS,
// expands every Z of x's delta row through the index of e, merges the
// produced Y values with LDS atomics and writes the next delta row.
struct FrontierArgs {
  const uint32_t* x;        // [nseg] first-key value of delta row sg (fixed after the seed)
  const uint32_t* in_cnt;   // [nseg] bits in delta row sg (0: skip)
  const uint32_t* in_diff;  // [nseg][row_words] delta bits
  int64_t nseg;
  IndexProbe idx;           // e indexed by its join column
  int32_t ybind_col;        // column of e bound to Y
  uint32_t* bits;           // dense membership bitmap of the head
  int32_t lo0, lo1;
  uint32_t row_words;
  uint32_t* out_cnt;        // next delta: counts and bitmap rows, same slots
  uint32_t* out_diff;
  unsigned long long* counters;  // CNT_CANDIDATES, CNT_APPENDED (= new tuples)
  // Pull direction: e indexed by the Y column; Z is rev.col[rev_zcol], the
  // rows of one Y ordered by the out-degree of their Z, most first;
  // rev_first[y - rev.key_lo] is the Z of Y's first row.  A workgroup pulls
  // when pull_ratio * |delta(x)| >= |unreached Y with an in-edge| (pull_ratio
  // 0: always push).
  IndexProbe rev;
  int32_t rev_zcol;
  const uint32_t* rev_first;
  // Resident form (x and in_cnt may be null: delta row sg then belongs to
  // first key lo0 + sg, and an empty row is found by counting its bits): each
  // workgroup takes first keys from *queue (zero at
  // launch) and runs all of a key's rounds with its row held in LDS, writing
  // the row back once; per round r (from 0) it adds the tuples found to
  // round_new[min(r, round_slots - 1)], raises *max_round to the rounds it
  // ran (the last one found nothing), and sets *overflow when a key still has
  // a delta after max_rounds rounds.
  uint32_t* queue;
  uint32_t* max_round;
  uint32_t* overflow;
  unsigned long long* round_new;
  uint32_t round_slots;
  uint32_t max_rounds;
  const uint32_t* hasin;    // bit (y - lo1): y has at least one in-edge
  uint32_t pull_ratio;
};

// Gathered round of h(X, Y) :- e1(X, A), delta h(A, B), e2(Y, B) over a dense
// set head (same generation's shape): head row X receives the Y values that
// e2 pairs with the B bits of the delta rows of X's A values.  A workgroup
// owns the head rows X it visits: row X is staged in LDS, the
// candidates are tested and set there, and the words that changed are
// written back with plain stores, their new bits into X's next delta row.
// Rows are visited in a grid-stride loop.  Delta rows are bitmap rows of the
// head's layout with a per-row flag (nonzero: the row has bits); in_bits is
// only read (rows are shared by all X of one A) and cleared by
// clear_flagged_rows after the round.
struct GatherArgs {
  uint32_t* in_bits;        // [range0][row_words] this round's delta (by_a: emptied as read)
  uint32_t* in_flag;        // [range0]
  uint32_t* out_bits;       // [range0][row_words] next delta (zero on entry)
  uint32_t* out_flag;       // [range0] (zero on entry)
  uint32_t* bits;           // the head's membership bitmap
  IndexProbe e1;            // e1 indexed by its X column
  int32_t e1_acol;          // column of e1 holding A
  FrontierArgs push;        // the push expansion through e2: idx = e2 indexed by
                            // its B column, ybind_col = e2's Y column, lo0, lo1,
                            // row_words as below
  int32_t lo0, lo1;
  uint32_t row_words;
  int64_t range0;
  unsigned long long* counters;  // CNT_CANDIDATES, CNT_APPENDED
  // by_a: one workgroup per flagged delta row A instead of per head row X;
  // e1a is e1 indexed by its A column, e1_xcol the column holding X.  Every
  // delta row r keeps word bounds: its bits lie in words [lo[r], hi[r])
  // (empty: lo = row_words, hi = 0); the next round's bounds only widen.
  // The by_a kernel also empties each delta row it reads (its nonzero words,
  // its flag and its bounds), so no clearing pass follows the round.
  int32_t by_a;
  IndexProbe e1a;
  int32_t e1_xcol;
  uint32_t* in_lo;
  uint32_t* in_hi;
  uint32_t* out_lo;
  uint32_t* out_hi;
};


// Worst-case-optimal triangle join (count -> scan -> materialize).  Driver
// rows (x, y) come from a's index in (X, Y) order; b is indexed by its Y
// column and c by its X column, each with the rows of one key sorted by the
// Z value.  Work item k of driver row i (items of row crow[q] are
// [cofs[q], cofs[q + 1])) probes the k-th Z value of the shorter of b(y) and
// c(x) into the longer one by binary search; a hit is the triple (x, y, z).
// A wavefront handles WC_CHUNK consecutive items; items, and so the output,
// follow (row, k) order, which is ascending (x, y, z).
struct WcojArgs {
  const uint32_t* ax;       // [na] X of driver row i (a's index order)
  const uint32_t* ay;       // [na] Y of driver row i
  int64_t na;
  IndexProbe ib;            // b by its Y column
  const uint32_t* bz;       // b's Z column in ib's row order
  IndexProbe ic;            // c by its X column
  const uint32_t* cz;       // c's Z column in ic's row order
  int32_t probe_shorter;    // 1: probe the shorter list; 0: always b's (the binary-join order)
  uint32_t* work;           // [na] items of row i (work pass)
  const uint32_t* crow;     // [nz] driver rows with items, ascending
  const unsigned long long* cofs;  // [nz + 1] first item of each such row
  int64_t nz;
  unsigned long long items;
  uint32_t* chunk_cnt;      // count pass: hits per chunk
  const uint32_t* chunk_off;  // materialize pass: first output row per chunk
  uint32_t* out0;           // materialize pass: X, Y, Z columns
  uint32_t* out1;
  uint32_t* out2;
};

}  // namespace xlh
