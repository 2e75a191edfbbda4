// Internal host-side structures of the fixpoint engine: workspace arena,
// context, relations, compiled programs and their per-rule join plans.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "../../include/xlh.h"
#include "device_types.h"

namespace xlh {

// ------------------------------------------------------------------ arena
// First-fit allocator over the caller's workspace.  Blocks are 256-byte
// aligned; freed neighbours coalesce.  Host-side bookkeeping only.
class Arena {
 public:
  void init(char* base, size_t size);
  void* alloc(size_t bytes);  // nullptr when no free block is large enough
  void release(void* p);
  size_t in_use() const { return in_use_; }
  size_t peak() const { return peak_; }
  void reset_peak() { peak_ = in_use_; }
  size_t capacity() const { return size_; }
  size_t largest_free() const;
  size_t block_size(const void* p) const;  // 0 for a pointer that is not a live block

 private:
  char* base_ = nullptr;
  size_t size_ = 0;
  std::map<size_t, size_t> free_;  // offset -> size
  std::map<size_t, size_t> used_;  // offset -> size
  size_t in_use_ = 0, peak_ = 0;
};

struct Program;

// Scalar types (xl_type values) and their stored int32 images: u32 and bool
// are stored as order-preserving int32 values, i64/u64/f64 as ranks in the
// context's dictionary of that type; f32 is stored as it is.
inline uint8_t phys_type(int ltype) { return ltype == XL_F32 ? T_F32 : T_I32; }
inline bool dict_type(int ltype) { return ltype == XL_I64 || ltype == XL_U64 || ltype == XL_F64; }
inline size_t elem_bytes(int ltype) { return ltype == XL_BOOL ? 1 : dict_type(ltype) ? 8 : 4; }
// Total-order key of an 8-byte value (the dictionary's sort key): i64 flips
// the sign bit, f64 follows IEEE 754 totalOrder, u64 is itself.
inline unsigned long long order_key64(unsigned long long bits, int ltype) {
  const unsigned long long sign = 1ull << 63;
  if (ltype == XL_I64) return bits ^ sign;
  if (ltype == XL_F64) return (bits & sign) ? ~bits : (bits | sign);
  return bits;
}
inline const char* type_name(int ltype) {
  static const char* n[] = {"?", "i32", "f32", "u32", "i64", "u64", "f64", "bool"};
  return ltype >= 1 && ltype <= 7 ? n[ltype] : n[0];
}

struct Relation {
  struct Context* ctx = nullptr;
  std::string name;
  int arity = 0;
  uint8_t ltypes[MAXC] = {};  // declared types (xl_type)
  uint8_t types[MAXC] = {};   // stored types (ValType of the int32 images)
  int64_t max_rows = 0;
  uint32_t* col[MAXC] = {};  // device columns (arena), nrows valid rows
  int64_t nrows = 0;
  int32_t lo[MAXC] = {}, hi[MAXC] = {};  // bounds of i32 columns when nrows > 0
  bool sorted = false;  // rows in ascending lexicographic order (as a load stores them)
  uint64_t generation = 0;  // new value (unique in the context) whenever the rows change
};

// An index of a relation kept across runs (option "index_cache_mb"): valid
// while the relation's generation is unchanged.  The blocks are arena memory
// owned by the cache.
struct CachedIndex {
  Relation* rel = nullptr;
  uint64_t generation = 0;
  int col = 0, order_col = -1, order_kind = 0;
  IndexProbe probe{};
  uint32_t* first = nullptr;
  std::vector<void*> blocks;
  size_t bytes = 0;
  uint64_t last_run = 0;
};

// The host control block (8192 bytes, pinned): control reads use its first
// CTL_CHECK_OFFSET bytes, the run's consistency flags its last word.
constexpr size_t CTL_BYTES = 8192;
constexpr size_t CTL_CHECK_OFFSET = CTL_BYTES - 64;

struct Context {
  int device = -1;
  hipStream_t stream = nullptr;
  Arena arena;
  std::string err;
  void* pinned = nullptr;                  // host control block
  unsigned long long* dcounters = nullptr; // device counters (arena)
  // internal consistency flags (arena word, CHECK_* bits) that kernels set
  // during a run; read once with the run's final synchronization
  unsigned long long* dcheck = nullptr;
  std::vector<Relation*> rels;
  std::vector<Program*> progs;
  int hash_min_log2 = 22;
  int index_mode = 0;
  int profile = 0;
  int pull_ratio = 64;
  int frontier_resident = 1;  // closure strata: 1 all rounds in one launch, 0 one launch per round
  int wcoj_shorter = 1;       // triangle joins: 1 probe the shorter list, 0 always b's (binary-join order)
  int product_joins = 1;      // two driver-keyed index steps in one launch (0: materialize between them)
  int batched_rounds = 4;     // tiled min/max strata: rounds per host read (0: one round at a time)
  int gather_rounds = 1;      // h(X,Y) :- e1(X,A), delta h(A,B), e2(Y,B): gathered rounds, 1 one
                              // workgroup per delta row A, 2 per head row X; 0 the generic join
  int dense_tiles = 0;  // tiled min/max rounds: 0 auto, k tiles per rank, -1 off
  int64_t control_bytes = 0;
  uint64_t generations = 0;      // source of Relation::generation values
  size_t index_cache_bytes = 0;  // budget of the cross-run index cache (0: off)
  uint64_t runs = 0;             // xl_fixpoint_run calls so far
  std::vector<CachedIndex> icache;
  // Dictionaries of the 8-byte types, indexed by xl_type: ascending distinct
  // total-order keys (arena blocks); a stored value is its key's rank.
  unsigned long long* dict[8] = {};
  int64_t dict_n[8] = {};
  // drop cached indexes of rel (all of them, or those of older generations)
  void icache_drop(const Relation* rel, bool stale_only) {
    for (size_t i = 0; i < icache.size();) {
      if (icache[i].rel == rel && (!stale_only || icache[i].generation != rel->generation)) {
        for (void* b : icache[i].blocks) arena.release(b);
        icache.erase(icache.begin() + (long)i);
      } else {
        ++i;
      }
    }
  }

  xl_status fail(xl_status st, const std::string& msg) {
    err = msg;
    return st;
  }
  Relation* find(const std::string& name) const {
    for (Relation* r : rels)
      if (r->name == name) return r;
    return nullptr;
  }
};

// ------------------------------------------------------------------ AST
enum class Agg { NONE, COUNT, SUM, MIN, MAX, LSE };

struct Term {
  enum Kind { VAR, ANON, INT, FLOAT } kind = ANON;
  std::string name;
  int64_t ival = 0;  // INT: the value (the low 64 bits when big)
  bool big = false;  // INT above the int64 range (a u64 value)
  double fval = 0.0;
};

struct AtomAst {
  std::string pred;
  std::vector<Term> args;
};

struct RuleAst {
  std::string head;
  std::vector<Term> head_args;  // key arguments (aggregate excluded)
  Agg agg = Agg::NONE;
  std::string agg_var;
  std::vector<AtomAst> atoms;
  std::vector<AtomAst> negs;  // literals "not q(...)" (stratified negation)
  struct Assign {
    std::string var;
    std::vector<std::pair<int, Term>> parts;  // (+1 / -1, term)
  };
  std::vector<Assign> assigns;
  struct Cmp {
    int op;
    Term lhs, rhs;
  };
  std::vector<Cmp> cmps;
  std::string text;
};

// ------------------------------------------------------------------ plans
struct NegPlan {         // a negated literal: the columns it constrains
  Relation* rel = nullptr;
  int ncols = 0;
  int col[2] = {0, 0};
};

// A constant of an 8-byte type in a plan.  Its stored image is the rank of
// the value in the context's dictionary, looked up when a run starts (a load
// between runs may renumber the dictionary).
struct WideConst {
  int8_t where;  // 0: driver_act[a].cval, 1: steps[a].act[b].cval, 2: stage_consts[a][b]
  uint8_t ltype;
  int16_t a, b;
  unsigned long long key;  // total-order key of the value
};

struct StepPlan {        // index join against a full relation
  Relation* rel = nullptr;
  int key_col = 0;
  int key_slot = 0;
  ColAct act[MAXC] = {};
};

struct RulePlan {
  int rule = 0;
  Relation* head = nullptr;
  Relation* driver = nullptr;   // relation scanned first
  bool driver_delta = false;    // scan the driver's delta instead of all rows
  ColAct driver_act[MAXC] = {};
  std::vector<StepPlan> steps;
  std::vector<NegPlan> negs;    // negated literals, referenced by OP_NOTIN ops
  // micro-ops executed by kernel stage k (k = max(0, #steps - 1) when no steps)
  std::vector<std::vector<MicroOp>> stage_ops;
  std::vector<std::vector<uint32_t>> stage_consts;
  std::vector<std::vector<int>> live_after;  // slots materialized after stage k
  std::vector<WideConst> wconsts;            // constants resolved per run
  int nkey = 0;
  int key_slot[2] = {0, 0};
  int val_slot = -1;
  uint8_t val_type = T_I32;
  // column -> (var slot or -1 for an is-result) binding source, for domains
  std::vector<std::pair<Relation*, int>> var_sources[MAXV];
  bool var_is_arith[MAXV] = {};
  // head(X, Y) :- delta head(X, Z), e(Z, Y) with nothing else: the first key
  // passes through from the delta, so the delta can be processed grouped by X.
  bool carried = false;
  int carried_ycol = -1;  // column of e bound to Y
  // head(S, Y, agg(P)) :- delta head(S, Z, P1), e(..Z..Y..), arithmetic and
  // comparisons: the first key passes through and Y comes from one column of
  // e, so a head key (s, y) can collect its contributions by scanning the
  // rows of e whose Y column is y (carried_ycol) against the delta.
  bool carried_val = false;
  int cv_slot_s = -1, cv_slot_z = -1, cv_slot_p = -1;  // P1's slot, -1 when unused
  // h(X, Y, Z) :- a(..X..Y..), b(..Y..Z..), c(..X..Z..) with three distinct
  // variables over binary int32 relations and nothing else (a triangle): a
  // worst-case-optimal join.  For each row (x, y) of a, the Z values of b's
  // rows with Y = y are intersected with those of c's rows with X = x.
  // driver = a; tri_a[0], tri_a[1] = a's X and Y columns; tri_b = b's Y and
  // Z columns; tri_c = c's X and Z columns (head order X, Y, Z).
  bool wcoj = false;
  Relation* tri_brel = nullptr;
  Relation* tri_crel = nullptr;
  int tri_a[2] = {0, 1}, tri_b[2] = {0, 1}, tri_c[2] = {0, 1};
};

struct HeadInfo {
  Relation* rel = nullptr;
  Agg agg = Agg::NONE;
};

struct Stratum {
  std::vector<Relation*> heads;
  bool recursive = false;
  std::vector<RulePlan> full;      // every rule, all atoms over full relations
  std::vector<RulePlan> variants;  // recursive strata: one per recursive atom
};

struct Program {
  Context* ctx = nullptr;
  std::vector<RuleAst> rules;
  std::vector<HeadInfo> heads;
  std::vector<Stratum> strata;
  Agg head_agg(const Relation* r) const {
    for (const HeadInfo& h : heads)
      if (h.rel == r) return h.agg;
    return Agg::NONE;
  }
  bool is_head(const Relation* r) const {
    for (const HeadInfo& h : heads)
      if (h.rel == r) return true;
    return false;
  }
};

// frontend.cpp
xl_status compile_program(Context* ctx, const char* text, Program** out);
std::string explain_program(const Program* p);

// engine.cpp
// h(X, Y) :- e1(X, A), delta h(A, B), e2(Y, B) with nothing else, e1 and e2
// binary relations outside the stratum: the shape of a gathered round.
struct GatherShape {
  int s1 = 0, s2 = 0;        // steps keyed by A (e1) and by B (e2)
  int x_col = 0, y_col = 0;  // e1's X column, e2's Y column
};
bool gather_shape(const RulePlan& p, GatherShape* g);
xl_status relation_load(Relation* r, const void* const* cols, int64_t n, int on_device);
xl_status relation_read(const Relation* r, void* const* cols, int64_t cap, int64_t* out_rows,
                        int on_device);
xl_status relation_clear(Relation* r);
xl_status run_program(Program* p, int64_t max_iterations, xl_fixpoint_stats* st);
void relation_free_storage(Relation* r);

const char* agg_name(Agg a);

}  // namespace xlh
