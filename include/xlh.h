/*
 * xlh -- semi-naive fixpoint evaluation of recursive Datalog rules on one
 * AMD Instinct MI355X (gfx950).  Plain C ABI: opaque handles, plain pointers
 * and sizes, no C++ or framework types.
 *
 * What is computed.  Relations are sets of typed tuples over int32 and
 * IEEE-754 binary32 columns (the paper's typed predicates, Sec. 3.1-3.2).
 * Rules use the paper's surface syntax (Sec. 3.1, 3.3, 3.5):
 *
 *     head(X, Y) :- body1(X, Z), body2(Z, Y), X != Y.
 *     dist(S, Y, min(D)) :- dist(S, Z, D1), edge(Z, Y, W), D is D1 + W.
 *
 * Body literals are atoms (variables, '_' or integer constants as arguments),
 * comparisons (!= == < <= > >=) and 'V is T (+|- T)*' arithmetic.  A head may
 * carry one aggregate -- count, sum, min, max, logsumexp -- in its last
 * position (Sec. 3.5).  xl_fixpoint_run evaluates the program stratum by
 * stratum; each recursive stratum runs semi-naive iteration (Sec. 4.1,
 * Algorithm 1): seed the delta from the rules, then repeatedly join the delta
 * against the full relations, project the head tuples, deduplicate or
 * aggregate them by key, take the difference with the full relation and
 * merge, until every delta is empty.
 *
 * Aggregates inside recursion go beyond the paper (its stratifier rejects
 * them, Sec. 3.5).  They are accepted as follows: min and max when each
 * recursive rule uses each recursive atom's value at most once, added into
 * the head's value (D is D1 + W, D is D1 + D2), and neither compares it nor
 * tests it in a negated literal (a monotone tropical product; the delta
 * holds keys that are new or strictly improved);
 * sum and logsumexp only when every recursive rule of the stratum is linear
 * (the delta of round k holds the fold of the contributions derived from the
 * delta of round k-1, and the full relation accumulates them -- finite only
 * when derivations are acyclic, otherwise the iteration cap is reached) and
 * carries the recursive atom's value through a semiring product: a
 * recursive sum takes that value unchanged (C is C1), a recursive logsumexp
 * that value plus other terms (P is P1 + W), and neither compares it or
 * tests it in a negated literal -- the forms for which accumulating the
 * rounds gives the naive fixpoint's values; count never.  Every other
 * recursive aggregate rule is XL_UNSUPPORTED at compile time.
 *
 * Memory.  The caller owns a device workspace and a HIP stream; the library
 * sub-allocates every relation, index, hash table and delta buffer from that
 * workspace and never allocates device memory of its own (it allocates one
 * small pinned host block per context for control reads).  Exceeding the
 * workspace is XL_RESOURCE_EXHAUSTED (Sec. 2.2: byte budget), exceeding a
 * relation's max_rows is XL_CAPACITY_EXCEEDED, reaching the iteration cap is
 * XL_CONVERGENCE_FAILURE.  There is no host fallback: every step of
 * evaluation runs in the library's HIP kernels.
 *
 * Threading.  Calls are blocking and a context must be used from one thread
 * at a time.  Every call returns an xl_status; out-parameters are written
 * only on XL_OK except where stated.  xl_last_error() describes the most
 * recent failure on a context.
 */
#ifndef XLH_H
#define XLH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    XL_OK = 0,
    XL_INVALID_ARGUMENT = 1,   /* null handle, bad size, wrong relation, ... */
    XL_TYPE_MISMATCH = 2,      /* a variable used at two column types (Sec. 3.2) */
    XL_UNSUPPORTED = 3,        /* a rule form outside the accepted subset */
    XL_RESOURCE_EXHAUSTED = 4, /* the workspace byte budget is exceeded (Sec. 2.2) */
    XL_CAPACITY_EXCEEDED = 5,  /* a fixed row capacity is exceeded (Sec. 2.2) */
    XL_CONVERGENCE_FAILURE = 6,/* the iteration cap was reached (Sec. 2.2, Alg. 1) */
    XL_DEVICE_ERROR = 7,       /* a HIP runtime call failed */
    XL_PARSE_ERROR = 8         /* the rule text does not parse */
} xl_status;

/*
 * Column types: the paper's scalar types (Sec. 3.2 "Type system") except
 * symbol.  Element sizes at the load/read boundary: XL_BOOL 1 byte (0 or 1),
 * XL_I32 / XL_U32 / XL_F32 4 bytes, XL_I64 / XL_U64 / XL_F64 8 bytes.
 * Values are equal when identical; order is signed for i32 and i64,
 * unsigned for u32 and u64, false < true, IEEE 754 totalOrder for f64
 * (so -0.0 < +0.0 and the two never join).  f32 keeps IEEE comparison and
 * equality.  Arithmetic (`is`), sum and logsumexp take i32 and f32 only.
 * Internally every column is 4 bytes: u32 and bool are stored as an
 * order-preserving int32 image; i64, u64 and f64 as ranks in a per-context
 * sorted dictionary of the distinct values loaded so far (8 bytes of
 * workspace per distinct value, never shrunk while the context lives; a load
 * that adds values renumbers the columns already stored, an O(rows) pass).
 */
typedef enum {
    XL_I32 = 1, XL_F32 = 2, XL_U32 = 3, XL_I64 = 4, XL_U64 = 5, XL_F64 = 6, XL_BOOL = 7
} xl_type;

typedef struct xl_context xl_context;
typedef struct xl_relation xl_relation;
typedef struct xl_program xl_program;

#define XL_MAX_ARITY 4
#define XL_STATS_ROUNDS 256

/*
 * Terminal receipt of one xl_fixpoint_run (the paper's bounded terminal
 * receipt, Sec. 4).  Always written by xl_fixpoint_run, also on failure.
 *   iterations       semi-naive passes over all recursive strata; the seed is
 *                    not a pass, the final pass that finds every delta empty is
 *   delta_rows[i]    rows in the delta after the i-th recorded round: for each
 *                    recursive stratum its seed then each pass; for each
 *                    non-recursive stratum the rows it produced (first
 *                    XL_STATS_ROUNDS rounds; rounds_recorded counts them all)
 *   candidates_total head tuples emitted by the join/project step, all rounds
 *   derived_tuples   final rows over all derived relations
 *   control_bytes_read  device->host bytes read to drive the loop
 *   ms_total         device time of the whole run (HIP events on the stream)
 */
typedef struct {
    int32_t status;
    int32_t iterations;
    int32_t strata;
    int32_t rounds_recorded;
    int64_t delta_rows[XL_STATS_ROUNDS];
    int64_t candidates_total;
    int64_t new_tuples_total;
    int64_t derived_tuples;
    int64_t peak_workspace_bytes;
    int64_t control_bytes_read;
    int64_t table_grows;
    int64_t index_builds;       /* join indexes built in this run */
    int64_t index_reuses;       /* join indexes taken from the cross-run cache */
    double ms_total;
    /* Fused join/insert kernels (set, min and max heads), timed with HIP
     * events on the context's stream when the "profile" option is 1. */
    double emit_ms;
    int64_t emit_launches;
    int64_t emit_source_rows;   /* delta or driver rows those launches read */
    int64_t emit_candidates;    /* head tuples they produced */
    int64_t emit_new;           /* keys they inserted (new or improved rows) */
    /* Frontier rounds of closure-shaped strata (one bitmap row per first key),
     * timed the same way. */
    double front_ms;
    int64_t front_launches;
    int64_t front_candidates;   /* edges examined: produced tuples when pushing,
                                   in-edges scanned when pulling */
    int64_t front_new;          /* tuples added */
    /* Segmented folds of carried sum / logsumexp rules over dense heads (each
     * marked key scans all its in-edges against the delta), timed the same
     * way. */
    double pull_ms;
    int64_t pull_launches;
    int64_t pull_candidates;    /* in-edges scanned */
    int64_t pull_new;           /* keys whose value was added or changed */
    /* Worst-case-optimal triangle joins: the probe passes (count and
     * materialize), timed the same way. */
    double wcoj_ms;
    int64_t wcoj_launches;
    int64_t wcoj_candidates;    /* probes: per driver row, the shorter list's length */
    int64_t wcoj_new;           /* triples produced */
    /* Gathered rounds of h(X,Y) :- e1(X,A), delta h(A,B), e2(Y,B) over dense
     * set heads (same generation's shape), timed the same way. */
    double gather_ms;
    int64_t gather_launches;
    int64_t gather_candidates;  /* head tuples produced (each X of a row times its Y union) */
    int64_t gather_new;         /* tuples added */
} xl_fixpoint_stats;

/*
 * Create a context on HIP device `device` that enqueues all work on
 * `hip_stream` (a hipStream_t, may be NULL for the null stream) and
 * sub-allocates from `workspace` (device memory of `workspace_bytes` bytes,
 * owned by the caller; it and the stream must outlive the context; the
 * library uses it from the first 256-byte boundary on, in blocks of whole
 * 256-byte units; at least 1 MiB, else XL_INVALID_ARGUMENT).
 * device = -1 creates a planning-only context: relations can be declared and
 * rules compiled (no device work), but loads and runs fail with
 * XL_INVALID_ARGUMENT.
 */
xl_status xl_context_create(int device, void* hip_stream, void* workspace,
                            size_t workspace_bytes, xl_context** out);

/*
 * Allocation-free variant of xl_context_create, for callers that cannot
 * allocate memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  The context sub-allocates from the
 * library's static device array of XL_STATIC_WORKSPACE_BYTES (64 MiB) on
 * `device` instead of a caller workspace, and keeps its control block in host
 * memory inside the handle instead of a pinned allocation; every GPU the
 * library runs on holds that array until the process ends.  Neither this
 * call nor any later call on the context calls hipMalloc, hipHostMalloc,
 * hipFree or another allocating routine (xl_fixpoint_run still creates two
 * HIP events per run, and four more with option "profile").  Work that does
 * not fit the array fails with XL_RESOURCE_EXHAUSTED and a message naming
 * the bytes asked for and the limit, as a too small workspace does.
 * The array is shared by every call on the device and keeps the last call's
 * contents (the library clears what must start at zero before each use), so
 * one such context may exist per device at a time: another
 * xl_context_create_static on that device returns XL_RESOURCE_EXHAUSTED until
 * the first is destroyed.  Calls on the context from several threads race,
 * as on any context.  XL_INVALID_ARGUMENT for a null `out` or a device
 * outside [0, 64); XL_DEVICE_ERROR if the device cannot be selected or the
 * array's device address cannot be taken.  No message is recorded for a
 * failed create (there is no context to hold it).
 */
#define XL_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
xl_status xl_context_create_static(int device, void* hip_stream, xl_context** out);

/*
 * Tunables (key, value):
 *   "hash_min_log2"   log2 of the smallest hash table (default 22)
 *   "index_mode"      0 = automatic, 1 = always open-addressing hash tables,
 *                     2 = prefer dense key-domain tables where they fit
 *   "profile"         1 = time the join kernels with HIP events (receipt
 *                     emit_*, front_*, pull_*, wcoj_*)
 *   "pull_ratio"      closure-shaped strata over dense heads: a source whose
 *                     delta row has d bits and u unreached targets with an
 *                     in-edge is expanded by pulling (scanning in-edges of the
 *                     unreached targets) when pull_ratio * d >= u; 0 = always
 *                     push (default 64)
 *   "index_cache_mb"  budget of a cache that keeps the join indexes of
 *                     relations that are not derived in the running stratum
 *                     (inputs, finished strata) across xl_fixpoint_run calls,
 *                     each valid until its relation's rows change (load,
 *                     clear, re-derivation), least recently used entries
 *                     evicted first (Sec. 4, runtime optimization: persistent
 *                     index manager); its blocks come from the workspace.
 *                     0 = off: every run builds its indexes (default)
 *   "frontier_resident"  closure-shaped strata over dense heads: 1 = every
 *                     pass in one launch, each source iterating its own rounds
 *                     with its row in LDS until its delta is empty, the pass
 *                     count and per-pass delta sizes read back once at the end
 *                     (default); 0 = one launch and one host read per pass
 *   "batched_rounds"  rounds of a tiled min/max stratum (see "dense_tiles"),
 *                     or of a sum/logsumexp stratum whose carried rule adds
 *                     or subtracts one column (segmented pull rounds),
 *                     enqueued per host read: every round takes its sizes
 *                     from device memory and reports its delta size to a
 *                     device array read once per batch; rounds past the
 *                     fixpoint change nothing (default 4; 0 = one round and
 *                     two host reads per pass; at most 64)
 *   "gather_rounds"   a recursive rule h(X,Y) :- e1(X,A), h(A,B), e2(Y,B)
 *                     with nothing else (same generation's shape) over a dense
 *                     set head runs gathered rounds: 1 = one workgroup per
 *                     delta row A builds the Y values of e2 for its B bits
 *                     once in LDS and ORs their nonzero words into the head
 *                     rows of A's X values (default); 2 = one workgroup per
 *                     head row X stages it in LDS and sets there the Y values
 *                     for the delta rows of its A values, writing back only
 *                     changed words; 0 = the generic join of each delta tuple
 *   "product_joins"   1 = a rule whose two join steps are both keyed by
 *                     variables of the driver row (into a set head) runs as
 *                     one launch over the product of the two match lists
 *                     (default); 0 = materialize the first step's bindings
 *   "wcoj_shorter"    triangle joins: 1 = probe each driver row's shorter Z
 *                     list into the longer (default); 0 = always probe b's
 *                     list (the candidate count of a binary join a x b)
 *   "dense_tiles"     rounds of a carried min/max rule over a dense head run
 *                     one workgroup per (first key, tile of second keys) with
 *                     the tile in LDS: 0 = choose the tile count (default),
 *                     k = k tiles per first key, -1 = untiled emission
 * XL_INVALID_ARGUMENT for an unknown key or value.
 */
xl_status xl_context_set_option(xl_context* ctx, const char* key, int64_t value);

/*
 * Declare relation `name` with `arity` columns of types `cols[0..arity)`.
 * max_rows bounds the rows it may hold (0 = bounded only by the workspace);
 * a load or a run that would exceed it fails with XL_CAPACITY_EXCEEDED.
 * The handle belongs to the context.
 */
xl_status xl_relation_create(xl_context* ctx, const char* name, int arity,
                             const xl_type* cols, int64_t max_rows, xl_relation** out);

/*
 * Replace the relation's contents with `nrows` rows given column-wise:
 * cols[j] points at nrows values of column j's type, packed at that type's
 * element size (host memory, or device memory when cols_on_device != 0).
 * The data is copied into the workspace; the pointers are only borrowed for
 * the call.  Duplicate rows are removed (relations are sets).  A bool byte
 * other than 0 or 1 is XL_INVALID_ARGUMENT (nothing is stored).  Returns
 * after the copy has completed.
 */
xl_status xl_relation_load(xl_relation* rel, const void* const* cols, int64_t nrows,
                           int cols_on_device);

/* Empty the relation (O(1); its storage returns to the workspace). */
xl_status xl_relation_clear(xl_relation* rel);

/* Number of rows currently held. */
xl_status xl_relation_size(const xl_relation* rel, int64_t* out_rows);

/*
 * Copy the relation out in canonical order: rows ascending lexicographically
 * by column, each column in its type's order (float32 by IEEE totalOrder).
 * cols[j] receives the j-th column at its type's element size (host or
 * device memory per cols_on_device) and must hold capacity_rows values.  If the relation has more rows, nothing is copied,
 * *out_rows is set to the number needed and XL_CAPACITY_EXCEEDED returned.
 */
xl_status xl_relation_read(const xl_relation* rel, void* const* cols, int64_t capacity_rows,
                           int64_t* out_rows, int cols_on_device);

/*
 * Compile rule text against the context's relations (every predicate must
 * have been declared with xl_relation_create).  Host-only work: parse, type
 * check, stratify (strongly connected components of the dependency graph),
 * derive the delta variants of recursive rules and plan each rule as a
 * pipeline of index joins.  XL_PARSE_ERROR, XL_TYPE_MISMATCH or
 * XL_UNSUPPORTED on failure, with the reason in xl_last_error().
 */
xl_status xl_rule_compile(xl_context* ctx, const char* rules_text, xl_program** out);

/*
 * Human-readable plan (strata, delta variants, join steps).  Writes at most
 * cap bytes including the terminating NUL; *needed receives the full size.
 */
xl_status xl_program_explain(const xl_program* prog, char* buf, size_t cap, size_t* needed);

/*
 * Evaluate the program to its fixpoint.  Set, min and max heads start from
 * their current contents (empty after xl_relation_clear; loaded rows act as
 * extra facts, so a loaded fixpoint is a resume point); count, sum and
 * logsumexp heads are recomputed from empty.  Relations that are not rule
 * heads are read only.
 * max_iterations caps the semi-naive passes of each recursive stratum;
 * reaching it returns XL_CONVERGENCE_FAILURE and leaves derived relations
 * unspecified.  out_stats (may be NULL) is written on success and failure.
 */
xl_status xl_fixpoint_run(xl_program* prog, int64_t max_iterations,
                          xl_fixpoint_stats* out_stats);

const char* xl_last_error(const xl_context* ctx);
const char* xl_status_string(xl_status status);

void xl_program_destroy(xl_program* prog);
void xl_relation_destroy(xl_relation* rel);
/* Destroys the context and every relation and program created on it. */
void xl_context_destroy(xl_context* ctx);

#ifdef __cplusplus
}
#endif

#endif /* XLH_H */
