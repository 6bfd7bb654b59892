/*
 * Oracle for the trace-attribution join: a plain, single-threaded CPU
 * implementation of what the join computes, written from the paper
 * ("Hardware-Attributed Operator Profiling for PyTorch").
 *
 * TEST INFRASTRUCTURE ONLY. Only the test-suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load this library. It shares no code,
 * header, table or helper with the GPU library.
 *
 * All pointers are host pointers. Every array is indexed by input position.
 * Functions return 0, or a negative value for an argument error.
 */
#ifndef OPATTR_ORACLE_H
#define OPATTR_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OREF_NC 20 /* the 20-counter set of the counter appendix table */

/* one timeline kernel record per index (nsys KernelRow, Alg. 1) */
typedef struct {
  int64_t n;
  const uint32_t *seq;      /* launch ordinal (CUPTI correlation order)          */
  const uint64_t *start_ns; /* GPU start time                                     */
  const uint32_t *dur_ns;   /* duration, the weight d_i of Eq. 1                  */
  const uint16_t *stream_id;
  const uint32_t *name_id;
  const int32_t *part_id;   /* layer partition instance, -1 none; NULL = none     */
  const uint64_t *query_ns; /* enclosure query point; NULL = start_ns             */
} oref_kernels;

/* profiled counter rows (ncu NcuRow), in replay order */
typedef struct {
  int64_t n;
  const uint32_t *name_id;
  const float *counters; /* value of counter c of row j at counters[j*rs + c*cs] */
  int64_t row_stride, col_stride;
  uint32_t absent_mask;  /* bit c: counter c absent for the whole capture        */
} oref_profiled;

/* operator ranges: closed intervals [start, end] on a stream (Alg. 2) */
typedef struct {
  int64_t n;
  const uint64_t *start_ns, *end_ns;
  const uint16_t *stream_id;
  const uint32_t *op_id;
  const uint8_t *kind; /* OREF_KIND_*; NULL = every range is an attributed op */
} oref_ranges;

/* Range kinds of the enclosure walk (Alg. 2): an attributed operator (an
   aten::, quantized:: or custom op range), a structural boundary (a range
   whose text has no namespace, e.g. a profiler step: the walk stops there),
   or a namespaced range that launches no kernel of its own (prims::,
   torch::: skipped). Other values make the range a bad record. */
enum { OREF_KIND_OP = 0, OREF_KIND_BOUNDARY = 1, OREF_KIND_SKIP = 2 };

typedef struct {
  uint32_t n_names, n_streams, n_ops, n_parts;
  const int32_t *part_rep; /* class representative of each partition; NULL = no dedup */
} oref_dims;

typedef struct {
  uint64_t kernel_count, total_ns, matched_count, matched_ns;
  double value[OREF_NC];
} oref_row;

typedef struct {
  uint64_t total_ns, attributed_ns, unattributed_ns, matched_ns;
  double attributed_fraction;
} oref_summary;

/* error classes, as bits of oref_diag.flags */
#define OREF_F_DATA 1u       /* an id out of range, or a range with start > end or
                                end >= 2^63 (such records are left out)          */
#define OREF_F_ORDER 2u      /* duplicate launch ordinal anywhere in the timeline */
#define OREF_F_LIMIT 4u      /* nesting deeper than 255                           */
#define OREF_F_NOT_NESTED 8u /* two ranges of a stream cross                      */
#define OREF_F_PARTITION 16u /* a partition is not one contiguous run of seq      */
#define OREF_F_DEDUP 32u     /* positional inheritance failed for some duplicate  */
#define OREF_F_COUNT 64u     /* per-name invocation counts differ                 */

/* status codes (highest precedence first when several classes are flagged) */
#define OREF_ERR_DATA (-9)
#define OREF_ERR_ORDER (-8)
#define OREF_ERR_LIMIT (-10)
#define OREF_ERR_NOT_NESTED (-5)
#define OREF_ERR_PARTITION (-7)
#define OREF_ERR_DEDUP (-6)
#define OREF_ERR_COUNT_MISMATCH (-4)
#define OREF_ERR_ARG (-1)

enum { OREF_PREFIX = 0, OREF_SKIP_NAME = 1, OREF_STRICT = 2 };
enum { OREF_SUM = 0, OREF_DWMEAN = 1, OREF_MAX = 2 };

typedef struct {
  int32_t status;
  uint32_t flags;
  uint32_t names_mismatched;
  uint32_t nesting_errors; /* streams whose ranges are not properly nested */
  uint64_t tl_unmatched, pf_unmatched, dedup_errors, bad_records;
} oref_diag;

void oref_diag_clear(oref_diag *d);
/* derive d->status from d->flags (STRICT makes COUNT an error) */
void oref_diag_finish(oref_diag *d, int policy);

int oref_match(const oref_kernels *k, const oref_profiled *p, const oref_dims *d,
               int policy, int32_t *match, uint32_t *name_counts, oref_diag *diag);
int oref_dedup(const oref_kernels *k, const oref_dims *d, int32_t *match,
               oref_diag *diag);
/* Counters inherited by position (Sec. 3.7): once the broadcast has given
   every duplicate its representative's match, each launch carries the counter
   row of the profiled row it is matched to. out[i*20 + c] = counter c of row
   match[i]; NaN when match[i] is outside [0, p->n) or counter c is absent. */
int oref_counters_out(const oref_profiled *p, const int32_t *match, int64_t n, float *out);
int oref_enclose(const oref_kernels *k, const oref_ranges *r, const oref_dims *d,
                 int32_t *range_id, uint8_t *range_depth, oref_diag *diag);
/* The full walk of Alg. 2. For each kernel, the ranges of its stream that
   contain its query point, innermost first, are walked outward: attributed
   ops are collected, skipped kinds passed over, and the walk stops at the
   first structural boundary. range_id = the first op collected (-1 none);
   fused = 1 when more than one op was collected; range_any = the innermost
   enclosing range of any kind (-1 none), from which range_parent (per range:
   the innermost range that contains it, -1 for a root or a bad range)
   leads through all enclosing ranges. Optional outputs may be NULL. Defined
   for properly nested ranges (NOT_NESTED is flagged otherwise). */
int oref_enclose_walk(const oref_kernels *k, const oref_ranges *r, const oref_dims *d,
                      int32_t *range_id, uint8_t *fused, int32_t *range_any,
                      int32_t *range_parent, uint8_t *range_depth, oref_diag *diag);
/* All enclosing ranges per kernel as CSR lists (Alg. 2's all_enclosing):
   ids[off[i] .. off[i+1]) = every valid range of the kernel's stream whose
   closed interval holds its query point, innermost first (reverse nesting
   order; kinds are not consulted). off has k->n + 1 entries and is always
   written; ids (capacity cap) receives the lists that end within cap. */
int oref_enclose_all(const oref_kernels *k, const oref_ranges *r, const oref_dims *d,
                     int64_t *off, int32_t *ids, int64_t cap, oref_diag *diag);
int oref_aggregate(const oref_kernels *k, const oref_profiled *p,
                   const int32_t *match, const int32_t *range_id,
                   const oref_ranges *r, const oref_dims *d, const uint8_t *agg_kind,
                   oref_row *table, oref_summary *sum, oref_diag *diag);
/* Eq. 1 with the operator row of each kernel given (op[i] in [0, n_ops), -1
   = UNATTRIBUTED; other values are bad records and go to UNATTRIBUTED). */
int oref_aggregate_ops(const oref_kernels *k, const oref_profiled *p, const int32_t *match,
                       const int32_t *op, const oref_dims *d, const uint8_t *agg_kind,
                       oref_row *table, oref_summary *sum, oref_diag *diag);

/* Per-dispatch table (the operators[] of profile.json, App. A.4): Eq. 1 by
   operator dispatch. Row rid (< r->n) collects the kernels of range rid
   whose operator (op[i], or the range's own op when op is NULL) is the
   range's op; row r->n + o the kernels attributed to operator o otherwise
   (no range, or a range of another operator); row r->n + n_ops the
   unattributed ones. table has r->n + n_ops + 1 rows; the summary counts
   the last row as unattributed. */
int oref_aggregate_dispatch(const oref_kernels *k, const oref_profiled *p, const int32_t *match,
                            const int32_t *range_id, const int32_t *op, const oref_ranges *r,
                            const oref_dims *d, const uint8_t *agg_kind, oref_row *table,
                            oref_summary *sum, oref_diag *diag);

/* Correlation map of the torch.profiler pass (Sec. 3.4): entry j says that
   one invocation of kernel name name_id[j] was launched by operator op_id[j]
   (-1: none recorded); the entries of a name are its invocation indices 0,
   1, ... in array order. */
typedef struct {
  int64_t n;
  const uint32_t *name_id;
  const int32_t *op_id;
} oref_corr;

/* Inductor fusion map (Sec. 3.6): for kernel name n, the operators fused
   into it are op_id[off[n] .. off[n+1]), the first one primary. off has
   n_names + 1 entries; a decreasing pair reads as an empty list. */
typedef struct {
  const uint32_t *off;
  const int32_t *op_id;
} oref_fusion;

/* Attribution tiers (Table "tiers", decision-tree figure). */
enum { OREF_TIER_UNATTRIBUTED = 0, OREF_TIER_HIGH = 1, OREF_TIER_NVTX = 2, OREF_TIER_FUSION = 3 };

/* kernels and nanoseconds per tier; frac = share of all kernel runtime (NaN
   when there is none) */
typedef struct {
  uint64_t count[4], ns[4];
  double frac[4];
} oref_coverage;

/* Tiered attribution. Per kernel, in order: HIGH when the correlation map
   has an entry with a valid operator for (name, invocation index), the index
   being the kernel's rank among all launches of its name in launch order
   (Alg. 1 over the map's entries under corr_policy; partitions play no
   part); NVTX when the enclosure walk found an op range (range_id, from
   oref_enclose_walk); FUSION when the fusion map lists operators for its
   name and the first is valid; else UNATTRIBUTED. op = the operator chosen
   (-1 for UNATTRIBUTED). fused = walk_fused (optional) or more than one
   operator listed for the name. corr and fm may be NULL. Map entries with
   an operator outside [-1, n_ops) and range ids outside [-1, r->n) are bad
   records. */
int oref_tiers(const oref_kernels *k, const oref_corr *corr, const oref_fusion *fm,
               const oref_ranges *r, const oref_dims *d, int corr_policy,
               const int32_t *range_id, const uint8_t *walk_fused, uint8_t *tier, int32_t *op,
               uint8_t *fused, oref_coverage *cov, oref_diag *diag);

/* Dedup class discovery (Sec. 3.7): partitions whose launches form the same
   sequence of (name, stream) in launch order are structural duplicates; each
   gets as representative the lowest-numbered partition of its class
   (part_rep[q], n_parts entries; d->part_rep is not read). Launches with a
   name or partition out of range take no part. A partition whose launches
   are not consecutive in launch order is its own class and raises
   PARTITION; equal seq values raise ORDER (ranks then tie by index).
   Partitions without launches share the empty sequence: one class. part_id
   is required when k->n > 0. */
int oref_dedup_classes(const oref_kernels *k, const oref_dims *d, int32_t *part_rep,
                       oref_diag *diag);

/* the four stages in order: match, dedup, enclose, aggregate */
int oref_attribute(const oref_kernels *k, const oref_profiled *p,
                   const oref_ranges *r, const oref_dims *d, int policy,
                   const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                   uint8_t *range_depth, uint32_t *name_counts, oref_row *table,
                   oref_summary *sum, oref_diag *diag);

#ifdef __cplusplus
}
#endif
#endif
