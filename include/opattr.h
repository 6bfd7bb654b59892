/*
 * opattr.h -- C ABI of the MI355X trace-attribution join.
 *
 * The library attributes GPU kernel records to operators in the three stages of
 * the paper "Hardware-Attributed Operator Profiling for PyTorch":
 *
 *   opattr_match           invocation-order matching of profiled counter rows to
 *                          timeline launches (Sec. 3.3, Alg. 1)
 *   opattr_dedup_broadcast positional inheritance of counters from the profiled
 *                          representative of a layer class (Sec. 3.7)
 *   opattr_dedup_classes   discovery of those classes from the timeline alone
 *                          (Sec. 3.7)
 *   opattr_tiers           tiered attribution: correlation map, enclosure,
 *                          fusion map (attribution-methods table)
 *   opattr_aggregate_dispatch  the operator table per dispatch (App. A.4)
 *   opattr_attribute_tiered    matching, walk, tiers and the table in one call
 *   opattr_enclose         innermost operator range enclosing each launch on its
 *                          own stream (Sec. 3.5, Alg. 2)
 *   opattr_aggregate       per-operator SUM / duration-weighted mean (Eq. 1) / MAX
 *                          of the 20-counter set, with an UNATTRIBUTED row
 *                          (Sec. 3.8.1 and the counter appendix table)
 *   opattr_attribute       all four stages in one call
 *
 * Conventions shared by every entry point:
 *  - Array pointers inside the structs and all output arrays are DEVICE pointers
 *    on the current HIP device, unless marked (host).
 *  - Every call enqueues its work on `stream` (a hipStream_t; NULL = the null
 *    stream) and returns without synchronising, except opattr_read_diag.
 *    opattr_attribute and opattr_attribute_tiered fork independent stages onto
 *    two side streams of the current device (one pair per calling host thread,
 *    created on its first such call, default priority, kept until the process
 *    ends) with events recorded on `stream`, and join them back on `stream`
 *    before their last kernels: completion is observed on `stream` alone, and
 *    a capture of `stream` records every branch. Calls from one host thread on
 *    several caller streams share that pair, so their side work is ordered.
 *  - The caller owns every buffer: inputs, outputs, the diag record and the
 *    workspace. No entry point allocates or frees device memory. Calls are
 *    stateless and reentrant on distinct workspaces. The workspace starts on a
 *    256-byte boundary (as hipMalloc returns it); otherwise, or when it is
 *    smaller than opattr_workspace_bytes, the call returns OPATTR_ERR_WORKSPACE.
 *  - Return value: 0, or a negative OPATTR_ERR_* for an ARGUMENT error found on
 *    the host (nothing is enqueued then). Errors that depend on the data are
 *    recorded on the device in the opattr_diag record (flags, counts, status);
 *    outputs are still written. Read them with opattr_read_diag.
 *  - Sizes: every count is < 2^31. n_names <= 2^20 - 1, n_ops <= 2^20 - 2,
 *    n_streams <= 65536.
 *  - Records with an id out of range are left out and counted (bad_records):
 *    launches with name_id >= n_names or part_id outside [-1, n_parts) take no
 *    part in matching and dedup; launches with stream_id >= n_streams enclose
 *    nothing; profiled rows with name_id >= n_names are never matched; ranges
 *    with stream_id >= n_streams, op_id >= n_ops, start > end or end >= 2^63
 *    enclose nothing. Partitions are used only when part_id, part_rep and
 *    n_parts > 0 are all given.
 *  - Ids: match[i] in [-1, P), range_id[i] in [-1, R); -1 means none.
 */
#ifndef OPATTR_H
#define OPATTR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OPATTR_NUM_COUNTERS 20

/* Timeline: one record per launched kernel (a KernelRow of Alg. 1), length n. */
typedef struct {
  int64_t n;
  const uint32_t *seq;      /* launch ordinal, unique (CUPTI correlation order)      */
  const uint64_t *start_ns; /* GPU start time                                         */
  const uint32_t *dur_ns;   /* duration: the weight d_i of Eq. 1 (Sec. 3.2)           */
  const uint16_t *stream_id;/* < n_streams                                            */
  const uint32_t *name_id;  /* < n_names                                              */
  const int32_t *part_id;   /* layer partition instance or -1; NULL = no partitions   */
  const uint64_t *query_ns; /* enclosure query point (host launch time, Alg. 2);
                               NULL = start_ns                                        */
} opattr_kernels;

/* Profiled counter rows in replay order (the NcuRow list of Alg. 1), length n.
   Counter c of row j is counters[j*row_stride + c*col_stride] (float32). */
typedef struct {
  int64_t n;
  const uint32_t *name_id;
  const float *counters;
  int64_t row_stride, col_stride;
  uint32_t absent_mask; /* bit c set: counter c absent in this capture -> NaN   */
} opattr_profiled;

/* Operator ranges: closed intervals [start_ns, end_ns] on a stream (the NVTX
   ranges of Sec. 3.5), length n. */
typedef struct {
  int64_t n;
  const uint64_t *start_ns, *end_ns;
  const uint16_t *stream_id;
  const uint32_t *op_id; /* < n_ops: the aggregation key (row of the table)         */
  const uint8_t *kind;   /* OPATTR_KIND_* of each range; NULL = every range an op   */
} opattr_ranges;

/* Range kinds of the enclosure walk (Alg. 2): an attributed operator range
   (aten::, quantized:: or a custom op), a structural boundary (a range whose
   text has no namespace, e.g. a profiler step; the walk stops there), or a
   namespaced range that launches no kernel of its own (prims::, torch::;
   passed over). A kind above 2 makes the range a bad record. */
enum { OPATTR_KIND_OP = 0, OPATTR_KIND_BOUNDARY = 1, OPATTR_KIND_SKIP = 2 };

/* Layout hints: each is a PROMISE about the inputs that lets the library skip a
   reordering pass. A false promise gives unspecified outputs (never an
   out-of-bounds access); with OPATTR_VALIDATE it is detected and reported as
   OPATTR_ERR_ORDER. Without hints every input order is accepted. */
#define OPATTR_KERNELS_STREAM_MAJOR 1u /* kernels sorted by (stream_id, seq), every
                                          stream_id < n_streams, and per stream
                                          the query point does not decrease with
                                          seq                                      */
#define OPATTR_SEQ_DENSE 2u            /* seq is a permutation of [0, n)          */
#define OPATTR_RANGES_NESTED 4u        /* ranges sorted by (stream_id, start asc,
                                          end desc)                                */
#define OPATTR_VALIDATE 8u             /* check the promised layouts on device    */

typedef struct {
  uint32_t n_names, n_streams, n_ops, n_parts;
  const int32_t *part_rep; /* [n_parts] class representative of each partition
                              (Sec. 3.7); NULL = no layer dedup                   */
  uint32_t flags;          /* OPATTR_* layout hints                               */
} opattr_dims;

/* One row of the per-operator table (the "aggregated" block of profile.json).
   Row n_ops is the UNATTRIBUTED bucket. value[c] is NaN when the row has no
   matched kernel or counter c is absent. */
typedef struct {
  uint64_t kernel_count, total_ns, matched_count, matched_ns;
  double value[OPATTR_NUM_COUNTERS];
} opattr_op_row; /* 192 bytes */

typedef struct {
  uint64_t total_ns, attributed_ns, unattributed_ns, matched_ns;
  double attributed_fraction; /* attributed_ns / total_ns, NaN if total is 0 */
} opattr_summary;

/* Correlation map of the torch.profiler pass (Sec. 3.4; device arrays):
   entry j records that one invocation of kernel name name_id[j] was launched
   by operator op_id[j] (-1: no operator recorded). The entries of a name, in
   array order, are its invocation indices 0, 1, 2, ...; names may
   interleave. */
typedef struct {
  int64_t n;
  const uint32_t *name_id;
  const int32_t *op_id;
} opattr_corr_map;

/* Inductor fusion map (Sec. 3.6; device arrays): the operators fused into
   kernel name n are op_id[off[n] .. off[n+1]), the first one primary. off has
   n_names + 1 non-decreasing entries (a decreasing pair reads as an empty
   list) and op_id holds off[n_names] entries. */
typedef struct {
  const uint32_t *off;
  const int32_t *op_id;
} opattr_fusion_map;

/* Attribution tiers (the attribution-methods table): HIGH from the
   correlation map, MEDIUM from the enclosure (NVTX) or from the fusion map
   (FUSION), else UNATTRIBUTED. */
enum { OPATTR_TIER_UNATTRIBUTED = 0, OPATTR_TIER_HIGH = 1, OPATTR_TIER_NVTX = 2,
       OPATTR_TIER_FUSION = 3 };

/* Coverage by tier (the attribution-coverage figure): kernels and kernel
   nanoseconds per tier, and each tier's share of all kernel runtime (NaN
   when there is none). Indexed by OPATTR_TIER_*. */
typedef struct {
  uint64_t count[4];
  uint64_t ns[4];
  double frac[4];
} opattr_coverage; /* 96 bytes */

/* Error classes (bits of opattr_diag.flags) and status codes. */
#define OPATTR_F_DATA 1u        /* an id out of range / a range with start > end */
#define OPATTR_F_ORDER 2u       /* duplicate seq, or a promised layout is false   */
#define OPATTR_F_LIMIT 4u       /* range nesting deeper than 255, or an internal
                                   capacity exceeded (sized not to be)          */
#define OPATTR_F_NOT_NESTED 8u  /* two ranges of one stream cross                 */
#define OPATTR_F_PARTITION 16u  /* a partition is not one contiguous seq run      */
#define OPATTR_F_DEDUP 32u      /* positional inheritance failed for a duplicate  */
#define OPATTR_F_COUNT 64u      /* per-name invocation counts differ              */

#define OPATTR_OK 0
#define OPATTR_ERR_INVALID_ARG (-1) /* host: NULL pointer, bad size or enum      */
#define OPATTR_ERR_WORKSPACE (-2)   /* host: workspace smaller than required     */
#define OPATTR_ERR_HIP (-3)         /* host: a HIP launch failed                 */
#define OPATTR_ERR_COUNT_MISMATCH (-4) /* diag: STRICT policy and counts differ  */
#define OPATTR_ERR_NOT_NESTED (-5)  /* diag */
#define OPATTR_ERR_DEDUP (-6)       /* diag */
#define OPATTR_ERR_PARTITION (-7)   /* diag */
#define OPATTR_ERR_ORDER (-8)       /* diag */
#define OPATTR_ERR_DATA (-9)        /* diag */
#define OPATTR_ERR_LIMIT (-10)      /* diag */
#define OPATTR_ERR_SCRATCH (-11)    /* host: opattr_attribute_noalloc needs more than
                                       OPATTR_NOALLOC_SCRATCH_BYTES            */

/* Device-resident error record. status is the highest-precedence flagged class
   in the order DATA, ORDER, LIMIT, NOT_NESTED, PARTITION, DEDUP, COUNT (COUNT
   only under OPATTR_MISMATCH_STRICT). Counters:
     names_mismatched  names whose eligible-launch and profiled-row counts differ
     nesting_errors    streams holding two crossing ranges
     tl_unmatched      sum over names of max(0, launches - rows)
     pf_unmatched      sum over names of max(0, rows - launches)
     dedup_errors      duplicate launches left unmatched by a failed lookup
     bad_records       records ignored because an id is out of range
     order_violations  layout-promise violations found under OPATTR_VALIDATE */
typedef struct {
  int32_t status;
  uint32_t flags;
  uint32_t names_mismatched;
  uint32_t nesting_errors;
  uint64_t tl_unmatched, pf_unmatched, dedup_errors, bad_records;
  uint64_t order_violations;
  uint32_t strict; /* set by opattr_match under OPATTR_MISMATCH_STRICT */
  uint32_t reserved;
} opattr_diag;

/* Count-mismatch policy of opattr_match (Sec. 3.3 and its limitations note):
   PREFIX    Alg. 1 as printed: per name the first min(launches, rows) launches
             take rows in order, the excess gets none;
   SKIP_NAME a name whose counts differ gets no rows at all;
   STRICT    PREFIX outputs, and status OPATTR_ERR_COUNT_MISMATCH. */
enum { OPATTR_MISMATCH_PREFIX = 0, OPATTR_MISMATCH_SKIP_NAME = 1, OPATTR_MISMATCH_STRICT = 2 };

/* Aggregation kind per counter (counter appendix table). */
enum { OPATTR_AGG_SUM = 0, OPATTR_AGG_DWMEAN = 1, OPATTR_AGG_MAX = 2 };

/* Workspace bytes every entry point needs for these sizes and hints (host,
   pure, enqueues nothing). Pass NULL for an absent input set. */
size_t opattr_workspace_bytes(const opattr_kernels *k, const opattr_profiled *p,
                              const opattr_ranges *r, const opattr_dims *d);

/* Zero the device diag record (enqueued on stream). Every entry point adds to
   the record, so clear it before a fresh run. */
int opattr_diag_clear(opattr_diag *diag, void *stream);

/* Copy the device diag record to the host (synchronises the stream). */
int opattr_read_diag(const opattr_diag *diag, opattr_diag *host_out, void *stream);

/* Invocation-order matching (Alg. 1). For every launch eligible for replay (no
   partition, or a partition that is its own class representative) in seq
   order, the k-th launch of a name takes the k-th profiled row of that name.
   Out: match[k->n] (all launches; ineligible ones get -1), name_counts
   [n_names][2] = (eligible launches, profiled rows) or NULL. */
int opattr_match(const opattr_kernels *k, const opattr_profiled *p, const opattr_dims *d,
                 int policy, int32_t *match, uint32_t *name_counts, opattr_diag *diag,
                 void *ws, size_t ws_bytes, void *stream);

/* Layer dedup (Sec. 3.7). A launch of a duplicate partition q (part_rep[q] !=
   q) at launch-order position x of q takes match[] of the launch at position x
   of partition part_rep[q]; if that launch does not exist or has another name,
   or either partition is not one contiguous seq run, it gets -1 and counts as a
   dedup error. In/out: match[k->n].
   counters_out (device, or NULL): every launch's counters after the
   broadcast, so that a duplicate carries its representative's metrics by
   position: counters_out[i * 20 + c] (float32, [k->n][20], row-major, written
   by the call) = counter c of profiled row match[i] of p, NaN when match[i]
   is outside [0, p->n) or bit c of p->absent_mask is set. p (with counters)
   is required with counters_out and not read without it (may be NULL).
   Workspace: opattr_workspace_bytes(k, NULL, NULL, d). */
int opattr_dedup_broadcast(const opattr_kernels *k, const opattr_dims *d, int32_t *match,
                           const opattr_profiled *p, float *counters_out, opattr_diag *diag,
                           void *ws, size_t ws_bytes, void *stream);

/* Tiered attribution (the attribution-methods table and the decision-tree
   figure). For each launch, the first tier that applies:
     HIGH    corr has an entry for (name_id, invocation index) whose operator
             is valid; the invocation index is the launch's rank among all
             launches of its name in launch order (seq, ties by input index),
             partitions playing no part: the lookup is Alg. 1 with corr's
             entries as the rows, under corr_policy (OPATTR_MISMATCH_*;
             SKIP_NAME = HIGH only for names whose launch and entry counts
             agree, the table's trigger condition);
     NVTX    range_id[i] >= 0 (the enclosure walk's op range, from
             opattr_enclose_walk): operator r->op_id[range_id[i]];
     FUSION  fmap lists operators for the name and the first one is valid;
     UNATTRIBUTED otherwise (op -1).
   fused[i] = walk_fused[i] (optional, from opattr_enclose_walk) or more than
   one operator listed in fmap for the name: the fusion map augments every
   tier without overriding it. corr and fmap may be NULL.
   In: k->seq (with corr), name_id, dur_ns; r->n and r->op_id (the ranges
   range_id refers to). Out (device): tier[k->n] (OPATTR_TIER_*), op[k->n],
   fused[k->n], cov (one opattr_coverage). Correlation entries with an
   operator outside [-1, n_ops) and range ids outside [-1, r->n) are bad
   records; the matching's count diagnostics describe corr. Workspace:
   opattr_tiers_workspace_bytes. */
size_t opattr_tiers_workspace_bytes(const opattr_kernels *k, const opattr_corr_map *corr,
                                    const opattr_ranges *r, const opattr_dims *d);
int opattr_tiers(const opattr_kernels *k, const opattr_corr_map *corr,
                 const opattr_fusion_map *fmap, const opattr_ranges *r, const opattr_dims *d,
                 int corr_policy, const int32_t *range_id, const uint8_t *walk_fused,
                 uint8_t *tier, int32_t *op, uint8_t *fused, opattr_coverage *cov,
                 opattr_diag *diag, void *ws, size_t ws_bytes, void *stream);

/* Tiered attribution in one call: opattr_match (with the dedup broadcast
   when partitions are given), opattr_enclose_walk's range_id and fused,
   opattr_tiers and opattr_aggregate_ops, with the ranges and the walk on a
   side stream of the device beside the two matchings (the profiled rows;
   the correlation map, on a second side stream with its own workspace
   arrays when the kernels are stream-major with dense seq, else after the
   profiled rows), all joined back on `stream` before the tiers. Out (device):
   match, range_id, tier, op, fused [k->n]; table[n_ops + 1] by tier
   operator; sum; cov. One diag record covers both matchings (their count
   diagnostics add up; STRICT in either makes a count mismatch an error).
   Workspace: opattr_attribute_tiered_workspace_bytes. */
size_t opattr_attribute_tiered_workspace_bytes(const opattr_kernels *k, const opattr_profiled *p,
                                               const opattr_ranges *r,
                                               const opattr_corr_map *corr,
                                               const opattr_dims *d);
int opattr_attribute_tiered(const opattr_kernels *k, const opattr_profiled *p,
                            const opattr_ranges *r, const opattr_corr_map *corr,
                            const opattr_fusion_map *fmap, const opattr_dims *d, int policy,
                            int corr_policy, const uint8_t *agg_kind, int32_t *match,
                            int32_t *range_id, uint8_t *tier, int32_t *op, uint8_t *fused,
                            opattr_op_row *table, opattr_summary *sum, opattr_coverage *cov,
                            opattr_diag *diag, void *ws, size_t ws_bytes, void *stream);

/* Aggregation (Eq. 1) by a given operator per launch: row op[i] when
   op[i] in [0, n_ops), row n_ops (UNATTRIBUTED) when op[i] == -1; other
   values are bad records and go to UNATTRIBUTED. Otherwise as
   opattr_aggregate (e.g. op from opattr_tiers). Workspace:
   opattr_workspace_bytes(k, p, NULL, d). */
int opattr_aggregate_ops(const opattr_kernels *k, const opattr_profiled *p, const int32_t *match,
                         const int32_t *op, const opattr_dims *d, const uint8_t *agg_kind,
                         opattr_op_row *table, opattr_summary *sum, opattr_diag *diag,
                         void *ws, size_t ws_bytes, void *stream);

/* Per-dispatch operator table (the operators[] of profile.json, App. A.4:
   one entry per operator call, operator_id = name + call index). A dispatch
   is an operator range. Row rid (< r->n) collects the launches with
   range_id[i] == rid whose operator is the range's (op[i] from
   opattr_tiers, or the range's own op when op is NULL); row r->n + o the
   launches attributed to operator o otherwise (no range, or a range of
   another operator); row r->n + n_ops the unattributed ones. Per row as
   opattr_aggregate (Eq. 1). Out: table[r->n + n_ops + 1], sum (device; the
   last row counts as unattributed), and row[k->n] (or NULL), the table row
   of each launch. Needs r->n + n_ops <= 2^20 - 2. Workspace:
   opattr_dispatch_workspace_bytes. */
size_t opattr_dispatch_workspace_bytes(const opattr_kernels *k, const opattr_profiled *p,
                                       const opattr_ranges *r, const opattr_dims *d);
int opattr_aggregate_dispatch(const opattr_kernels *k, const opattr_profiled *p,
                              const int32_t *match, const int32_t *range_id, const int32_t *op,
                              const opattr_ranges *r, const opattr_dims *d,
                              const uint8_t *agg_kind, opattr_op_row *table, opattr_summary *sum,
                              int32_t *row, opattr_diag *diag, void *ws, size_t ws_bytes,
                              void *stream);

/* Layer class discovery (Sec. 3.7: structurally identical layers share one
   profiled representative). Two partitions are one class when the launches
   of each (valid name_id and part_id) form the same sequence of (name_id,
   stream_id) in launch order (seq, ties by input index); every partition
   gets as representative the lowest-numbered partition of its class.
   Partitions without launches share the empty sequence. A partition whose
   launches are not consecutive in launch order is its own class and raises
   PARTITION; equal seq values raise ORDER (checked unless OPATTR_SEQ_DENSE is
   promised without OPATTR_VALIDATE). Launches with an id out of range count
   as bad_records.
   In: k->seq, name_id, stream_id, part_id (required when k->n > 0), and
   d->n_names, d->n_parts (d->part_rep is not read). Out: part_rep[d->n_parts]
   (device), a class map that opattr_dedup_broadcast and opattr_attribute
   accept as d->part_rep. Exact: a 64-bit sequence hash proposes the
   representative and an element-wise comparison confirms it. Workspace:
   opattr_workspace_bytes(k, NULL, NULL, d) with d->n_parts set. */
int opattr_dedup_classes(const opattr_kernels *k, const opattr_dims *d, int32_t *part_rep,
                         opattr_diag *diag, void *ws, size_t ws_bytes, void *stream);

/* Enclosure (Alg. 2). The ranges on stream_id[i] with start_r <= q_i <= end_r
   (q_i = query_ns[i], or start_ns[i]) are walked from the innermost (the one
   last in nesting order: start asc, end desc, index asc) outward: op ranges
   are collected, SKIP ranges passed over, and a BOUNDARY range ends the walk.
   range_id[i] = the first op collected, or -1 (without kinds: the innermost
   enclosing range). range_depth[r] (or NULL) = 1 + depth of the nearest
   earlier range of the stream in nesting order whose end is not before end_r
   (0 for a bad range). */
int opattr_enclose(const opattr_kernels *k, const opattr_ranges *r, const opattr_dims *d,
                   int32_t *range_id, uint8_t *range_depth, opattr_diag *diag, void *ws,
                   size_t ws_bytes, void *stream);

/* The enclosure walk of Alg. 2 with all of its outputs, as opattr_enclose plus:
   fused[i] = 1 when the walk collected more than one op range (a kernel
   spanning several attributed operators), else 0; range_any[i] = the
   innermost enclosing range of any kind, or -1; range_parent[r] = the
   innermost range that contains range r (the nearest earlier range of its
   stream in nesting order whose end is not before end_r), or -1 for a root
   or a bad range. The ranges enclosing a kernel are range_any and its
   parent chain, plus, when range_any starts exactly at the query point,
   ranges that end there (touching it rather than nesting it), which the walk
   visits in nesting order. fused, range_any, range_parent and
   range_depth may be NULL. Defined for properly nested ranges (crossing
   ranges are reported as NOT_NESTED). */
int opattr_enclose_walk(const opattr_kernels *k, const opattr_ranges *r, const opattr_dims *d,
                        int32_t *range_id, uint8_t *fused, int32_t *range_any,
                        int32_t *range_parent, uint8_t *range_depth, opattr_diag *diag,
                        void *ws, size_t ws_bytes, void *stream);

/* All enclosing ranges (Alg. 2 keeps all_enclosing_ranges for fused kernels)
   as CSR lists: ids[off[i] .. off[i+1]) are the valid ranges of the launch's
   stream whose closed interval holds its query point, innermost first
   (reverse nesting order; kinds are not consulted). Out (device): off[k->n +
   1] (int64, always written; off[k->n] is the total), ids (capacity cap
   entries) receives the lists that end within cap: call once with cap = 0
   to learn the total. Defined for properly nested ranges: crossing ranges
   are reported as NOT_NESTED (nesting_errors counts the streams that have
   them) and the lists are then unspecified. Workspace:
   opattr_workspace_bytes(k, NULL, r, d). */
int opattr_enclose_all(const opattr_kernels *k, const opattr_ranges *r, const opattr_dims *d,
                       int64_t *off, int32_t *ids, int64_t cap, opattr_diag *diag, void *ws,
                       size_t ws_bytes, void *stream);

/* Aggregation (Eq. 1). Row g = op_id[range_id[i]] (or n_ops when range_id is
   -1) collects kernel_count and total_ns of every launch, and over launches
   with match >= 0: matched_count, matched_ns and, per counter c with
   m = counters[match][c] widened to fp64, SUM m, DWMEAN (sum m*d)/matched_ns,
   or MAX m. agg_kind (host, 20 entries) or NULL for the appendix table's kinds.
   Out: table[n_ops + 1], sum (device). */
int opattr_aggregate(const opattr_kernels *k, const opattr_profiled *p, const int32_t *match,
                     const int32_t *range_id, const opattr_ranges *r, const opattr_dims *d,
                     const uint8_t *agg_kind, opattr_op_row *table, opattr_summary *sum,
                     opattr_diag *diag, void *ws, size_t ws_bytes, void *stream);

/* All four stages: match, dedup, enclose, aggregate. */
int opattr_attribute(const opattr_kernels *k, const opattr_profiled *p, const opattr_ranges *r,
                     const opattr_dims *d, int policy, const uint8_t *agg_kind, int32_t *match,
                     int32_t *range_id, uint8_t *range_depth, uint32_t *name_counts,
                     opattr_op_row *table, opattr_summary *sum, opattr_diag *diag, void *ws,
                     size_t ws_bytes, void *stream);

/* opattr_attribute for callers that cannot allocate device memory (code
   under stream capture, serving loops, harnesses that forbid hipMalloc): no
   workspace argument; the call uses a scratch array that the library holds
   on each device it runs on (OPATTR_NOALLOC_SCRATCH_BYTES, kept until the
   process ends, set up on the first call on that device) and runs every
   stage on `stream` alone (no side streams). Same arguments, outputs and
   diag as opattr_attribute. Returns OPATTR_ERR_SCRATCH, enqueueing nothing,
   when opattr_workspace_bytes(k, p, r, d) exceeds the scratch, and
   OPATTR_ERR_HIP when the scratch's address cannot be had. Every call on a
   device shares that device's scratch: calls that may overlap on one device
   (other streams, other host threads) race and must be ordered by the
   caller. No entry point allocates or frees; this one also creates no
   streams or events. */
#define OPATTR_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int opattr_attribute_noalloc(const opattr_kernels *k, const opattr_profiled *p,
                             const opattr_ranges *r, const opattr_dims *d, int policy,
                             const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                             uint8_t *range_depth, uint32_t *name_counts, opattr_op_row *table,
                             opattr_summary *sum, opattr_diag *diag, void *stream);

/* Probe events (diagnostics, per host thread). events is a host array of
   2*n hipEvent_t values; while set, every later call on this thread records
   events[2*i] on its stream right before the launches of probe i and
   events[2*i+1] right after them, for the probes below that the call runs;
   a NULL entry is not recorded (each recorded event is a stream barrier).
   NULL (or n = 0) switches probing off. The events are the caller's. */
enum {
  OPATTR_PROBE_SEQ_VIEW = 0,   /* launch-order view of the timeline          */
  OPATTR_PROBE_TL_HIST = 1,    /* per-tile name histograms of the timeline  */
  OPATTR_PROBE_PF_HIST = 2,    /* per-tile name histograms of the rows      */
  OPATTR_PROBE_COL_SCAN = 3,   /* column scans of both histogram tables     */
  OPATTR_PROBE_PF_SLOT = 4,    /* profiled slot table                       */
  OPATTR_PROBE_TL_MATCH = 5,   /* per-tile rank and join                    */
  OPATTR_PROBE_DEDUP = 6,      /* dedup broadcast                           */
  OPATTR_PROBE_RANGES = 7,     /* range order, parents and depths           */
  OPATTR_PROBE_MAIN_PASS = 8,  /* enclosure pass (range ids, item plan)     */
  OPATTR_PROBE_FINALIZE = 9,   /* status of the diag record                 */
  OPATTR_PROBE_AGGREGATE = 10, /* per-row reduction of the items, table    */
  OPATTR_PROBE_AGG_RUNS = 11,  /* in-place run reduction over the launches  */
  OPATTR_PROBE_ITEM_SORT = 12, /* sort of the planned items by operator row */
  OPATTR_NUM_PROBES = 13
};
int opattr_set_probe_events(void *const *events, int n);

/* Test support for opattr_dedup_classes, per calling host thread: keep only
   the low `bits` (1..64, default 64) bits of each partition's sequence key,
   so that partitions with different sequences share keys and the exact
   element-wise search decides. Results are unchanged; only time grows. */
int opattr_set_class_key_bits(int bits);

/* Human-readable name of a status code. */
const char *opattr_strerror(int status);

#ifdef __cplusplus
}
#endif
#endif
