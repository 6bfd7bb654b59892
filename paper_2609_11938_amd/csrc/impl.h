// Internal interfaces of libopattr: workspace plan and kernel launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/opattr.h"

namespace opa {

constexpr int kRangeTile = 1024;    // ranges per local-NPG tile
constexpr int kColChunk = 64;       // rows per chunk of the column scans
constexpr int kEncThreads = 256;    // threads per enclose/aggregate block
constexpr int kEncSpan = 2048;      // launches per enclose/aggregate block
constexpr int kEncRowsPerWave = 32; // runs a wave of that block reduces in place
constexpr int kEncWindow = 2048;    // range starts staged in LDS per block
// Default aggregation kinds (counter appendix table) as bit masks over the
// counters: MAX for the two per-kernel constants, SUM for the six additive
// counts (neither mask), DW-mean otherwise.
constexpr uint32_t kDefMaxMask = (1u << 17) | (1u << 19);
constexpr uint32_t kDefDwMask = 0x1BBF8u;
// Key counts ranked with per-wave LDS counters (8 bytes of LDS per key); the
// seq-tile kernels also hold a 16 KB partition array, hence a lower limit.
constexpr uint32_t kFastKeys = 6144;
constexpr uint32_t kFastNames = 4096;
constexpr int kMaxWalk = 300;       // bound on parent-chain walks (depth <= 255)
constexpr uint32_t kMaxNames = (1u << 20) - 1;  // names and rows are packed above a 12-bit slot
constexpr uint32_t kMaxOps = (1u << 20) - 2;    // rows = n_ops + 1
constexpr int kSumBlocks = 256;  // blocks of the summary's first pass over the table

// Byte offsets of every scratch array inside the caller's workspace.
struct Plan {
  int64_t T, P, R;
  uint32_t NN, NS, G, NP;
  int64_t nt, ntp, ncht, nchp, ntr_max, nencb, ntrt, nchr;
  bool seq_dense, ranges_nested;
  bool seg;  // seq tiles read from per-stream segments (kernels stream-major, seq dense)
  // opattr_attribute on dense seq in another order: the launches permuted
  // into stream-major order first, then the fused path (the sizes below and
  // the segment path's are taken; seg and fused stay false for the other
  // entry points, which read the launches as given)
  bool remap;
  size_t rm_hist, rm_perm, rm_inv, rm_seq, rm_name, rm_dur, rm_st, rm_start, rm_query, rm_part, rm_match,
      rm_rid;
  size_t total;
  // IOM
  size_t sv, rk, seqsort_k0, seqsort_k1, seqsort_v0, seqsort_v1, rs_hist, kblk, tbnd;
  size_t tlh, pfh, tlch, pfch, tlc, pfc, off, slot;
  size_t pfirst, plast, pheads, prec, mbs, nbs;
  size_t bcnt;  // bucket path: bucket size of every seq tile
  // fused attribution (segment path, sparse ranges, few rows): row
  // accumulators, kept partials (aliasing the partial rows of the other
  // aggregation), their bucket entries, and the per-bucket shares
  bool fused;
  size_t acc, fparts, fbkt, fsplit, forder, fhot;
  bool m2;  // the second set below exists
  size_t kblk2, tbnd2, tlh2, pfh2, tlch2, pfch2, tlc2, pfc2, off2, slot2, nbs2;
  // ranges
  size_t rperm, rs_c, re_c, rst_c, rop_c, rkd_c, rsort_k0, rsort_k1, rsort_v0, rsort_st;
  size_t ree, npg, mxv, rblk, tbase, tM, tnpg, tnpg2, tmx, tmx2, tfirst, tlast, sflag;
  size_t wfirst, wfused;  // per range with kinds: the walk's first op range and fused
  // aggregation
  int64_t cap_items, cap_rows, max_windows, hcap;
  size_t wi, wr, hmb, ig, ia, ib, rows, meta, ith, itch, gcnt, goff, heavy, multi, sit, part;
  size_t hch, hpart;
  size_t isort_k0, isort_k1, isort_v0, isort_v1, isort_hist;  // item sort, many rows
  // dedup class discovery
  size_t c_first, c_last, c_runs, c_key, c_cand, c_fail, c_list, c_tkey, c_tmin;
  size_t ident;    // 0 .. n_ops - 1 (aggregation by a given operator)
  size_t sumpart;  // per-block sums of the summary
  size_t misc;   // small device scalars
};

// second_match: also a second set of the segment path's matching arrays
Plan make_plan(const opattr_kernels *k, const opattr_profiled *p, const opattr_ranges *r,
               const opattr_dims *d, bool second_match = false);

// First HIP error of the calling host thread since the last reset; entry
// points report it as OPATTR_ERR_HIP.
inline thread_local hipError_t g_hip_error = hipSuccess;
inline void note(hipError_t e) {
  if (e != hipSuccess && g_hip_error == hipSuccess) g_hip_error = e;
}

// Probe events of the calling host thread (opattr_set_probe_events).
struct Probes {
  hipEvent_t ev[2 * OPATTR_NUM_PROBES];
  int n = 0;
};
inline thread_local Probes g_probes;
inline void probe_begin(int id, hipStream_t s) {
  if (id < g_probes.n && g_probes.ev[2 * id]) note(hipEventRecord(g_probes.ev[2 * id], s));
}
inline void probe_end(int id, hipStream_t s) {
  if (id < g_probes.n && g_probes.ev[2 * id + 1])
    note(hipEventRecord(g_probes.ev[2 * id + 1], s));
}

template <typename T>
inline T *at(void *ws, size_t off) {
  return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

// Core view of the ranges: nesting order per stream.
struct CoreRanges {
  int64_t n;
  const uint64_t *s;
  const uint64_t *e;
  const uint16_t *st;
  const uint32_t *op;
  const uint8_t *kind;  // range kinds of the walk; NULL = every range an op
  const int32_t *perm;  // core position -> input index; NULL = identity
};

// ---- radix sort (sort.hip) -------------------------------------------------
// Stable LSD sort of (key, value) pairs over bits [begin_bit, end_bit).
// Result ends in (k0, v0) when the pass count is even, else (k1, v1); returns
// true when the result is in k1/v1.
// Exclusive scan of in[0..n) into out (one block); *total_out = the sum.
void launch_scan_excl(const uint32_t *in, uint32_t *out, int64_t n, int64_t *total_out,
                      hipStream_t s);
// Exclusive prefix down each column of a [rows][cols] table in place, column
// totals in totals; rows_dev (optional) holds the actual row count on device.
void column_scan(uint32_t *tab, int64_t rows, uint32_t cols, uint32_t *chs, uint32_t *totals,
                 hipStream_t s, const int64_t *rows_dev);
// bits to hold the values 0..v (host)
inline int bits_for_host(uint32_t v) {
  int b = 1;
  while (b < 32 && (v >> b) != 0) ++b;
  return b;
}
// inclusive scan of n int64 values in place; scratch holds n / 4096 + 1 values
void scan_incl_i64_inplace(int64_t *a, int64_t n, int64_t *scratch, hipStream_t s);
// Stable LSD sort of (32-bit key, value) pairs by key bits [begin_bit,
// end_bit), 8 bits a pass; true when the result is in (k1, v1). n_dev
// (optional): the element count on the device (<= n); only that many are
// sorted
bool radix_sort_pairs(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, int64_t n,
                      int begin_bit, int end_bit, uint32_t *hist, hipStream_t s,
                      const int64_t *n_dev = nullptr);
size_t radix_hist_entries(int64_t n);
// Several 32-bit fills in one launch (up to 8 arrays).
struct FillJobs {
  static constexpr int kMaxJobs = 8;
  uint32_t *p[kMaxJobs];
  uint32_t v[kMaxJobs];
  int64_t n[kMaxJobs];
  int count = 0;
  void add(void *ptr, uint32_t value, int64_t words);
};
void fill_many(const FillJobs &j, hipStream_t s);
// Fill kernels (used instead of memset nodes, which misbehave under graph replay).
void fill_u32(uint32_t *p, uint32_t v, int64_t n, hipStream_t s);
void fill_u8(uint8_t *p, uint8_t v, int64_t n, hipStream_t s);
void launch_iota(uint32_t *v, int64_t n, hipStream_t s);
// k[i] = src[i], v[i] = i
void launch_key_pairs(const uint32_t *src, uint32_t *k, uint32_t *v, int64_t n, hipStream_t s);

// ---- IOM (iom.hip) -----------------------------------------------------------
// Per partition p, how its launches find their row:
//   hi == kRecEligible  p is its own class representative: its launches rank
//                       themselves;
//   hi == kRecNone      p has no valid representative: no row, no dedup error;
//   otherwise           a duplicate: the launch at seq rank x takes the row of
//                       the launch at x + delta when x < hi (the representative
//                       partition is shorter otherwise), else a dedup error;
//                       hi == 0 when either partition is not one run.
struct PartRec {
  int32_t delta;
  uint32_t hi;
};
constexpr uint32_t kRecEligible = 0xFFFFFFFFu, kRecNone = 0xFFFFFFFEu;

struct IomArgs {
  const opattr_kernels *k;
  const opattr_profiled *p;
  const opattr_dims *d;
  int policy;
  int32_t *match;
  uint32_t *name_counts;
  opattr_diag *diag;
  void *ws;
  const Plan *pl;
  bool want_dedup;  // also broadcast to duplicate partitions
  bool validate;
  // bucket path (segment plans only): stop at the eligible launches' rows
  // by seq rank (mbs, nbs); match is left to run_fused_agg
  bool buckets = false;
  // optional second stream for the profiled side, with the events that fork
  // it from and join it back to the main stream
  hipStream_t pf_stream = nullptr;
  hipEvent_t pf_fork = nullptr, pf_join = nullptr;
  // fused path: the run reduction's block order, computed on the profiled side
  bool fused_order = false;
};
void build_seq_view(const opattr_kernels *k, const opattr_dims *d, void *ws, const Plan &pl,
                    opattr_diag *diag, bool validate, hipStream_t s);
void run_match(const IomArgs &a, hipStream_t s);
// the launches of a remapped call in stream-major order (the launch-order
// view must be built): the permutation and the permuted arrays into the
// plan's rm_* regions; *out gets the arrays
void remap_launches(const opattr_kernels *k, const opattr_dims *d, void *ws, const Plan &pl,
                    opattr_kernels *out, hipStream_t s);
size_t remap_hist_entries(const Plan &pl);
// the permuted launch arrays' addresses (host only)
void remap_view(const opattr_kernels *k, void *ws, const Plan &pl, opattr_kernels *out);
// exclusive scan of a[0, n) in place; scratch holds scan_scratch_entries(n)
void scan_excl_inplace(uint32_t *a, int64_t n, uint32_t *scratch, hipStream_t s);
size_t scan_scratch_entries(int64_t n);
// match and range_id of the permuted launches back to the caller's order
void remap_back(void *ws, const Plan &pl, int32_t *match, int32_t *range_id, hipStream_t s);
// OPATTR_VALIDATE: check the kernels' stream-major promise (if given)
void check_kernel_layout(const opattr_kernels *k, const opattr_dims *d, opattr_diag *diag,
                         hipStream_t s);
// blk[s] = first index with st[i] >= s, s in [0, NS] (st sorted)
void launch_stream_blocks(const uint16_t *st, int64_t n, uint32_t NS, int64_t *blk,
                          hipStream_t s);
// Standalone dedup broadcast over a given match array (run_match already
// broadcasts when IomArgs::want_dedup is set).
void run_dedup(const opattr_kernels *k, const opattr_dims *d, int32_t *match, opattr_diag *diag,
               void *ws, const Plan &pl, hipStream_t s);
// every launch's counter row by its (broadcast) match: out[i][20], NaN for
// no row or an absent counter
void run_counters_out(const opattr_profiled *p, const int32_t *match, int64_t T, float *out,
                      hipStream_t s);

// ---- dedup class discovery (classes.hip) -----------------------------------------
// bits of the class key kept by the calling host thread (opattr_set_class_key_bits)
inline thread_local int g_class_key_bits = 64;
// slots of the key table for NP partitions (a power of two >= 2 NP)
int64_t class_table_slots(uint32_t NP);
// part_rep[NP] from the partitions' (name, stream) sequences in launch order;
// needs the launch-order view (build_seq_view)
void run_classes(const opattr_kernels *k, const opattr_dims *d, int32_t *part_rep,
                 opattr_diag *diag, void *ws, const Plan &pl, hipStream_t s);

// ---- tiered attribution (tiers.hip) ---------------------------------------------
struct TierIn {
  const opattr_kernels *k;
  const opattr_corr_map *corr;
  const opattr_fusion_map *fmap;
  const opattr_ranges *r;
  const opattr_dims *d;
  const int32_t *entry;  // correlation entry per launch (from the matching), or NULL
  const int32_t *range_id;
  const uint8_t *walk_fused;
  uint8_t *tier;
  int32_t *op;
  uint8_t *fused;
  opattr_coverage *cov;
  opattr_diag *diag;
  void *ws;
  const Plan *pl;
};
void run_tiers(const TierIn &x, hipStream_t s);
// per-dispatch row of every launch (see opattr_aggregate_dispatch)
void launch_dispatch_keys(const int32_t *range_id, const int32_t *op, const opattr_ranges *r,
                          uint32_t NOPS, int64_t T, int32_t *key, int32_t *row,
                          opattr_diag *diag, hipStream_t s);

// ---- ranges and enclosure (ranges.hip, enclose.hip) ----------------------------
// nesting order, validity, effective ends and stream blocks of the ranges,
// with the range stage's clears and the caller's extra clears (extra)
CoreRanges prepare_ranges(const opattr_ranges *r, const opattr_dims *d, void *ws, const Plan &pl,
                          opattr_diag *diag, bool validate, hipStream_t s,
                          const FillJobs *extra = nullptr);
// parents, crossing flags and depths (defer_depth: the enclosure pass writes
// the depths, EncArgs::depth)
void resolve_ranges(const CoreRanges &cr, const opattr_dims *d, void *ws, const Plan &pl,
                    uint8_t *range_depth, opattr_diag *diag, hipStream_t s,
                    bool defer_depth = false);
// words of the per-stream crossing flags (one byte per stream, whole words)
inline int64_t sflag_words(uint32_t NS) { return (int64_t)NS / 4 + 1; }
// all enclosing ranges per launch as CSR (off[T + 1] always, ids within cap)
void run_enclose_all(const CoreRanges &cr, const opattr_kernels *k, const opattr_dims *d, void *ws,
                     const Plan &pl, int64_t *off, int32_t *ids, int64_t cap, opattr_diag *diag,
                     hipStream_t s);
// range_parent[input index] = input index of the range's parent, -1 root / bad
void write_range_parents(const CoreRanges &cr, void *ws, const Plan &pl, int32_t *range_parent,
                         hipStream_t s);

struct PartRow;
struct AggIn;
// Items planned by the enclosure pass for the aggregation (see agg.hip).
struct EmitOut {
  uint32_t *wi, *wr;          // [waves] item / partial-row counts, then bases
  uint8_t *hmb;               // [blocks * threads] run starts among a thread's launches
  uint32_t *ig, *ia, *ib;     // item: row, partial-row index or first launch, 0 or length
  PartRow *rows;
  int64_t *meta;
};
EmitOut emit_out(void *ws, const Plan &pl);

struct EncArgs {
  uint8_t *fused = nullptr;      // walk outputs (enclosure), optional
  int32_t *range_any = nullptr;
  const opattr_kernels *k;
  const opattr_profiled *p;  // aggregation
  const int32_t *match;      // aggregation
  const opattr_ranges *r;    // input ranges (aggregate-only: op ids by input index)
  CoreRanges cr;             // enclosure
  const opattr_dims *d;
  int32_t *range_id;         // out (enclose) or in (aggregate-only)
  const uint8_t *agg_kind;   // host, 20 entries
  opattr_op_row *table;
  opattr_summary *sum;
  opattr_diag *diag;
  void *ws;
  const Plan *pl;
  bool depth = false;            // run_enclose also writes the range depths
  uint8_t *range_depth = nullptr;
};
AggIn agg_inputs(const EncArgs &x);
// range_id of every launch (Alg. 2)
void run_enclose(const EncArgs &a, hipStream_t s);
// the innermost range of every launch (core position, -1 for none), kinds
// not consulted; counts launches with bad stream ids
void launch_innermost(const CoreRanges &cr, const opattr_kernels *k, const opattr_dims *d,
                      void *ws, const Plan &pl, int32_t *core, opattr_diag *diag, hipStream_t s);
// The aggregation in four parts. Plan (no matches needed): per-wave item and
// row counts and their scan (with the enclosure when enclose is set), then
// the items and their sort by operator row. Reduction: the runs in place
// (needs the counts and the matches), then the per-row reduction of the
// sorted items (needs the runs and the sort).
void plan_counts(const EncArgs &a, bool enclose, hipStream_t s);
void plan_emit(const EncArgs &a, hipStream_t s);
void reduce_runs(const EncArgs &a, hipStream_t s);
// operator table from range_id and match: all four parts on one stream
void run_aggregate_all(const EncArgs &a, hipStream_t s);
// item sort by row (agg.hip), and the per-row reduction of the sorted items
void plan_items(const EncArgs &a, hipStream_t s);
// triaged: triage_rows already ran (on a stream joined before this one)
void reduce_items(const EncArgs &a, hipStream_t s, bool triaged = false);
void triage_rows(const EncArgs &a, hipStream_t s);

// ---- fused dedup broadcast and aggregation (fused.hip) ---------------------------
struct FusedIn {
  const opattr_kernels *k;
  const opattr_ranges *r;
  const opattr_dims *d;
  const int32_t *range_id;  // from the enclosure
  int32_t *match;           // out
  const AggIn *in;
  uint32_t absent;
  opattr_op_row *table;
  opattr_summary *sum;
  opattr_diag *diag;
  void *ws;
  const Plan *pl;
  bool ordered = false;  // run_fused_order filled the block order
};
// every launch's match (from the bucket path's mbs / nbs, with the dedup
// broadcast and its errors), the operator table from it and range_id, the
// summary and the final status (the row accumulators and the done count must
// be zero: fused_acc_clear)
void run_fused_agg(const FusedIn &x, hipStream_t s);
// the processing order of the run reduction's blocks (reads only seq)
void run_fused_order(const opattr_kernels *k, void *ws, const Plan &pl, hipStream_t s);
int64_t fused_agg_blocks(int64_t T);  // blocks of the run reduction
// the clear of the row accumulators and the done count, as a fill job
void fused_acc_clear(FillJobs &j, void *ws, const Plan &pl);
// workspace sizes of the fused aggregation
size_t fused_parts_bytes(int64_t T);
size_t fused_bkt_bytes(int64_t T);
size_t fused_split_bytes(uint32_t G);
size_t fused_hot_bytes();
size_t fused_acc_bytes(uint32_t G);
constexpr uint32_t kFusedMaxRows = 16384;  // rows the per-bucket LDS tables hold

// ---- finish (api.hip) ---------------------------------------------------------
// status of the diag record; with a table, also the summary over its G rows
// (rows below NOPS attributed)
// (with prepart > 0, part already holds that many blocks' summary sums)
void launch_finish(opattr_diag *diag, const uint8_t *sflag, uint32_t ns, hipStream_t s,
                   const opattr_op_row *table = nullptr, opattr_summary *sum = nullptr,
                   uint32_t G = 0, uint32_t NOPS = 0, unsigned long long *part = nullptr,
                   int prepart = 0);

}  // namespace opa
