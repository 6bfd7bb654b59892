/*
 * Oracle for the trace-attribution join (test infrastructure only; see the
 * header). Plain single-threaded C: every stage is the paper's definition
 * written out with sorting and stacks, no blocking, fusion or reordering.
 *
 *   match     -- invocation-order matching, Alg. 1 (Sec. 3.3)
 *   dedup     -- positional inheritance from the class representative (Sec. 3.7)
 *   enclose   -- innermost enclosing range at the query point (Alg. 2, Sec. 3.5)
 *   aggregate -- per-operator SUM / duration-weighted mean (Eq. 1) / MAX
 *                (Sec. 3.8.1 and the counter appendix table)
 */
#include "opattr_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ----------------------------------------------------------------------- */
/* small helpers                                                            */
/* ----------------------------------------------------------------------- */

typedef struct {
  uint64_t a, b, c; /* sort key, most significant first */
  int64_t idx;      /* last tie-break: input index */
} key3;

static int cmp_key3(const void *x, const void *y) {
  const key3 *p = (const key3 *)x, *q = (const key3 *)y;
  if (p->a != q->a) return p->a < q->a ? -1 : 1;
  if (p->b != q->b) return p->b < q->b ? -1 : 1;
  if (p->c != q->c) return p->c < q->c ? -1 : 1;
  if (p->idx != q->idx) return p->idx < q->idx ? -1 : 1;
  return 0;
}

static void *xcalloc(size_t n, size_t sz) { return calloc(n ? n : 1, sz); }

static int cmp_u32(const void *x, const void *y) {
  uint32_t a = *(const uint32_t *)x, b = *(const uint32_t *)y;
  return a < b ? -1 : (a > b);
}

void oref_diag_clear(oref_diag *d) { memset(d, 0, sizeof(*d)); }

void oref_diag_finish(oref_diag *d, int policy) {
  uint32_t f = d->flags;
  int32_t s = 0;
  if (f & OREF_F_DATA) s = OREF_ERR_DATA;
  else if (f & OREF_F_ORDER) s = OREF_ERR_ORDER;
  else if (f & OREF_F_LIMIT) s = OREF_ERR_LIMIT;
  else if (f & OREF_F_NOT_NESTED) s = OREF_ERR_NOT_NESTED;
  else if (f & OREF_F_PARTITION) s = OREF_ERR_PARTITION;
  else if (f & OREF_F_DEDUP) s = OREF_ERR_DEDUP;
  else if ((f & OREF_F_COUNT) && policy == OREF_STRICT) s = OREF_ERR_COUNT_MISMATCH;
  d->status = s;
}

/* a kernel takes part in matching and dedup only if its name and partition
   ids are in range */
static int dedup_on(const oref_kernels *k, const oref_dims *d) {
  return k->part_id && d->part_rep && d->n_parts > 0;
}

static int kernel_ok(const oref_kernels *k, const oref_dims *d, int64_t i) {
  if (k->name_id[i] >= d->n_names) return 0;
  if (dedup_on(k, d)) {
    int32_t p = k->part_id[i];
    if (p < -1 || (p >= 0 && (uint32_t)p >= d->n_parts)) return 0;
  }
  return 1;
}

static int32_t part_of(const oref_kernels *k, const oref_dims *d, int64_t i) {
  return dedup_on(k, d) ? k->part_id[i] : -1;
}

static int rep_ok(const oref_dims *d, int32_t p) {
  int32_t r = d->part_rep[p];
  return r >= 0 && (uint32_t)r < d->n_parts;
}

/* Eligibility for replay: kernels outside any partition, and kernels of a
   class representative; structural duplicates are skipped in replay
   (Sec. 3.7). */
static int eligible(const oref_kernels *k, const oref_dims *d, int64_t i) {
  if (!kernel_ok(k, d, i)) return 0;
  int32_t p = part_of(k, d, i);
  if (p < 0) return 1;
  return rep_ok(d, p) && d->part_rep[p] == p;
}

/* ----------------------------------------------------------------------- */
/* Stage 1: invocation-order matching (Alg. 1, Sec. 3.3)                    */
/* ----------------------------------------------------------------------- */

int oref_match(const oref_kernels *k, const oref_profiled *p, const oref_dims *d,
               int policy, int32_t *match, uint32_t *name_counts, oref_diag *diag) {
  if (!k || !p || !d || !match || !diag || k->n < 0 || p->n < 0) return OREF_ERR_ARG;
  if (k->n > 0 && (!k->seq || !k->name_id)) return OREF_ERR_ARG;
  if (p->n > 0 && !p->name_id) return OREF_ERR_ARG;
  if (policy < 0 || policy > 2) return OREF_ERR_ARG;
  const int64_t T = k->n, P = p->n;
  const uint32_t NN = d->n_names;

  /* bad records: ids out of range are counted and left out */
  for (int64_t i = 0; i < T; ++i)
    if (!kernel_ok(k, d, i)) diag->bad_records++;
  for (int64_t j = 0; j < P; ++j)
    if (p->name_id[j] >= NN) diag->bad_records++;
  if (dedup_on(k, d))
    for (uint32_t q = 0; q < d->n_parts; ++q)
      if (!rep_ok(d, (int32_t)q)) diag->bad_records++;

  /* ncu_rows[name]: profiled rows of each name in replay order, which is the
     per-name invocation index order required by Alg. 1 */
  int64_t *pf_cnt = xcalloc(NN, sizeof(int64_t));
  int64_t *pf_off = xcalloc((size_t)NN + 1, sizeof(int64_t));
  for (int64_t j = 0; j < P; ++j)
    if (p->name_id[j] < NN) pf_cnt[p->name_id[j]]++;
  for (uint32_t n = 0; n < NN; ++n) pf_off[n + 1] = pf_off[n] + pf_cnt[n];
  int64_t *rows = xcalloc((size_t)pf_off[NN], sizeof(int64_t));
  int64_t *fill = xcalloc(NN, sizeof(int64_t));
  for (int64_t j = 0; j < P; ++j) {
    uint32_t n = p->name_id[j];
    if (n < NN) rows[pf_off[n] + fill[n]++] = j;
  }

  /* timeline kernels eligible for replay, in launch (seq) order */
  key3 *ord = xcalloc((size_t)T, sizeof(key3));
  int64_t ne = 0;
  for (int64_t i = 0; i < T; ++i) {
    match[i] = -1;
    if (eligible(k, d, i)) {
      ord[ne].a = k->seq[i];
      ord[ne].b = ord[ne].c = 0;
      ord[ne].idx = i;
      ne++;
    }
  }
  qsort(ord, (size_t)ne, sizeof(key3), cmp_key3);
  /* launch ordinals must be unique over the whole timeline */
  {
    uint32_t *all = xcalloc((size_t)T, sizeof(uint32_t));
    for (int64_t i = 0; i < T; ++i) all[i] = k->seq[i];
    qsort(all, (size_t)T, sizeof(uint32_t), cmp_u32);
    for (int64_t x = 1; x < T; ++x)
      if (all[x] == all[x - 1]) { diag->flags |= OREF_F_ORDER; break; }
    free(all);
  }

  /* The matching of Alg. 1 as a definition: the launch of rank r among the
     eligible launches of its name, in launch order, takes that name's
     profiled row of rank r (replay order); a name with fewer rows than
     launches leaves its launches of rank >= its row count unmatched.
     tl_cnt[name] ends as the name's launch count. */
  int64_t *tl_cnt = xcalloc(NN, sizeof(int64_t));
  for (int64_t x = 0; x < ne; ++x) {
    const int64_t i = ord[x].idx;
    const uint32_t n = k->name_id[i];
    const int64_t r = tl_cnt[n]++; /* rank of launch i within its name */
    if (r < pf_cnt[n]) match[i] = (int32_t)rows[pf_off[n] + r];
  }

  /* count validation (Sec. 3.3 text, limitations paragraph) */
  for (uint32_t n = 0; n < NN; ++n) {
    if (name_counts) {
      name_counts[2 * (size_t)n] = (uint32_t)tl_cnt[n];
      name_counts[2 * (size_t)n + 1] = (uint32_t)pf_cnt[n];
    }
    if (tl_cnt[n] != pf_cnt[n]) {
      diag->names_mismatched++;
      diag->flags |= OREF_F_COUNT;
      if (tl_cnt[n] > pf_cnt[n]) diag->tl_unmatched += (uint64_t)(tl_cnt[n] - pf_cnt[n]);
      else diag->pf_unmatched += (uint64_t)(pf_cnt[n] - tl_cnt[n]);
    }
  }
  /* SKIP_NAME: a name whose counts disagree gets no assignment at all */
  if (policy == OREF_SKIP_NAME)
    for (int64_t x = 0; x < ne; ++x) {
      int64_t i = ord[x].idx;
      uint32_t n = k->name_id[i];
      if (tl_cnt[n] != pf_cnt[n]) match[i] = -1;
    }
  if (diag->bad_records) diag->flags |= OREF_F_DATA;

  free(pf_cnt); free(pf_off); free(rows); free(fill); free(ord); free(tl_cnt);
  return 0;
}

/* ----------------------------------------------------------------------- */
/* Stage 2: layer dedup, positional inheritance (Sec. 3.7)                  */
/* ----------------------------------------------------------------------- */

/* Launch-order rank of every kernel: its position when the whole timeline is
   sorted by seq (ties by input index). Launch ordinals are unique over the
   timeline, as for the matching: equal seq values raise ORDER. */
static int64_t *launch_ranks(const oref_kernels *k, oref_diag *diag) {
  const int64_t T = k->n;
  key3 *all = xcalloc((size_t)T, sizeof(key3));
  for (int64_t i = 0; i < T; ++i) {
    all[i].a = k->seq[i];
    all[i].b = all[i].c = 0;
    all[i].idx = i;
  }
  qsort(all, (size_t)T, sizeof(key3), cmp_key3);
  int64_t *rank = xcalloc((size_t)T, sizeof(int64_t));
  for (int64_t x = 0; x < T; ++x) rank[all[x].idx] = x;
  for (int64_t x = 1; x < T; ++x)
    if (all[x].a == all[x - 1].a) { diag->flags |= OREF_F_ORDER; break; }
  free(all);
  return rank;
}

int oref_dedup(const oref_kernels *k, const oref_dims *d, int32_t *match,
               oref_diag *diag) {
  if (!k || !d || !match || !diag || k->n < 0) return OREF_ERR_ARG;
  if (!dedup_on(k, d)) return 0; /* no partitions: nothing to do */
  const int64_t T = k->n;
  const uint32_t NP = d->n_parts;

  int64_t *rank = launch_ranks(k, diag);

  /* members[p]: the kernels of partition p in launch order */
  int64_t *cnt = xcalloc(NP, sizeof(int64_t));
  int64_t *off = xcalloc((size_t)NP + 1, sizeof(int64_t));
  for (int64_t i = 0; i < T; ++i)
    if (kernel_ok(k, d, i) && k->part_id[i] >= 0) cnt[k->part_id[i]]++;
  for (uint32_t q = 0; q < NP; ++q) off[q + 1] = off[q] + cnt[q];
  key3 *mem = xcalloc((size_t)off[NP], sizeof(key3));
  int64_t *fill = xcalloc(NP, sizeof(int64_t));
  for (int64_t i = 0; i < T; ++i) {
    if (!kernel_ok(k, d, i) || k->part_id[i] < 0) continue;
    int32_t q = k->part_id[i];
    key3 *e = &mem[off[q] + fill[q]++];
    e->a = (uint64_t)q;
    e->b = (uint64_t)rank[i];
    e->c = 0;
    e->idx = i;
  }
  qsort(mem, (size_t)off[NP], sizeof(key3), cmp_key3); /* by (partition, rank) */

  /* a partition is the run of launches between its tags: its launches must be
     consecutive in launch order (no other launch between them) */
  char *contig = xcalloc(NP, 1);
  for (uint32_t q = 0; q < NP; ++q) {
    if (cnt[q] == 0) { contig[q] = 1; continue; }
    uint64_t lo = mem[off[q]].b, hi = mem[off[q + 1] - 1].b;
    contig[q] = (hi - lo + 1 == (uint64_t)cnt[q]);
    if (!contig[q]) diag->flags |= OREF_F_PARTITION;
  }

  /* every duplicate takes the match of the representative's kernel at the same
     position of its partition; the position must exist and hold the same
     kernel name, otherwise the duplicate stays unmatched */
  for (uint32_t q = 0; q < NP; ++q) {
    if (!rep_ok(d, (int32_t)q)) continue;
    int32_t r = d->part_rep[q];
    if (r == (int32_t)q) continue; /* representative itself */
    int bad_class = !contig[q] || !rep_ok(d, r) || d->part_rep[r] != r || cnt[r] == 0 ||
                    !contig[r];
    for (int64_t pos = 0; pos < cnt[q]; ++pos) {
      int64_t i = mem[off[q] + pos].idx;
      int ok = !bad_class && pos < cnt[r];
      if (ok) {
        int64_t src = mem[off[r] + pos].idx;
        ok = k->name_id[src] == k->name_id[i];
        if (ok) match[i] = match[src];
      }
      if (!ok) { match[i] = -1; diag->dedup_errors++; }
    }
  }
  if (diag->dedup_errors) diag->flags |= OREF_F_DEDUP;
  free(cnt); free(off); free(mem); free(fill); free(contig); free(rank);
  return 0;
}

int oref_counters_out(const oref_profiled *p, const int32_t *match, int64_t n, float *out) {
  if (!p || n < 0 || (n > 0 && (!match || !out))) return OREF_ERR_ARG;
  for (int64_t i = 0; i < n; ++i) {
    const int32_t m = match[i];
    for (int c = 0; c < OREF_NC; ++c) {
      float v = NAN; /* no row, or the counter was not captured */
      if (m >= 0 && m < p->n && !((p->absent_mask >> c) & 1u))
        v = p->counters[(int64_t)m * p->row_stride + (int64_t)c * p->col_stride];
      out[i * OREF_NC + c] = v;
    }
  }
  return 0;
}

/* ----------------------------------------------------------------------- */
/* Dedup class discovery (Sec. 3.7)                                         */
/* ----------------------------------------------------------------------- */

/* the sequences being compared by qsort (file-scope: qsort takes no context) */
static const oref_kernels *cls_k;
static const int64_t *cls_cnt, *cls_off;
static const key3 *cls_mem;
static const char *cls_contig;

/* partitions ordered by their (name, stream) sequence in launch order:
   non-consecutive partitions last, then by length, then element by element;
   ties by partition number */
static int cmp_part_seq(const void *x, const void *y) {
  const int64_t p = *(const int64_t *)x, q = *(const int64_t *)y;
  if (cls_contig[p] != cls_contig[q]) return cls_contig[p] ? -1 : 1;
  if (cls_contig[p]) {
    if (cls_cnt[p] != cls_cnt[q]) return cls_cnt[p] < cls_cnt[q] ? -1 : 1;
    for (int64_t j = 0; j < cls_cnt[p]; ++j) {
      const int64_t a = cls_mem[cls_off[p] + j].idx, b = cls_mem[cls_off[q] + j].idx;
      if (cls_k->name_id[a] != cls_k->name_id[b])
        return cls_k->name_id[a] < cls_k->name_id[b] ? -1 : 1;
      if (cls_k->stream_id[a] != cls_k->stream_id[b])
        return cls_k->stream_id[a] < cls_k->stream_id[b] ? -1 : 1;
    }
  }
  return p < q ? -1 : (p > q ? 1 : 0);
}

int oref_dedup_classes(const oref_kernels *k, const oref_dims *d, int32_t *part_rep,
                       oref_diag *diag) {
  if (!k || !d || !diag || k->n < 0 || (d->n_parts > 0 && !part_rep)) return OREF_ERR_ARG;
  if (k->n > 0 && (!k->seq || !k->name_id || !k->stream_id || !k->part_id)) return OREF_ERR_ARG;
  const int64_t T = k->n;
  const uint32_t NP = d->n_parts;
  if (NP == 0) return 0;

  /* a launch takes part with an in-range name and partition */
  for (int64_t i = 0; i < T; ++i) {
    const int32_t p = k->part_id[i];
    if (k->name_id[i] >= d->n_names || p < -1 || (p >= 0 && (uint32_t)p >= NP))
      diag->bad_records++;
  }
  if (diag->bad_records) diag->flags |= OREF_F_DATA;

  int64_t *rank = launch_ranks(k, diag);

  /* members of each partition in launch order */
  int64_t *cnt = xcalloc(NP, sizeof(int64_t));
  int64_t *off = xcalloc((size_t)NP + 1, sizeof(int64_t));
  for (int64_t i = 0; i < T; ++i) {
    const int32_t p = k->part_id[i];
    if (k->name_id[i] < d->n_names && p >= 0 && (uint32_t)p < NP) cnt[p]++;
  }
  for (uint32_t q = 0; q < NP; ++q) off[q + 1] = off[q] + cnt[q];
  key3 *mem = xcalloc((size_t)off[NP], sizeof(key3));
  int64_t *fill = xcalloc(NP, sizeof(int64_t));
  for (int64_t i = 0; i < T; ++i) {
    const int32_t p = k->part_id[i];
    if (k->name_id[i] >= d->n_names || p < 0 || (uint32_t)p >= NP) continue;
    key3 *e = &mem[off[p] + fill[p]++];
    e->a = (uint64_t)p;
    e->b = (uint64_t)rank[i];
    e->c = 0;
    e->idx = i;
  }
  qsort(mem, (size_t)off[NP], sizeof(key3), cmp_key3);

  /* consecutive in launch order (as for the dedup broadcast) */
  char *contig = xcalloc(NP, 1);
  for (uint32_t q = 0; q < NP; ++q) {
    if (cnt[q] == 0) { contig[q] = 1; continue; }
    const uint64_t lo = mem[off[q]].b, hi = mem[off[q + 1] - 1].b;
    contig[q] = (hi - lo + 1 == (uint64_t)cnt[q]);
    if (!contig[q]) diag->flags |= OREF_F_PARTITION;
  }

  /* sort partitions by sequence; each run of equal sequences is a class,
     represented by its first (lowest-numbered) partition */
  int64_t *ord = xcalloc(NP, sizeof(int64_t));
  for (uint32_t q = 0; q < NP; ++q) ord[q] = q;
  cls_k = k;
  cls_cnt = cnt;
  cls_off = off;
  cls_mem = mem;
  cls_contig = contig;
  qsort(ord, NP, sizeof(int64_t), cmp_part_seq);
  int64_t head = -1;
  for (uint32_t j = 0; j < NP; ++j) {
    const int64_t q = ord[j];
    if (!contig[q]) { part_rep[q] = (int32_t)q; continue; }
    /* same class as the current head: the same sequence, element by element */
    int eq = 0;
    if (head >= 0 && cnt[head] == cnt[q]) {
      eq = 1;
      for (int64_t t = 0; t < cnt[q] && eq; ++t) {
        const int64_t a = mem[off[head] + t].idx, b = mem[off[q] + t].idx;
        eq = k->name_id[a] == k->name_id[b] && k->stream_id[a] == k->stream_id[b];
      }
    }
    if (!eq) head = q;
    part_rep[q] = (int32_t)head;
  }
  free(ord); free(cnt); free(off); free(mem); free(fill); free(contig); free(rank);
  return 0;
}

/* ----------------------------------------------------------------------- */
/* Stage 3: enclosure (Alg. 2, Sec. 3.5)                                    */
/* ----------------------------------------------------------------------- */

/* a range takes part only with in-range ids and kind, start <= end and
   end < 2^63 */
static int range_ok(const oref_ranges *r, const oref_dims *d, int64_t x) {
  return r->stream_id[x] < d->n_streams && r->op_id[x] < d->n_ops &&
         r->start_ns[x] <= r->end_ns[x] && r->end_ns[x] < (UINT64_C(1) << 63) &&
         (!r->kind || r->kind[x] <= OREF_KIND_SKIP);
}

/* valid ranges in nesting order per stream: (stream, start asc, end desc,
   index asc); an identical interval with a lower index is the outer one */
static key3 *nesting_order(const oref_ranges *r, const oref_dims *d, int64_t *nr_out) {
  key3 *rs = xcalloc((size_t)r->n, sizeof(key3));
  int64_t nr = 0;
  for (int64_t x = 0; x < r->n; ++x) {
    if (!range_ok(r, d, x)) continue;
    rs[nr].a = r->stream_id[x];
    rs[nr].b = r->start_ns[x];
    rs[nr].c = UINT64_MAX - r->end_ns[x];
    rs[nr].idx = x;
    nr++;
  }
  qsort(rs, (size_t)nr, sizeof(key3), cmp_key3);
  *nr_out = nr;
  return rs;
}

/* kernels on a valid stream, per stream by query point */
static key3 *kernels_by_query(const oref_kernels *k, const oref_dims *d, const uint64_t *q,
                              int64_t *nk_out) {
  key3 *ks = xcalloc((size_t)k->n, sizeof(key3));
  int64_t nk = 0;
  for (int64_t i = 0; i < k->n; ++i) {
    if (k->stream_id[i] >= d->n_streams) continue;
    ks[nk].a = k->stream_id[i];
    ks[nk].b = q[i];
    ks[nk].c = 0;
    ks[nk].idx = i;
    nk++;
  }
  qsort(ks, (size_t)nk, sizeof(key3), cmp_key3);
  *nk_out = nk;
  return ks;
}

/* the sweep's stack at query point t: every range of the stream that has
   started (s <= t) pushed in nesting order, then the finished ones (e < t)
   dropped from the top (closed intervals) */
static void stack_advance(const key3 *rs, int64_t a_end, int64_t *x, int64_t *stack,
                          int64_t *top, const oref_ranges *r, uint64_t t) {
  while (*x < a_end && rs[*x].b <= t) stack[(*top)++] = rs[(*x)++].idx;
  while (*top > 0 && r->end_ns[stack[*top - 1]] < t) (*top)--;
}

/* Depth, parents and the nesting check of one stream's ranges (rs[a ..
   a_end) in nesting order). */
static void stream_structure(const key3 *rs, int64_t a, int64_t a_end, const oref_ranges *r,
                             int64_t *stack, uint32_t *depth, int32_t *range_parent,
                             uint8_t *range_depth, oref_diag *diag) {
  /* depth: 1 + depth of the nearest earlier range (nesting order) whose end
     is not before this one's end -- that range contains it */
  int64_t top = 0;
  for (int64_t x = a; x < a_end; ++x) {
    int64_t id = rs[x].idx;
    while (top > 0 && r->end_ns[stack[top - 1]] < r->end_ns[id]) top--;
    depth[id] = top > 0 ? depth[stack[top - 1]] + 1 : 1;
    if (range_parent) range_parent[id] = top > 0 ? (int32_t)stack[top - 1] : -1;
    if (depth[id] > 255) diag->flags |= OREF_F_LIMIT;
    if (range_depth) range_depth[id] = (uint8_t)(depth[id] > 255 ? 255 : depth[id]);
    stack[top++] = id;
  }
  /* proper nesting: no two ranges with s_A < s_B < e_A < e_B. Walking in
     nesting order, after dropping ranges that end at or before s_B the top
     has the smallest end of those still open at s_B; B crosses one of them
     exactly when it crosses the top. */
  top = 0;
  int crossed = 0;
  for (int64_t x = a; x < a_end; ++x) {
    int64_t id = rs[x].idx;
    while (top > 0 && r->end_ns[stack[top - 1]] <= r->start_ns[id]) top--;
    if (top > 0 && r->end_ns[stack[top - 1]] < r->end_ns[id]) crossed = 1;
    stack[top++] = id;
  }
  if (crossed) { diag->nesting_errors++; diag->flags |= OREF_F_NOT_NESTED; }
}

int oref_enclose(const oref_kernels *k, const oref_ranges *r, const oref_dims *d,
                 int32_t *range_id, uint8_t *range_depth, oref_diag *diag) {
  return oref_enclose_walk(k, r, d, range_id, NULL, NULL, NULL, range_depth, diag);
}

int oref_enclose_walk(const oref_kernels *k, const oref_ranges *r, const oref_dims *d,
                      int32_t *range_id, uint8_t *fused, int32_t *range_any,
                      int32_t *range_parent, uint8_t *range_depth, oref_diag *diag) {
  if (!k || !r || !d || !range_id || !diag || k->n < 0 || r->n < 0) return OREF_ERR_ARG;
  if (k->n > 0 && (!k->stream_id || !(k->query_ns || k->start_ns))) return OREF_ERR_ARG;
  const int64_t T = k->n, R = r->n;
  const uint32_t NS = d->n_streams;
  const uint64_t *q = k->query_ns ? k->query_ns : k->start_ns;

  for (int64_t x = 0; x < R; ++x)
    if (!range_ok(r, d, x)) diag->bad_records++;
  for (int64_t i = 0; i < T; ++i)
    if (k->stream_id[i] >= NS) diag->bad_records++;
  if (diag->bad_records) diag->flags |= OREF_F_DATA;
  if (range_depth)
    for (int64_t x = 0; x < R; ++x) range_depth[x] = 0;
  if (range_parent)
    for (int64_t x = 0; x < R; ++x) range_parent[x] = -1;

  for (int64_t i = 0; i < T; ++i) {
    range_id[i] = -1;
    if (fused) fused[i] = 0;
    if (range_any) range_any[i] = -1;
  }
  int64_t nr, nk;
  key3 *rs = nesting_order(r, d, &nr);
  key3 *ks = kernels_by_query(k, d, q, &nk);

  int64_t *stack = xcalloc((size_t)nr + 1, sizeof(int64_t));
  uint32_t *depth = xcalloc((size_t)R, sizeof(uint32_t));
  int64_t a = 0, b = 0; /* cursors into rs and ks */
  while (a < nr || b < nk) {
    uint64_t s = a < nr ? rs[a].a : UINT64_MAX;
    if (b < nk && ks[b].a < s) s = ks[b].a;
    int64_t a_end = a, b_end = b;
    while (a_end < nr && rs[a_end].a == s) a_end++;
    while (b_end < nk && ks[b_end].a == s) b_end++;

    stream_structure(rs, a, a_end, r, stack, depth, range_parent, range_depth, diag);
    int64_t top = 0;

    /* sweep: for each kernel in query order, push every range that has
       started (s <= T), drop finished ones from the top (e < T); the top is
       the last range in nesting order with s <= T <= e, i.e. the innermost
       enclosing range, and (properly nested) the stack below it holds the
       other enclosing ranges, outward. The walk of Alg. 2 goes down the
       stack: ops are collected, skipped kinds passed over, a boundary ends
       it. */
    top = 0;
    int64_t x = a;
    for (int64_t y = b; y < b_end; ++y) {
      const uint64_t t = ks[y].b;
      stack_advance(rs, a_end, &x, stack, &top, r, t);
      const int64_t i = ks[y].idx;
      if (range_any) range_any[i] = top > 0 ? (int32_t)stack[top - 1] : -1;
      int32_t first = -1;
      int nops = 0;
      for (int64_t u = top - 1; u >= 0; --u) {
        const int64_t id = stack[u];
        if (r->end_ns[id] < t) continue; /* only under broken nesting */
        const uint8_t kd = r->kind ? r->kind[id] : OREF_KIND_OP;
        if (kd == OREF_KIND_BOUNDARY) break;
        if (kd == OREF_KIND_SKIP) continue;
        if (first < 0) first = (int32_t)id;
        nops++;
      }
      range_id[i] = first;
      if (fused) fused[i] = nops > 1 ? 1 : 0;
    }
    a = a_end;
    b = b_end;
  }
  free(rs); free(ks); free(stack); free(depth);
  return 0;
}

/* All enclosing ranges (the all_enclosing output of Alg. 2) as CSR lists:
   for each kernel, every valid range of its stream containing its query
   point, innermost first. The same sweep as the walk: at a kernel's point
   the stack holds, bottom to top in nesting order, the ranges that have
   started; those not ended before the point are the enclosing ones. */
int oref_enclose_all(const oref_kernels *k, const oref_ranges *r, const oref_dims *d,
                     int64_t *off, int32_t *ids, int64_t cap, oref_diag *diag) {
  if (!k || !r || !d || !off || !diag || k->n < 0 || r->n < 0 || cap < 0) return OREF_ERR_ARG;
  if (cap > 0 && !ids) return OREF_ERR_ARG;
  if (k->n > 0 && (!k->stream_id || !(k->query_ns || k->start_ns))) return OREF_ERR_ARG;
  const int64_t T = k->n, R = r->n;
  const uint32_t NS = d->n_streams;
  const uint64_t *q = k->query_ns ? k->query_ns : k->start_ns;
  for (int64_t x = 0; x < R; ++x)
    if (!range_ok(r, d, x)) diag->bad_records++;
  for (int64_t i = 0; i < T; ++i)
    if (k->stream_id[i] >= NS) diag->bad_records++;
  if (diag->bad_records) diag->flags |= OREF_F_DATA;

  int64_t nr, nk;
  key3 *rs = nesting_order(r, d, &nr);
  key3 *ks = kernels_by_query(k, d, q, &nk);

  /* first pass: the count per kernel; second pass: the lists */
  int64_t *cnt = xcalloc((size_t)T + 1, sizeof(int64_t));
  int64_t *stack = xcalloc((size_t)nr + 1, sizeof(int64_t));
  uint32_t *depth = xcalloc((size_t)R, sizeof(uint32_t));
  for (int pass = 0; pass < 2; ++pass) {
    int64_t a = 0, b = 0;
    while (a < nr || b < nk) {
      uint64_t st = a < nr ? rs[a].a : UINT64_MAX;
      if (b < nk && ks[b].a < st) st = ks[b].a;
      int64_t a_end = a, b_end = b;
      while (a_end < nr && rs[a_end].a == st) a_end++;
      while (b_end < nk && ks[b_end].a == st) b_end++;
      if (pass == 0) stream_structure(rs, a, a_end, r, stack, depth, NULL, NULL, diag);
      int64_t top = 0, x = a;
      for (int64_t y = b; y < b_end; ++y) {
        const uint64_t t = ks[y].b;
        stack_advance(rs, a_end, &x, stack, &top, r, t);
        const int64_t i = ks[y].idx;
        int64_t c = 0;
        for (int64_t u = top - 1; u >= 0; --u) {
          const int64_t id = stack[u];
          if (r->end_ns[id] < t) continue; /* ended before the point */
          if (pass == 1 && off[i + 1] <= cap) ids[off[i] + c] = (int32_t)id;
          c++;
        }
        if (pass == 0) cnt[i] = c;
      }
      a = a_end;
      b = b_end;
    }
    if (pass == 0) {
      off[0] = 0;
      for (int64_t i = 0; i < T; ++i) off[i + 1] = off[i] + cnt[i];
    }
  }
  free(rs); free(ks); free(stack); free(cnt); free(depth);
  return 0;
}

/* ----------------------------------------------------------------------- */
/* Stage 4: per-operator aggregation (Eq. 1, Sec. 3.8.1)                    */
/* ----------------------------------------------------------------------- */

/* compensated (Neumaier) summation keeps the oracle's sum within a few ulps of
   the exact sum at ten million terms */
typedef struct { double s, c; } nsum;
static void nadd(nsum *a, double x) {
  double t = a->s + x;
  if (fabs(a->s) >= fabs(x)) a->c += (a->s - t) + x;
  else a->c += (x - t) + a->s;
  a->s = t;
}

static const uint8_t DEFAULT_KIND[OREF_NC] = {
    /* counter appendix table, rows 1..20 */
    OREF_SUM, OREF_SUM, OREF_SUM, OREF_DWMEAN, OREF_DWMEAN, OREF_DWMEAN, OREF_DWMEAN,
    OREF_DWMEAN, OREF_DWMEAN, OREF_DWMEAN, OREF_SUM, OREF_DWMEAN, OREF_DWMEAN,
    OREF_DWMEAN, OREF_SUM, OREF_DWMEAN, OREF_DWMEAN, OREF_MAX, OREF_SUM, OREF_MAX};

/* Eq. 1 per operator row: row_of[i] is the row of kernel i (n_ops =
   UNATTRIBUTED) */
static int aggregate_rows(const oref_kernels *k, const oref_profiled *p, const int32_t *match,
                          const uint32_t *row_of, const oref_dims *d, const uint8_t *kind,
                          oref_row *table, oref_summary *sum, oref_diag *diag) {
  const int64_t T = k->n;
  const uint32_t G = d->n_ops + 1; /* row n_ops is UNATTRIBUTED */
  nsum *acc = xcalloc((size_t)G * OREF_NC, sizeof(nsum));
  double *mx = xcalloc((size_t)G * OREF_NC, sizeof(double));
  for (size_t x = 0; x < (size_t)G * OREF_NC; ++x) mx[x] = -INFINITY;
  memset(table, 0, sizeof(oref_row) * G);

  for (int64_t i = 0; i < T; ++i) {
    const uint32_t g = row_of[i];
    oref_row *row = &table[g];
    uint64_t dur = k->dur_ns[i];
    row->kernel_count++;
    row->total_ns += dur; /* nsys durations, not replay time (Sec. 3.2) */
    int32_t m = match[i];
    if (m < -1 || m >= p->n) { diag->bad_records++; continue; }
    if (m < 0) continue; /* unmatched kernels carry no counters */
    row->matched_count++;
    row->matched_ns += dur;
    for (int c = 0; c < OREF_NC; ++c) {
      double v = (double)p->counters[(int64_t)m * p->row_stride + (int64_t)c * p->col_stride];
      size_t x = (size_t)g * OREF_NC + c;
      if (kind[c] == OREF_DWMEAN) nadd(&acc[x], v * (double)dur); /* m_i * d_i */
      else if (kind[c] == OREF_SUM) nadd(&acc[x], v);
      else if (isnan(v) || v > mx[x]) mx[x] = v;
    }
  }
  if (diag->bad_records) diag->flags |= OREF_F_DATA;

  memset(sum, 0, sizeof(*sum));
  for (uint32_t g = 0; g < G; ++g) {
    oref_row *row = &table[g];
    for (int c = 0; c < OREF_NC; ++c) {
      size_t x = (size_t)g * OREF_NC + c;
      double v;
      if (((p->absent_mask >> c) & 1u) || row->matched_count == 0) v = NAN;
      else if (kind[c] == OREF_DWMEAN)
        v = row->matched_ns ? (acc[x].s + acc[x].c) / (double)row->matched_ns : NAN;
      else if (kind[c] == OREF_SUM) v = acc[x].s + acc[x].c;
      else v = mx[x];
      row->value[c] = v;
    }
    sum->total_ns += row->total_ns;
    sum->matched_ns += row->matched_ns;
    if (g < d->n_ops) sum->attributed_ns += row->total_ns;
    else sum->unattributed_ns += row->total_ns;
  }
  sum->attributed_fraction =
      sum->total_ns ? (double)sum->attributed_ns / (double)sum->total_ns : NAN;
  free(acc); free(mx);
  return 0;
}

static const uint8_t *agg_kinds(const uint8_t *agg_kind) {
  const uint8_t *kind = agg_kind ? agg_kind : DEFAULT_KIND;
  for (int c = 0; c < OREF_NC; ++c)
    if (kind[c] > OREF_MAX) return NULL;
  return kind;
}

int oref_aggregate(const oref_kernels *k, const oref_profiled *p,
                   const int32_t *match, const int32_t *range_id,
                   const oref_ranges *r, const oref_dims *d, const uint8_t *agg_kind,
                   oref_row *table, oref_summary *sum, oref_diag *diag) {
  if (!k || !p || !match || !range_id || !r || !d || !table || !sum || !diag) return OREF_ERR_ARG;
  if (k->n < 0 || (k->n > 0 && !k->dur_ns)) return OREF_ERR_ARG;
  const uint8_t *kind = agg_kinds(agg_kind);
  if (!kind) return OREF_ERR_ARG;
  /* the operator row of a kernel: the op of its range (Alg. 2 output) */
  uint32_t *row_of = xcalloc((size_t)k->n, sizeof(uint32_t));
  for (int64_t i = 0; i < k->n; ++i) {
    const int32_t rid = range_id[i];
    row_of[i] = d->n_ops;
    if (rid >= 0 && rid < r->n && r->op_id[rid] < d->n_ops) row_of[i] = r->op_id[rid];
    else if (rid < -1 || rid >= r->n || (rid >= 0 && r->op_id[rid] >= d->n_ops))
      diag->bad_records++;
  }
  const int rc = aggregate_rows(k, p, match, row_of, d, kind, table, sum, diag);
  free(row_of);
  return rc;
}

int oref_aggregate_ops(const oref_kernels *k, const oref_profiled *p, const int32_t *match,
                       const int32_t *op, const oref_dims *d, const uint8_t *agg_kind,
                       oref_row *table, oref_summary *sum, oref_diag *diag) {
  if (!k || !p || !match || !op || !d || !table || !sum || !diag) return OREF_ERR_ARG;
  if (k->n < 0 || (k->n > 0 && !k->dur_ns)) return OREF_ERR_ARG;
  const uint8_t *kind = agg_kinds(agg_kind);
  if (!kind) return OREF_ERR_ARG;
  uint32_t *row_of = xcalloc((size_t)k->n, sizeof(uint32_t));
  for (int64_t i = 0; i < k->n; ++i) {
    const int32_t o = op[i];
    row_of[i] = (o >= 0 && (uint32_t)o < d->n_ops) ? (uint32_t)o : d->n_ops;
    if (o < -1 || (o >= 0 && (uint32_t)o >= d->n_ops)) diag->bad_records++;
  }
  const int rc = aggregate_rows(k, p, match, row_of, d, kind, table, sum, diag);
  free(row_of);
  return rc;
}

int oref_aggregate_dispatch(const oref_kernels *k, const oref_profiled *p, const int32_t *match,
                            const int32_t *range_id, const int32_t *op, const oref_ranges *r,
                            const oref_dims *d, const uint8_t *agg_kind, oref_row *table,
                            oref_summary *sum, oref_diag *diag) {
  if (!k || !p || !match || !range_id || !r || !d || !table || !sum || !diag) return OREF_ERR_ARG;
  if (k->n < 0 || (k->n > 0 && !k->dur_ns) || r->n < 0 || (r->n > 0 && !r->op_id))
    return OREF_ERR_ARG;
  const uint8_t *kind = agg_kinds(agg_kind);
  if (!kind) return OREF_ERR_ARG;
  const int64_t R = r->n;
  const uint32_t NOPS = d->n_ops;
  /* a dispatch is an operator range (its op's call); a kernel attributed to
     an operator outside any range of that operator is grouped per operator */
  uint32_t *row_of = xcalloc((size_t)k->n, sizeof(uint32_t));
  for (int64_t i = 0; i < k->n; ++i) {
    const int32_t rid = range_id[i];
    const int32_t o = op ? op[i] : (rid >= 0 && rid < R ? (int32_t)r->op_id[rid] : -1);
    if (rid < -1 || rid >= R) diag->bad_records++;
    if (op && (o < -1 || (o >= 0 && (uint32_t)o >= NOPS))) diag->bad_records++;
    if (rid >= 0 && rid < R && o >= 0 && (uint32_t)o == r->op_id[rid] && (uint32_t)o < NOPS)
      row_of[i] = (uint32_t)rid;
    else if (o >= 0 && (uint32_t)o < NOPS)
      row_of[i] = (uint32_t)(R + o);
    else
      row_of[i] = (uint32_t)(R + NOPS);
  }
  oref_dims dd = *d;
  dd.n_ops = (uint32_t)(R + NOPS);
  const int rc = aggregate_rows(k, p, match, row_of, &dd, kind, table, sum, diag);
  free(row_of);
  return rc;
}

/* ----------------------------------------------------------------------- */
/* Tiered attribution (Table "tiers", decision-tree figure, Sec. 3.4-3.6)    */
/* ----------------------------------------------------------------------- */

int oref_tiers(const oref_kernels *k, const oref_corr *corr, const oref_fusion *fm,
               const oref_ranges *r, const oref_dims *d, int corr_policy,
               const int32_t *range_id, const uint8_t *walk_fused, uint8_t *tier, int32_t *op,
               uint8_t *fused, oref_coverage *cov, oref_diag *diag) {
  if (!k || !r || !d || !diag || !cov || k->n < 0 || corr_policy < 0 || corr_policy > 2)
    return OREF_ERR_ARG;
  const int64_t T = k->n;
  if (T > 0 && (!k->name_id || !k->dur_ns || !range_id || !tier || !op || !fused))
    return OREF_ERR_ARG;
  if (corr && (corr->n < 0 || (corr->n > 0 && (!corr->name_id || !corr->op_id)))) return OREF_ERR_ARG;
  if (corr && T > 0 && !k->seq) return OREF_ERR_ARG;
  if (fm && (!fm->off || !fm->op_id)) return OREF_ERR_ARG;
  const uint32_t NN = d->n_names, NOPS = d->n_ops;

  /* HIGH: the correlation map gives, per kernel name, the operator of each
     invocation index; a kernel's index is its rank among all launches of its
     name in launch order, every launch counting (the correlation pass runs
     the whole model, so layer dedup does not apply). This is Alg. 1 with
     the map's entries in place of the profiled rows. */
  int32_t *entry = xcalloc((size_t)T, sizeof(int32_t));
  for (int64_t i = 0; i < T; ++i) entry[i] = -1;
  if (corr) {
    oref_kernels kk = *k;
    kk.part_id = NULL;
    oref_dims dd = *d;
    dd.part_rep = NULL;
    dd.n_parts = 0;
    oref_profiled pc = {corr->n, corr->name_id, NULL, 0, 0, 0};
    const int rc = oref_match(&kk, &pc, &dd, corr_policy, entry, NULL, diag);
    if (rc) { free(entry); return rc; }
    for (int64_t j = 0; j < corr->n; ++j)
      if (corr->op_id[j] < -1 || (corr->op_id[j] >= 0 && (uint32_t)corr->op_id[j] >= NOPS))
        diag->bad_records++;
  }

  memset(cov, 0, sizeof(*cov));
  for (int64_t i = 0; i < T; ++i) {
    const uint32_t nm = k->name_id[i];
    int t = OREF_TIER_UNATTRIBUTED;
    int32_t o = -1;
    const int32_t e = entry[i];
    const int32_t rid = range_id[i];
    if (rid < -1 || rid >= r->n) diag->bad_records++;
    int64_t nf = 0; /* operators the fusion map lists for this kernel name */
    if (fm && nm < NN && fm->off[nm + 1] > fm->off[nm]) nf = (int64_t)fm->off[nm + 1] - fm->off[nm];
    if (e >= 0 && corr->op_id[e] >= 0 && (uint32_t)corr->op_id[e] < NOPS) {
      t = OREF_TIER_HIGH; /* pre-empts the enclosure and the fusion map */
      o = corr->op_id[e];
    } else if (rid >= 0 && rid < r->n) {
      t = OREF_TIER_NVTX; /* the enclosure walk's operator range */
      o = (int32_t)r->op_id[rid];
    } else if (nf > 0 && fm->op_id[fm->off[nm]] >= 0 && (uint32_t)fm->op_id[fm->off[nm]] < NOPS) {
      t = OREF_TIER_FUSION; /* no enclosing op range: the fused kernel's first operator */
      o = fm->op_id[fm->off[nm]];
    }
    tier[i] = (uint8_t)t;
    op[i] = o;
    /* the fusion map augments every tier: more than one listed operator
       marks the kernel fused, as does more than one enclosing op range */
    fused[i] = (uint8_t)(((walk_fused && walk_fused[i]) || nf > 1) ? 1 : 0);
    cov->count[t]++;
    cov->ns[t] += k->dur_ns[i];
  }
  uint64_t total = 0;
  for (int t = 0; t < 4; ++t) total += cov->ns[t];
  for (int t = 0; t < 4; ++t) cov->frac[t] = total ? (double)cov->ns[t] / (double)total : NAN;
  if (diag->bad_records) diag->flags |= OREF_F_DATA;
  free(entry);
  return 0;
}

int oref_attribute(const oref_kernels *k, const oref_profiled *p,
                   const oref_ranges *r, const oref_dims *d, int policy,
                   const uint8_t *agg_kind, int32_t *match, int32_t *range_id,
                   uint8_t *range_depth, uint32_t *name_counts, oref_row *table,
                   oref_summary *sum, oref_diag *diag) {
  int rc = oref_match(k, p, d, policy, match, name_counts, diag);
  if (rc) return rc;
  rc = oref_dedup(k, d, match, diag);
  if (rc) return rc;
  rc = oref_enclose(k, r, d, range_id, range_depth, diag);
  if (rc) return rc;
  rc = oref_aggregate(k, p, match, range_id, r, d, agg_kind, table, sum, diag);
  if (rc) return rc;
  oref_diag_finish(diag, policy);
  return 0;
}
