// Range structure for the enclosure (Sec. 3.5, Alg. 2).
//
// The paper keeps a per-stream interval tree. Here the ranges of each stream
// sit in nesting order (start asc, end desc, index asc) and every range gets
// its parent: the nearest earlier range of the stream whose end is not before
// its own (that range contains it). A launch's innermost range is then the last
// range starting at or before its query point, or the first ancestor of that
// range whose end is not before the query point.
//
// Parents are "nearest previous greater-or-equal" values, found without a
// sequential stack: pointer jumping inside LDS tiles of 1024 ranges, the same
// jumping over tile maxima, then one bounded walk for the ranges whose parent
// lies in an earlier tile. While jumping, each range also records the largest
// end it skipped; a skipped end beyond the range's start is a crossing.
#include "common.h"
#include "impl.h"

namespace opa {

constexpr uint64_t kEndLimit = 1ull << 63;  // valid ends stay below 2^63

// validity and effective end of range x (-1 marks a bad range); parents unknown
__device__ __forceinline__ bool rprep_one(const CoreRanges &cr, uint32_t NS, uint32_t NOPS,
                                          int64_t *ree, int32_t *npg, int64_t x) {
  const uint64_t s = cr.s[x], e = cr.e[x];
  const bool ok = cr.st[x] < NS && cr.op[x] < NOPS && s <= e && e < kEndLimit &&
                  (!cr.kind || cr.kind[x] <= OPATTR_KIND_SKIP);
  ree[x] = ok ? (int64_t)e : -1;
  npg[x] = -1;
  return !ok;
}

__device__ __forceinline__ void count_bad(bool bad, opattr_diag *diag) {
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)__popcll(m));
}

__global__ void k_rprep(CoreRanges cr, uint32_t NS, uint32_t NOPS, int64_t *ree, int32_t *npg,
                        opattr_diag *diag) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  count_bad(x < cr.n && rprep_one(cr, NS, NOPS, ree, npg, x), diag);
}

// The range preparation in one launch, three jobs by block ranges: [0, na)
// validity and effective ends, 256 ranges a block; [na, na + nb) the stream
// blocks, one wave per stream s = 0..NS; then the clears (fill jobs).
struct RangePro {
  CoreRanges cr;
  uint32_t NS, NOPS;
  int64_t *ree;
  int32_t *npg;
  int64_t *rblk;
  opattr_diag *diag;
  int na, nb, nf;
  FillJobs fill;
};

__global__ void __launch_bounds__(256) k_range_pro(RangePro a) {
  const int b = blockIdx.x;
  if (b < a.na) {
    const int64_t x = (int64_t)b * blockDim.x + threadIdx.x;
    count_bad(x < a.cr.n && rprep_one(a.cr, a.NS, a.NOPS, a.ree, a.npg, x), a.diag);
  } else if (b < a.na + a.nb) {
    const uint32_t sw = (uint32_t)(b - a.na) * (blockDim.x / OPA_WAVE) + wave_id();
    if (sw <= a.NS) stream_block_wave(a.cr.st, a.cr.n, sw, a.rblk);
  } else {
    const int fb = b - a.na - a.nb;
    const int64_t stride = (int64_t)a.nf * blockDim.x;
    for (int q = 0; q < a.fill.count; ++q)
      for (int64_t i = (int64_t)fb * blockDim.x + threadIdx.x; i < a.fill.n[q]; i += stride)
        a.fill.p[q][i] = a.fill.v[q];
  }
}

// promised nesting order: (stream, start asc, end desc) never decreases
__global__ void k_rcheck(CoreRanges cr, opattr_diag *diag) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (x > 0 && x < cr.n) {
    const uint16_t a = cr.st[x - 1], b = cr.st[x];
    bad = a > b || (a == b && (cr.s[x - 1] > cr.s[x] ||
                               (cr.s[x - 1] == cr.s[x] && cr.e[x - 1] < cr.e[x])));
  }
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1) {
    atomicAdd((unsigned long long *)&diag->order_violations, (unsigned long long)__popcll(m));
    atomicOr(&diag->flags, OPATTR_F_ORDER);
  }
}

// blk[s] = first position with stream >= s, s = 0..NS (one wave per s)
__global__ void __launch_bounds__(256) k_blocks16(const uint16_t *st, int64_t n, uint32_t NS,
                                                  int64_t *blk) {
  const uint32_t s = blockIdx.x * (blockDim.x / OPA_WAVE) + wave_id();
  if (s <= NS) stream_block_wave(st, n, s, blk);
}

void launch_stream_blocks(const uint16_t *st, int64_t n, uint32_t NS, int64_t *blk,
                          hipStream_t s) {
  const uint32_t waves = NS + 1;
  k_blocks16<<<(waves + 3) / 4, 256, 0, s>>>(st, n, NS, blk);
}

// tbase[s] = first tile of stream s (tiles never straddle streams), by one
// block of 1024 threads
__device__ inline void tile_bases(const int64_t *rblk, uint32_t NS, int32_t *tbase) {
  __shared__ uint32_t sh[16];
  uint32_t carry = 0;
  for (uint32_t base = 0; base < NS; base += 1024) {
    const uint32_t s = base + threadIdx.x;
    uint32_t c = 0;
    if (s < NS) c = (uint32_t)((rblk[s + 1] - rblk[s] + kRangeTile - 1) / kRangeTile);
    uint32_t tot;
    const uint32_t pre = block_excl_scan_add<uint32_t>(c, sh, &tot);
    if (s < NS) tbase[s] = (int32_t)(carry + pre);
    carry += tot;
  }
  if (threadIdx.x == 0) tbase[NS] = (int32_t)carry;
}

__global__ void __launch_bounds__(1024) k_rtile_base(const int64_t *rblk, uint32_t NS,
                                                     int32_t *tbase) {
  tile_bases(rblk, NS, tbase);
}

constexpr uint32_t kInlineBases = 1024;  // streams whose tile bases k_rlocal finds itself

__device__ __forceinline__ uint32_t stream_of_tile(const int32_t *tbase, uint32_t NS, int32_t t) {
  uint32_t lo = 0, hi = NS;  // last s with tbase[s] <= t
  while (lo + 1 < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (tbase[mid] <= t) lo = mid;
    else hi = mid;
  }
  return lo;
}

struct RangeWork {
  CoreRanges cr;
  uint32_t NS;
  const int64_t *rblk;
  int32_t *tbase;  // written by k_rtile_base, or by k_rlocal with inline_bases
  int64_t *ree;
  int32_t *npg;
  int64_t *mxv;
  int64_t *tM;
  int32_t *tnpg, *tnpg2;
  int64_t *tmx, *tmx2;
  int32_t *tstr, *tlast;
  uint8_t *sflag;
  opattr_diag *diag;
  int inline_bases;  // k_rlocal finds the tile bases (NS <= kInlineBases)
};

// Local parents inside one tile by pointer jumping (Jacobi rounds): cand[i]
// starts at i-1; while the candidate's end is before ours, jump to the
// candidate's candidate. Every skipped range ends before ours, so cand stays a
// valid candidate and converges to the nearest one with end >= ours, or -1 when
// none is in the tile. mx[i] accumulates the largest end skipped.
__global__ void __launch_bounds__(kRangeTile) k_rlocal(RangeWork w) {
  __shared__ int64_t e[kRangeTile];
  __shared__ int64_t mx[kRangeTile];
  __shared__ int32_t cand[kRangeTile];
  __shared__ int64_t red[kRangeTile / OPA_WAVE];
  __shared__ int32_t stb[kInlineBases + 1];
  static_assert(kRangeTile == 1024, "one thread per range of a tile, 1024 for the bases");
  const int32_t *tb = w.tbase;
  if (w.inline_bases) {
    tile_bases(w.rblk, w.NS, stb);
    __syncthreads();
    if (blockIdx.x == 0)
      for (uint32_t k = threadIdx.x; k <= w.NS; k += blockDim.x) w.tbase[k] = stb[k];
    tb = stb;
  }
  const int32_t t = blockIdx.x, ntr = tb[w.NS];
  if (t >= ntr) return;
  const uint32_t s = stream_of_tile(tb, w.NS, t);
  const int64_t x0 = w.rblk[s] + (int64_t)(t - tb[s]) * kRangeTile;
  const int64_t x1 = min(x0 + kRangeTile, w.rblk[s + 1]);
  const int i = threadIdx.x;
  const bool valid = x0 + i < x1;
  e[i] = valid ? w.ree[x0 + i] : -1;
  mx[i] = -1;
  cand[i] = i - 1;
  __syncthreads();
  for (;;) {
    const int c = cand[i];
    int nc = c;
    int64_t nm = mx[i];
    if (valid && c >= 0 && e[c] < e[i]) {
      nc = cand[c];
      const int64_t v = e[c] > mx[c] ? e[c] : mx[c];
      nm = v > nm ? v : nm;
    }
    __syncthreads();
    cand[i] = nc;
    mx[i] = nm;
    if (!__syncthreads_or(nc != c)) break;
  }
  if (valid) {
    const int64_t x = x0 + i;
    const int c = cand[i];
    w.npg[x] = c >= 0 ? (int32_t)(x0 + c) : -2;  // -2: parent lies before the tile
    w.mxv[x] = mx[i];
    if (c >= 0 && e[i] >= 0 && mx[i] > (int64_t)w.cr.s[x]) w.sflag[s] = 1;
  }
  // tile maximum
  int64_t v = e[i];
  for (int o = OPA_WAVE / 2; o > 0; o >>= 1) {
    const int64_t y = __shfl_xor(v, o, OPA_WAVE);
    v = y > v ? y : v;
  }
  if (lane_id() == 0) red[wave_id()] = v;
  __syncthreads();
  if (i == 0) {
    int64_t m = -1;
    for (int k = 0; k < kRangeTile / OPA_WAVE; ++k) m = red[k] > m ? red[k] : m;
    w.tM[t] = m;
    w.tstr[t] = (int32_t)s;
    w.tlast[t] = (int32_t)(x1 - 1);
  }
}

// The same jumping over tile maxima (one block, tiles in global memory).
__global__ void __launch_bounds__(1024) k_rtiles(RangeWork w) {
  const int32_t ntr = w.tbase[w.NS];
  int32_t *cn = w.tnpg, *nn = w.tnpg2;
  int64_t *cm = w.tmx, *nm = w.tmx2;
  for (int32_t t = threadIdx.x; t < ntr; t += 1024) {
    cn[t] = (t > 0 && w.tstr[t - 1] == w.tstr[t]) ? t - 1 : -1;
    cm[t] = -1;
  }
  __threadfence_block();
  __syncthreads();
  for (;;) {
    int changed = 0;
    for (int32_t t = threadIdx.x; t < ntr; t += 1024) {
      const int32_t c = cn[t];
      int32_t n2 = c;
      int64_t m2 = cm[t];
      if (c >= 0 && w.tM[c] < w.tM[t]) {
        n2 = cn[c];
        const int64_t v = w.tM[c] > cm[c] ? w.tM[c] : cm[c];
        m2 = v > m2 ? v : m2;
      }
      nn[t] = n2;
      nm[t] = m2;
      changed |= n2 != c;
    }
    __threadfence_block();
    const int any = __syncthreads_or(changed);
    int32_t *tn = cn;
    cn = nn;
    nn = tn;
    int64_t *tm = cm;
    cm = nm;
    nm = tm;
    if (!any) break;
  }
  if (cn != w.tnpg)
    for (int32_t t = threadIdx.x; t < ntr; t += 1024) {
      w.tnpg[t] = cn[t];
      w.tmx[t] = cm[t];
    }
}

// Parents of the ranges whose parent lies in an earlier tile: walk back over
// tiles (tile parents skip tiles whose maximum end is below ours), then down
// the local parents of the tile found, from its last range.
__global__ void k_rresolve(RangeWork w) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= w.cr.n || w.npg[x] != -2) return;
  const uint32_t s = w.cr.st[x];
  const int64_t ex = w.ree[x];
  const int32_t t = w.tbase[s] + (int32_t)((x - w.rblk[s]) / kRangeTile);
  int64_t acc = w.mxv[x];
  int32_t u = (t > w.tbase[s]) ? t - 1 : -1;
  int steps = 0;
  while (u >= 0 && w.tM[u] < ex && steps < (1 << 20)) {
    const int64_t v = w.tM[u] > w.tmx[u] ? w.tM[u] : w.tmx[u];
    acc = v > acc ? v : acc;
    u = w.tnpg[u];
    ++steps;
  }
  int32_t par = -1;
  if (u >= 0) {
    int32_t y = w.tlast[u];
    steps = 0;
    while (w.ree[y] < ex && steps < (1 << 20)) {
      const int64_t v = w.ree[y] > w.mxv[y] ? w.ree[y] : w.mxv[y];
      acc = v > acc ? v : acc;
      y = w.npg[y];
      ++steps;
      if (y < 0) break;  // defensive: cannot happen, a tile maximum stops the walk
    }
    par = y;
  }
  w.npg[x] = par;
  if (ex >= 0 && acc > (int64_t)w.cr.s[x]) w.sflag[s] = 1;
}

// depth = length of the parent chain (1 for a root, 0 for a bad range)
__global__ void k_rdepth(RangeWork w, uint8_t *range_depth) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  range_depth_one(w.npg, w.ree, w.cr.st, w.cr.perm, w.cr.n, w.NS, x, range_depth, w.diag);
}

static RangeWork range_work(const CoreRanges &cr, const opattr_dims *d, void *ws, const Plan &pl,
                            opattr_diag *diag) {
  RangeWork w;
  w.cr = cr;
  w.NS = d->n_streams;
  w.rblk = at<int64_t>(ws, pl.rblk);
  w.tbase = at<int32_t>(ws, pl.tbase);
  w.ree = at<int64_t>(ws, pl.ree);
  w.npg = at<int32_t>(ws, pl.npg);
  w.mxv = at<int64_t>(ws, pl.mxv);
  w.tM = at<int64_t>(ws, pl.tM);
  w.tnpg = at<int32_t>(ws, pl.tnpg);
  w.tnpg2 = at<int32_t>(ws, pl.tnpg2);
  w.tmx = at<int64_t>(ws, pl.tmx);
  w.tmx2 = at<int64_t>(ws, pl.tmx2);
  w.tstr = at<int32_t>(ws, pl.tfirst);
  w.tlast = at<int32_t>(ws, pl.tlast);
  w.sflag = at<uint8_t>(ws, pl.sflag);
  w.diag = diag;
  w.inline_bases = d->n_streams <= kInlineBases ? 1 : 0;
  return w;
}

// ---------------------------------------------------------------------------
// Nesting order of ranges given in any order: a merge sort of the records
// (stream, start, end, index) by stream asc, start asc, end desc, index asc.
// Blocks first sort tiles of kRsTile records in LDS (bitonic network), then
// each pass merges pairs of sorted runs; a block takes kRsTile outputs of one
// pair, finds where they begin in each run along the merge path (a search on
// the diagonal, 64 probes per step across a wave), stages the two slices in
// LDS and places every record by its rank in the other slice (binary
// searches, a thread's records searched together). The index makes the
// order strict, so no two records compare equal. The last pass writes the
// sorted start, end, stream and index and gathers the operator and kind by
// the index.
// ---------------------------------------------------------------------------
constexpr int kRsTile = 1024, kRsThreads = 256, kRsPer = kRsTile / kRsThreads;
constexpr int kRsSteps = 11;  // binary search steps over at most kRsTile records

struct RSortBuf {
  uint64_t *s, *e;
  uint32_t *x;
  uint16_t *st;
};
struct RSortOut {  // the last pass's extra outputs (op, kind gathered by index)
  const uint32_t *op;
  const uint8_t *kd;
  uint32_t *op_o;
  uint8_t *kd_o;
};

struct RRec {
  uint64_t s, e;
  uint32_t x, st;
};
__device__ __forceinline__ bool rrec_less(const RRec &a, const RRec &b) {
  if (a.st != b.st) return a.st < b.st;
  if (a.s != b.s) return a.s < b.s;
  if (a.e != b.e) return a.e > b.e;
  return a.x < b.x;
}

struct RsLds {
  uint64_t s[kRsTile], e[kRsTile];
  uint32_t x[kRsTile], st[kRsTile];
  __device__ __forceinline__ RRec get(int k) const { return RRec{s[k], e[k], x[k], st[k]}; }
  __device__ __forceinline__ void put(int k, const RRec &r) {
    s[k] = r.s;
    e[k] = r.e;
    x[k] = r.x;
    st[k] = r.st;
  }
};

__device__ __forceinline__ RRec rrec_load(const RSortBuf &b, int64_t i) {
  return RRec{b.s[i], b.e[i], b.x[i], b.st[i]};
}
__device__ __forceinline__ void rrec_store(const RSortBuf &b, const RSortOut &f, bool last,
                                           int64_t i, const RRec &r) {
  b.s[i] = r.s;
  b.e[i] = r.e;
  b.x[i] = r.x;
  b.st[i] = (uint16_t)r.st;
  if (last) {
    f.op_o[i] = f.op[r.x];
    if (f.kd) f.kd_o[i] = f.kd[r.x];
  }
}

__global__ void __launch_bounds__(kRsThreads) k_rsort_tile(const opattr_ranges r, int64_t R,
                                                           RSortBuf out, RSortOut f, int last) {
  __shared__ RsLds t;
  const int tid = threadIdx.x;
  const int64_t base = (int64_t)blockIdx.x * kRsTile;
  for (int k = tid; k < kRsTile; k += kRsThreads) {
    const int64_t i = base + k;
    // records past R sort after every real one (streams are 16-bit)
    t.put(k, i < R ? RRec{r.start_ns[i], r.end_ns[i], (uint32_t)i, r.stream_id[i]}
                   : RRec{~0ull, 0ull, 0xFFFFFFFFu, 0xFFFFFFFFu});
  }
  __syncthreads();
  for (int k = 2; k <= kRsTile; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int q = tid; q < kRsTile / 2; q += kRsThreads) {
        const int i = 2 * q - (q & (j - 1)), p = i + j;
        const RRec a = t.get(i), b = t.get(p);
        if (rrec_less(b, a) == ((i & k) == 0)) {
          t.put(i, b);
          t.put(p, a);
        }
      }
      __syncthreads();
    }
  const int n = (int)(R - base < kRsTile ? R - base : kRsTile);
  for (int k = tid; k < n; k += kRsThreads) rrec_store(out, f, last != 0, base + k, t.get(k));
}

// Records of run A among the first d outputs of merging A = in[pa, pa + la)
// with B = in[pb, pb + lb): the first m where A[m] does not precede
// B[d - 1 - m]. One wave; each step probes 64 evenly spaced candidates.
__device__ int64_t merge_split(const RSortBuf &in, int64_t pa, int64_t la, int64_t pb,
                               int64_t lb, int64_t d) {
  int64_t lo = d - lb > 0 ? d - lb : 0, hi = d < la ? d : la;
  const int ln = lane_id();
  while (lo < hi) {  // uniform over the wave
    const int64_t step = (hi - lo + OPA_WAVE - 1) / OPA_WAVE, m = lo + ln * step;
    const bool p = m < hi && rrec_less(rrec_load(in, pa + m), rrec_load(in, pb + d - 1 - m));
    const int c = __popcll(__ballot(p));  // the predicate holds on a prefix of the probes
    if (c == 0) break;
    const int64_t ff = lo + (int64_t)c * step;  // first probe where it fails (or past hi)
    lo = lo + (int64_t)(c - 1) * step + 1;
    hi = ff < hi ? ff : hi;
  }
  return lo;
}

__global__ void __launch_bounds__(kRsThreads) k_rsort_merge(RSortBuf in, RSortBuf out, int64_t R,
                                                            int64_t w, RSortOut f, int last) {
  __shared__ RsLds t;
  __shared__ int64_t split[2];
  const int tid = threadIdx.x, wv = wave_id();
  const int64_t o0 = (int64_t)blockIdx.x * kRsTile;  // first output of the block
  const int64_t p0 = o0 / (2 * w) * (2 * w);          // first record of the pair of runs
  const int64_t la = R - p0 < w ? R - p0 : w;
  const int64_t rb = R - p0 - la, lb = rb < 0 ? 0 : (rb < w ? rb : w);
  const int64_t d0 = o0 - p0, d1 = d0 + kRsTile < la + lb ? d0 + kRsTile : la + lb;
  if (wv < 2) {
    const int64_t sp = merge_split(in, p0, la, p0 + la, lb, wv ? d1 : d0);
    if (lane_id() == 0) split[wv] = sp;
  }
  __syncthreads();
  const int64_t i0 = split[0], i1 = split[1];
  const int na = (int)(i1 - i0), nt = (int)(d1 - d0);
  const int64_t b0 = p0 + la + (d0 - i0);
  for (int k = tid; k < nt; k += kRsThreads)
    t.put(k, rrec_load(in, k < na ? p0 + i0 + k : b0 + (k - na)));
  __syncthreads();
  // rank of each record among the other slice: how many of its records precede it
  RRec v[kRsPer];
  int lo[kRsPer], hi[kRsPer], first[kRsPer];
#pragma unroll
  for (int u = 0; u < kRsPer; ++u) {
    const int k = tid + u * kRsThreads;
    const bool inA = k < na;
    v[u] = t.get(k < nt ? k : 0);
    lo[u] = k >= nt ? 0 : (inA ? na : 0);
    hi[u] = k >= nt ? 0 : (inA ? nt : na);
    first[u] = lo[u];
  }
#pragma unroll
  for (int q = 0; q < kRsSteps; ++q)
#pragma unroll
    for (int u = 0; u < kRsPer; ++u)
      if (lo[u] < hi[u]) {
        const int mid = (lo[u] + hi[u]) >> 1;
        if (rrec_less(t.get(mid), v[u]))
          lo[u] = mid + 1;
        else
          hi[u] = mid;
      }
#pragma unroll
  for (int u = 0; u < kRsPer; ++u) {
    const int k = tid + u * kRsThreads;
    if (k < nt) {
      const int pos = (k < na ? k : k - na) + (lo[u] - first[u]);
      rrec_store(out, f, last != 0, o0 + pos, v[u]);
    }
  }
}

// Sorts ranges into nesting order; the result lands in `fin` (with op and
// kind in f), `tmp` is the other buffer of the passes.
static void sort_ranges(const opattr_ranges *r, int64_t R, const RSortBuf &fin,
                        const RSortBuf &tmp, const RSortOut &f, hipStream_t s) {
  int np = 0;
  for (int64_t w = kRsTile; w < R; w *= 2) ++np;
  const unsigned nb = (unsigned)((R + kRsTile - 1) / kRsTile);
  // the passes alternate buffers; start so that the last one writes fin
  const RSortBuf *cur = (np % 2 == 0) ? &fin : &tmp;
  k_rsort_tile<<<nb, kRsThreads, 0, s>>>(*r, R, *cur, f, np == 0 ? 1 : 0);
  int q = 0;
  for (int64_t w = kRsTile; w < R; w *= 2, ++q) {
    const RSortBuf *nxt = cur == &fin ? &tmp : &fin;
    k_rsort_merge<<<nb, kRsThreads, 0, s>>>(*cur, *nxt, R, w, f, q == np - 1 ? 1 : 0);
    cur = nxt;
  }
}

// range_parent[perm(x)] = perm(parent of x) for valid ranges, else -1
__global__ void k_range_parent(CoreRanges cr, const int64_t *ree, const int32_t *npg,
                               int32_t *range_parent) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= cr.n) return;
  const int32_t par = ree[x] >= 0 ? npg[x] : -1;
  const int64_t o = cr.perm ? cr.perm[x] : x;
  range_parent[o] = par >= 0 ? (cr.perm ? cr.perm[par] : par) : -1;
}

void write_range_parents(const CoreRanges &cr, void *ws, const Plan &pl, int32_t *range_parent,
                         hipStream_t s) {
  if (range_parent && cr.n > 0)
    k_range_parent<<<(unsigned)((cr.n + 255) / 256), 256, 0, s>>>(
        cr, at<int64_t>(ws, pl.ree), at<int32_t>(ws, pl.npg), range_parent);
}

CoreRanges prepare_ranges(const opattr_ranges *r, const opattr_dims *d, void *ws, const Plan &pl,
                          opattr_diag *diag, bool validate, hipStream_t s, const FillJobs *extra) {
  CoreRanges cr;
  cr.n = pl.R;
  const int64_t R = pl.R;
  if (pl.ranges_nested) {
    cr.s = r->start_ns;
    cr.e = r->end_ns;
    cr.st = r->stream_id;
    cr.op = r->op_id;
    cr.kind = r->kind;
    cr.perm = nullptr;
    if (validate && R > 1) k_rcheck<<<(unsigned)((R + 255) / 256), 256, 0, s>>>(cr, diag);
  } else if (R > 0) {
    RSortBuf fin{at<uint64_t>(ws, pl.rs_c), at<uint64_t>(ws, pl.re_c), at<uint32_t>(ws, pl.rperm),
                 at<uint16_t>(ws, pl.rst_c)};
    RSortBuf tmp{at<uint64_t>(ws, pl.rsort_k0), at<uint64_t>(ws, pl.rsort_k1),
                 at<uint32_t>(ws, pl.rsort_v0), at<uint16_t>(ws, pl.rsort_st)};
    RSortOut f{r->op_id, r->kind, at<uint32_t>(ws, pl.rop_c), at<uint8_t>(ws, pl.rkd_c)};
    sort_ranges(r, R, fin, tmp, f, s);
    const uint64_t *sc = fin.s, *ec = fin.e;
    cr.s = sc;
    cr.e = ec;
    cr.st = at<uint16_t>(ws, pl.rst_c);
    cr.op = at<uint32_t>(ws, pl.rop_c);
    cr.kind = r->kind ? at<uint8_t>(ws, pl.rkd_c) : nullptr;
    cr.perm = reinterpret_cast<const int32_t *>(at<uint32_t>(ws, pl.rperm));
  } else {
    cr.s = cr.e = nullptr;
    cr.st = nullptr;
    cr.op = nullptr;
    cr.kind = nullptr;
    cr.perm = nullptr;
  }
  const uint32_t NS = d->n_streams;
  int64_t *rblk = at<int64_t>(ws, pl.rblk);
  // the clears: the caller's and the crossing flags
  FillJobs clr = extra ? *extra : FillJobs{};
  clr.add(at<uint8_t>(ws, pl.sflag), 0, sflag_words(NS));
  if (R > 0) {
    RangePro a{};
    a.cr = cr;
    a.NS = NS;
    a.NOPS = d->n_ops;
    a.ree = at<int64_t>(ws, pl.ree);
    a.npg = at<int32_t>(ws, pl.npg);
    a.rblk = rblk;
    a.diag = diag;
    a.na = (int)((R + 255) / 256);
    a.nb = (int)((NS + 1 + 3) / 4);
    int64_t mx = 0;
    for (int q = 0; q < clr.count; ++q) mx = clr.n[q] > mx ? clr.n[q] : mx;
    a.nf = (int)((mx + 255) / 256 < 1024 ? (mx + 255) / 256 : 1024);
    a.fill = clr;
    k_range_pro<<<(unsigned)(a.na + a.nb + a.nf), 256, 0, s>>>(a);
  } else {
    clr.add(rblk, 0, 2 * ((int64_t)NS + 1));
    fill_many(clr, s);
  }
  return cr;
}

// With range kinds: Alg. 2's walk from every range as the innermost one
// (outward through the parents; a boundary ends it, skipped kinds are passed
// over): the first op range (core position, -1 none) and whether more than
// one op range is reached. A launch whose innermost range does not start at
// its query point walks exactly this way, so the enclosure pass looks the
// result up instead of walking.
__global__ void k_range_walk(CoreRanges cr, const int32_t *npg, int32_t *wfirst,
                             uint8_t *wfused) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= cr.n) return;
  int32_t first = -1;
  int nops = 0, hops = 0;
  for (int64_t j = x; j >= 0 && hops < kMaxWalk; j = npg[j], ++hops) {
    const uint8_t kd = cr.kind[j];
    if (kd == OPATTR_KIND_BOUNDARY) break;
    if (kd != OPATTR_KIND_OP) continue;
    if (first < 0) first = (int32_t)j;
    if (++nops > 1) break;  // fused: the rest of the walk changes nothing
  }
  wfirst[x] = first;
  wfused[x] = nops > 1 ? 1 : 0;
}

void resolve_ranges(const CoreRanges &cr, const opattr_dims *d, void *ws, const Plan &pl,
                    uint8_t *range_depth, opattr_diag *diag, hipStream_t s, bool defer_depth) {
  const uint32_t NS = d->n_streams;
  if (pl.R <= 0 || NS == 0) {
    if (range_depth && pl.R > 0) fill_u8(range_depth, 0, pl.R, s);
    return;
  }
  RangeWork w = range_work(cr, d, ws, pl, diag);
  if (!w.inline_bases) k_rtile_base<<<1, 1024, 0, s>>>(w.rblk, NS, at<int32_t>(ws, pl.tbase));
  k_rlocal<<<(unsigned)pl.ntr_max, kRangeTile, 0, s>>>(w);
  k_rtiles<<<1, 1024, 0, s>>>(w);
  const unsigned nb = (unsigned)((pl.R + 255) / 256);
  k_rresolve<<<nb, 256, 0, s>>>(w);
  if (!defer_depth) k_rdepth<<<nb, 256, 0, s>>>(w, range_depth);
  if (cr.kind)
    k_range_walk<<<nb, 256, 0, s>>>(cr, at<int32_t>(ws, pl.npg), at<int32_t>(ws, pl.wfirst),
                                   at<uint8_t>(ws, pl.wfused));
}

}  // namespace opa
