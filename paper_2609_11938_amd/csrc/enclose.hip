// Enclosure (Alg. 2) and the first level of the aggregation (Eq. 1), two
// passes over the launches in storage order.
//
// A block takes 2048 consecutive launches, eight consecutive ones per thread.
// Enclosure: the range starts that can matter for the block's main stream
// (between its smallest and largest query point) are staged in LDS; the two
// bounds come from 64-ary searches in which every lane of a wave probes one
// sample. A launch's innermost range is the last range starting at or before
// its query point, lifted along the parent chain while that range ends before
// the query point.
//
// Aggregation: each wave cuts its 512 launches into runs of one operator row.
// With at most kRowCap runs the wave reduces them in place: every thread
// accumulates its launches in registers, leaving each run that ends inside it
// in an LDS row, and a segmented scan over the lanes carries the runs that
// cross threads. The rows then go out with coalesced stores. With more runs
// the wave writes references (row, first launch, length <= 16) that the
// per-row reduction resolves later. Partial rows and references land in
// launch order at offsets found by a decoupled look-back over the blocks,
// which take their positions from a counter in the order they start.
#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kPer = 8;                         // launches per thread
constexpr int kSpan = kEncThreads * kPer;       // launches per block
constexpr int kRowCap = 32;                     // runs a wave reduces in place
constexpr unsigned long long kLbAgg = 1ull << 62, kLbInc = 2ull << 62;
constexpr long kLbSpinLimit = 1l << 26;

static_assert(kSpan == kEncSpan, "block span");
static_assert(kEncRowsPerWave == kRowCap, "row cap");

struct EncParams {
  int64_t T;
  const uint64_t *q;  // query_ns or start_ns
  const uint16_t *stream;
  CoreRanges cr;
  const int64_t *rblk;
  const int64_t *ree;
  const int32_t *npg;
  uint32_t NS, NOPS;
  int64_t R_in;           // aggregate-only: input ranges
  const uint32_t *op_in;  // aggregate-only: op ids by input range index
  int32_t *range_id;
  AggIn ag;
  EmitOut em;
  opattr_diag *diag;
};

// first index in [lo, hi) with a[idx] > x (or hi); called by a whole wave
__device__ inline int64_t wave_upper_bound(const uint64_t *a, int64_t lo, int64_t hi, uint64_t x) {
  const int l = lane_id();
  while (hi - lo > OPA_WAVE) {
    const int64_t step = (hi - lo + OPA_WAVE - 1) / OPA_WAVE;
    int64_t p = lo + (int64_t)(l + 1) * step - 1;
    if (p > hi - 1) p = hi - 1;
    const uint64_t m = __ballot(a[p] > x);
    if (m == 0) return hi;
    const int f = __ffsll((unsigned long long)m) - 1;
    const int64_t nlo = f == 0 ? lo : lo + (int64_t)f * step;
    int64_t pf = lo + (int64_t)(f + 1) * step - 1;
    if (pf > hi - 1) pf = hi - 1;
    lo = nlo;
    hi = pf + 1;
  }
  const int64_t p = lo + l;
  const uint64_t m = __ballot(p < hi && a[p] > x);
  return m ? lo + __ffsll((unsigned long long)m) - 1 : hi;
}

__device__ __forceinline__ int64_t thread_upper_bound(const uint64_t *a, int64_t lo, int64_t hi,
                                                      uint64_t x) {
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// kPer consecutive elements from p[i..), 16-byte vector loads when aligned
template <typename T>
__device__ __forceinline__ void load_run(const T *p, int64_t i, int nv, T (&o)[kPer]) {
  static_assert(sizeof(T) * kPer % 16 == 0, "vector width");
  if (nv == kPer && (reinterpret_cast<uintptr_t>(p + i) & 15) == 0) {
    const uint4 *v = reinterpret_cast<const uint4 *>(p + i);
#pragma unroll
    for (int q = 0; q < (int)(sizeof(T) * kPer / 16); ++q) {
      const uint4 t = v[q];
      memcpy(reinterpret_cast<char *>(o) + 16 * q, &t, 16);
    }
  } else {
#pragma unroll
    for (int k = 0; k < kPer; ++k) o[k] = k < nv ? p[i + k] : T(0);
  }
}

template <typename T>
__device__ __forceinline__ void store_run(T *p, int64_t i, int nv, const T (&o)[kPer]) {
  if (nv == kPer && (reinterpret_cast<uintptr_t>(p + i) & 15) == 0) {
    uint4 *v = reinterpret_cast<uint4 *>(p + i);
#pragma unroll
    for (int q = 0; q < (int)(sizeof(T) * kPer / 16); ++q) {
      uint4 t;
      memcpy(&t, reinterpret_cast<const char *>(o) + 16 * q, 16);
      v[q] = t;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kPer; ++k)
      if (k < nv) p[i + k] = o[k];
  }
}

// g[k] for a run-time k without indexing the register array
__device__ __forceinline__ uint32_t pick(const uint32_t (&g)[kPer], int k) {
  uint32_t r = g[0];
#pragma unroll
  for (int j = 1; j < kPer; ++j)
    if (j == k) r = g[j];
  return r;
}

__device__ __forceinline__ unsigned long long lb_load(const unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void lb_store(unsigned long long *p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// state word: flag (2 bits) | items (31 bits) | rows (31 bits)
__device__ __forceinline__ unsigned long long lb_pack(unsigned long long flag, uint32_t items,
                                                      uint32_t rows) {
  return flag | ((unsigned long long)items << 31) | rows;
}

// Exclusive prefix of (items, rows) over the blocks before bid; one wave.
// Returns false if the wait bound ran out (reported as a limit error).
__device__ inline bool lookback(const unsigned long long *state, int64_t bid, uint32_t &items,
                                uint32_t &rows) {
  const int ln = lane_id();
  unsigned long long si = 0, sr = 0;
  int64_t j = bid - 1;
  long spins = 0;
  while (j >= 0) {
    const int64_t idx = j - ln;
    unsigned long long st = idx >= 0 ? lb_load(state + idx) : kLbInc;
    unsigned long long flag = st & (3ull << 62);
    const unsigned long long inc = __ballot(flag == kLbInc);
    // lanes up to and including the nearest inclusive predecessor matter
    const int last = inc ? __ffsll(inc) - 1 : OPA_WAVE - 1;
    const unsigned long long need = last == 63 ? ~0ull : ((2ull << last) - 1);
    if (__ballot(flag == 0) & need) {
      if (++spins > kLbSpinLimit) return false;
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    unsigned long long ci = ln <= last ? ((st >> 31) & 0x7FFFFFFFull) : 0;
    unsigned long long cr = ln <= last ? (st & 0x7FFFFFFFull) : 0;
    si += wave_reduce_add(ci);
    sr += wave_reduce_add(cr);
    if (inc) break;
    j -= OPA_WAVE;
  }
  items = (uint32_t)si;
  rows = (uint32_t)sr;
  return true;
}

__global__ void __launch_bounds__(kEncThreads) k_enclose(EncParams a) {
  __shared__ uint64_t sS[kEncWindow];
  __shared__ uint64_t red[2][kEncThreads / OPA_WAVE];
  __shared__ int64_t win[2];
  __shared__ uint32_t sbad;
  const int tid = threadIdx.x, w = wave_id(), ln = lane_id();
  if (tid == 0) sbad = 0;
  const int64_t i0 = (int64_t)blockIdx.x * kSpan;
  const int64_t ib = i0 + (int64_t)tid * kPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kPer ? a.T - ib : kPer));
  uint32_t bad = 0;
  uint16_t st[kPer];
  uint64_t q[kPer];
  load_run(a.stream, ib, nv, st);
  load_run(a.q, ib, nv, q);
  const uint16_t s0 = a.stream[i0];
  // smallest and largest query point of the block's main stream
  uint64_t mn = ~0ull, mx = 0ull;
#pragma unroll
  for (int k = 0; k < kPer; ++k)
    if (k < nv && st[k] == s0) {
      mn = q[k] < mn ? q[k] : mn;
      mx = q[k] > mx ? q[k] : mx;
    }
  for (int o = OPA_WAVE / 2; o > 0; o >>= 1) {
    const uint64_t y = __shfl_xor(mn, o, OPA_WAVE), z = __shfl_xor(mx, o, OPA_WAVE);
    mn = y < mn ? y : mn;
    mx = z > mx ? z : mx;
  }
  if (ln == 0) {
    red[0][w] = mn;
    red[1][w] = mx;
  }
  __syncthreads();
  // wave 0 finds the window start, wave 1 its end
  if (w < 2) {
    uint64_t qa = ~0ull, qb = 0;
    for (int k = 0; k < kEncThreads / OPA_WAVE; ++k) {
      qa = red[0][k] < qa ? red[0][k] : qa;
      qb = red[1][k] > qb ? red[1][k] : qb;
    }
    int64_t p = -1;
    if (s0 < a.NS && qa <= qb) {
      const int64_t lo = a.rblk[s0], hi = a.rblk[s0 + 1];
      p = wave_upper_bound(a.cr.s, lo, hi, w == 0 ? qa : qb) - 1;
      if (w == 0 && p < lo) p = lo;
    }
    if (ln == 0) win[w] = p;
  }
  __syncthreads();
  const int64_t wlo = win[0];
  int64_t wn = (s0 < a.NS) ? win[1] - wlo + 1 : 0;
  if (wn < 0) wn = 0;
  const bool staged = wn > 0 && wn <= kEncWindow;
  if (staged)
    for (int k = tid; k < wn; k += kEncThreads) sS[k] = a.cr.s[wlo + k];
  __syncthreads();

  int32_t rout[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    int32_t rid = -1;
    if (k < nv && st[k] < a.NS && q[k] < (1ull << 63)) {
      const int64_t lo = a.rblk[st[k]], hi = a.rblk[st[k] + 1];
      const bool in0 = st[k] == s0;
      int64_t p;
      if (in0 && wn == 0) {
        p = lo - 1;  // no range of the stream starts at or before the block's queries
      } else if (in0 && staged) {
        int l2 = 0, h2 = (int)wn;
        while (l2 < h2) {
          const int mid = (l2 + h2) >> 1;
          if (sS[mid] <= q[k]) l2 = mid + 1;
          else h2 = mid;
        }
        p = wlo + l2 - 1;
        if (p < lo) p = lo - 1;
      } else {
        p = thread_upper_bound(a.cr.s, lo, hi, q[k]) - 1;
      }
      int64_t j = p;
      int steps = 0;
      while (j >= lo && a.ree[j] < (int64_t)q[k] && steps < kMaxWalk) {
        j = a.npg[j];
        ++steps;
      }
      if (j >= lo && a.ree[j] >= (int64_t)q[k]) rid = (int32_t)j;
    } else if (k < nv && st[k] >= a.NS) {
      bad++;
    }
    rout[k] = rid >= 0 ? (a.cr.perm ? a.cr.perm[rid] : rid) : -1;
  }
  store_run(a.range_id, ib, nv, rout);
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (tid == 0 && sbad)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)sbad);
}

// a += b, field by field (rows staged in LDS)
__device__ __forceinline__ void row_add(PartRow *r, const Acc &b, uint32_t maxmask) {
  r->kc += b.kc;
  r->tns += b.tns;
  r->mc += b.mc;
  r->mns += b.mns;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    const unsigned long long x = r->v[c];
    if ((maxmask >> c) & 1u) r->v[c] = b.v[c] > x ? b.v[c] : x;
    else r->v[c] = d2bits(bits2d(x) + bits2d(b.v[c]));
  }
  r->nan |= b.nan;
}

template <bool DEF>  // DEF: the default aggregation kinds
__global__ void __launch_bounds__(kEncThreads) __attribute__((amdgpu_waves_per_eu(4)))
k_agg_runs(EncParams a) {
  __shared__ PartRow stage[kEncThreads / OPA_WAVE][kRowCap];
  __shared__ uint32_t wcnt[2][kEncThreads / OPA_WAVE];
  __shared__ uint32_t spre[2];
  __shared__ uint32_t sbid, sbad, sfail;
  const int tid = threadIdx.x, w = wave_id(), ln = lane_id();
  const AggIn &in = a.ag;
  const uint32_t mx = DEF ? kDefMaxMask : in.maxmask, dw = DEF ? kDefDwMask : in.dwmask;
  if (tid == 0) {
    sbad = 0;
    sfail = 0;
    sbid = atomicAdd(a.em.ctr, 1u);
  }
  __syncthreads();
  const int64_t bid = sbid;
  const int64_t ib = bid * kSpan + (int64_t)tid * kPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kPer ? a.T - ib : kPer));
  uint32_t bad = 0;
  uint32_t g[kPer];
  int32_t mt[kPer];
  uint32_t du[kPer];
  {
    int32_t rin[kPer];
    load_run(a.range_id, ib, nv, rin);
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      g[k] = k < nv ? a.NOPS : 0xFFFFFFFFu;
      if (k >= nv) continue;
      const int32_t r = rin[k];
      if (r >= 0 && r < a.R_in && a.op_in[r] < a.NOPS) g[k] = a.op_in[r];
      else if (r < -1 || r >= a.R_in || r >= 0) bad++;
    }
  }
  load_run(in.match, ib, nv, mt);
  load_run(in.dur, ib, nv, du);
#pragma unroll
  for (int k = 0; k < kPer; ++k)
    if (k < nv && (mt[k] < -1 || (int64_t)mt[k] >= in.P)) bad++;  // aggregates as unmatched

  // ---- runs of one operator row inside the wave, in launch order
  const uint32_t gl = __shfl_up(g[kPer - 1], 1, OPA_WAVE);
  uint32_t hm = 0;  // bit k: launch k starts a run
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const uint32_t prev = k ? g[k - 1] : (ln ? gl : 0xFFFFFFFFu);
    if (k < nv && g[k] != prev) hm |= 1u << k;
  }
  // pieces for references: runs cut at every 16th launch as well
  const uint32_t hp = hm | ((nv > 0 && (ln & 1) == 0) ? 1u : 0u);
  const uint32_t nh = __popc(hm), nhp = __popc(hp);
  const uint32_t hb = wave_incl_scan_add(nh) - nh;
  const uint32_t hpb = wave_incl_scan_add(nhp) - nhp;
  const uint32_t nr_w = __shfl(hb + nh, OPA_WAVE - 1, OPA_WAVE);
  const uint32_t np_w = __shfl(hpb + nhp, OPA_WAVE - 1, OPA_WAVE);
  const bool rowmode = nr_w <= (uint32_t)kRowCap;
  if (ln == 0) {
    wcnt[0][w] = rowmode ? nr_w : np_w;
    wcnt[1][w] = rowmode ? nr_w : 0u;
  }
  __syncthreads();
  uint32_t bi = 0, br = 0, wi = 0, wr = 0;
  for (int k = 0; k < kEncThreads / OPA_WAVE; ++k) {
    if (k < w) {
      wi += wcnt[0][k];
      wr += wcnt[1][k];
    }
    bi += wcnt[0][k];
    br += wcnt[1][k];
  }
  if (tid == 0) lb_store(a.em.state + bid, lb_pack(bid == 0 ? kLbInc : kLbAgg, bi, br));

  // ---- in-place reduction (row mode). Each thread accumulates its launches;
  // a run that ends inside the thread goes to its LDS row (the first one of
  // them still lacks the part from earlier threads, added after the scan).
  // The thread's last run is scanned across the lanes.
  PartRow *wst = stage[w];
  Acc inc;
  acc_zero(inc);
  if (rowmode) {
    uint32_t gk = g[0];
#pragma unroll 1
    for (int k = 0; k < nv; ++k) {
      if (k > 0 && ((hm >> k) & 1u)) {
        acc_store(wst + hb + __popc(hm & ((1u << k) - 1u)) - 1u, inc, gk);
        acc_zero(inc);
      }
      acc_launch(inc, in, in.match[ib + k], in.dur[ib + k], mx, dw);
      gk = pick(g, k);
    }
    const unsigned long long hl = __ballot(hm != 0) | 1ull;
    const unsigned long long upto = ln == 63 ? ~0ull : ((2ull << ln) - 1);
    const int sl = 63 - __clzll(hl & upto);
#pragma unroll
    for (int o = 1; o < OPA_WAVE; o <<= 1) acc_scan_step(inc, o, ln - o >= sl, mx);
    // the lane's last run: ends here, or continues into the next lane and
    // (if it ends inside that lane) completes the row that lane left
    const uint32_t nvn = __shfl_down((uint32_t)nv, 1, OPA_WAVE);
    const uint32_t hmn = __shfl_down(hm, 1, OPA_WAVE);
    if (nv > 0) {
      PartRow *r = wst + hb + nh - 1u;
      if (ln == OPA_WAVE - 1 || nvn == 0 || (hmn & 1u)) acc_store(r, inc, g[nv - 1]);
      else if (hmn & 0xFEu) row_add(r, inc, mx);
    }
  }

  // ---- block offsets
  if (w == 0) {
    uint32_t pi = 0, pr = 0;
    bool ok = true;
    if (bid > 0) ok = lookback(a.em.state, bid, pi, pr);
    if (ln == 0) {
      if (bid > 0) lb_store(a.em.state + bid, lb_pack(kLbInc, pi + bi, pr + br));
      spre[0] = pi;
      spre[1] = pr;
      if (!ok) sfail = 1;
      if (bid == a.em.nblocks - 1) {
        a.em.meta[0] = (int64_t)pi + bi;
        a.em.meta[1] = (int64_t)pr + br;
      }
    }
  }
  __syncthreads();
  const uint32_t ibase = spre[0] + wi, rbase = spre[1] + wr;

  if (rowmode) {
    // coalesced copy of the wave's rows, then one item per row
    const unsigned long long *src = reinterpret_cast<const unsigned long long *>(wst);
    unsigned long long *dst = reinterpret_cast<unsigned long long *>(a.em.rows + rbase);
    const uint32_t nw = nr_w * (uint32_t)(sizeof(PartRow) / 8);
    for (uint32_t x = ln; x < nw; x += OPA_WAVE) dst[x] = src[x];
    if ((uint32_t)ln < nr_w) {
      a.em.ig[ibase + ln] = wst[ln].g;
      a.em.ia[ibase + ln] = rbase + ln;
      a.em.ib[ibase + ln] = 0;
    }
  } else {
    // references: every piece start writes (row, first launch, length)
    const uint32_t hpn = __shfl_down(hp, 1, OPA_WAVE);
    const uint32_t nvn = __shfl_down((uint32_t)nv, 1, OPA_WAVE);
    const uint32_t spill = ln < OPA_WAVE - 1 ? (hpn ? (uint32_t)__ffs(hpn) - 1u : nvn) : 0u;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (!((hp >> k) & 1u)) continue;
      const uint32_t rest = hp >> (k + 1);
      const uint32_t len = rest ? (uint32_t)__ffs(rest) : (uint32_t)(nv - k) + spill;
      const uint32_t idx = hpb + __popc(hp & ((1u << k) - 1u));
      a.em.ig[ibase + idx] = g[k];
      a.em.ia[ibase + idx] = (uint32_t)(ib + k);
      a.em.ib[ibase + idx] = len;
    }
  }
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (tid == 0 && sbad)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)sbad);
  if (tid == 0 && sfail) atomicOr(&a.diag->flags, OPATTR_F_LIMIT);
}

static EncParams enc_params(const EncArgs &x) {
  const Plan &pl = *x.pl;
  const opattr_kernels *k = x.k;
  EncParams a{};
  a.T = pl.T;
  a.q = k->query_ns ? k->query_ns : k->start_ns;
  a.stream = k->stream_id;
  a.NS = x.d->n_streams;
  a.NOPS = x.d->n_ops;
  a.range_id = x.range_id;
  a.diag = x.diag;
  a.cr = x.cr;
  a.rblk = at<int64_t>(x.ws, pl.rblk);
  a.ree = at<int64_t>(x.ws, pl.ree);
  a.npg = at<int32_t>(x.ws, pl.npg);
  // the aggregation reads range ids by input range index
  a.R_in = x.r ? x.r->n : 0;
  a.op_in = x.r ? x.r->op_id : nullptr;
  return a;
}

void run_enclose(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const EncParams a = enc_params(x);
  probe_begin(OPATTR_PROBE_MAIN_PASS, s);
  if (pl.T > 0) k_enclose<<<(unsigned)pl.nencb, kEncThreads, 0, s>>>(a);
  probe_end(OPATTR_PROBE_MAIN_PASS, s);
}

void run_aggregate_all(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  EncParams a = enc_params(x);
  a.ag = agg_inputs(x);
  a.em = emit_out(x.ws, pl);
  // look-back states, the start counter, the per-row item counts (and with
  // no launches the item totals), cleared by one kernel (graph-safe)
  FillJobs clr;
  clr.add(a.em.state, 0, 2 * (pl.nencb + 1));
  clr.add(at<uint32_t>(x.ws, pl.gcnt), 0, pl.G);
  if (pl.T <= 0) clr.add(a.em.meta, 0, 8);
  fill_many(clr, s);
  probe_begin(OPATTR_PROBE_AGG_RUNS, s);
  if (pl.T > 0) {
    const unsigned nb = (unsigned)pl.nencb;
    if (a.ag.maxmask == kDefMaxMask && a.ag.dwmask == kDefDwMask)
      k_agg_runs<true><<<nb, kEncThreads, 0, s>>>(a);
    else
      k_agg_runs<false><<<nb, kEncThreads, 0, s>>>(a);
  }
  probe_end(OPATTR_PROBE_AGG_RUNS, s);
  run_aggregate(x, s);
}

}  // namespace opa
