// Enclosure (Alg. 2) and per-operator aggregation (Eq. 1) in one pass over
// the timeline.
//
// Each block takes 256 consecutive launches. The range starts that can matter
// for the block's main stream (those between the block's smallest and largest
// query point) are staged in LDS; the two bounds are found by 64-ary searches
// in which every lane of a wave probes one sample. A launch's innermost range
// is the last range starting at or before its query point, lifted along the
// parent chain while that range ends before the query point.
//
// Aggregation reduces runs of equal operator inside each wave (segmented
// scans over lanes, lanes = consecutive launches) and adds each run's totals to
// the operator's accumulator row with device-scope atomics: u64 for the exact
// integer fields, fp64 for the sums, and an order-preserving u32 key for the
// fp32 maximum (NaN tracked in a separate bit).
#include "common.h"
#include "impl.h"

namespace opa {

struct EncParams {
  int64_t T;
  const uint64_t *q;       // query_ns or start_ns
  const uint16_t *stream;
  const uint32_t *dur;
  const int32_t *match;
  int64_t P;
  const float *counters;
  int64_t rs, cs;
  uint32_t dwmask, summask, maxmask;
  CoreRanges cr;
  const int64_t *rblk;
  const int64_t *ree;
  const int32_t *npg;
  uint32_t NS, NOPS;
  int64_t R_in;             // aggregate-only: input ranges
  const uint32_t *op_in;    // aggregate-only: op ids by input range index
  int32_t *range_id;
  AccRow *acc;
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

__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

template <typename T>
__device__ __forceinline__ T seg_sum(T x, int segstart) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    const T y = __shfl_up(x, o, OPA_WAVE);
    if (l - o >= segstart) x += y;
  }
  return x;
}
__device__ __forceinline__ uint32_t seg_max(uint32_t x, int segstart) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, OPA_WAVE);
    if (l - o >= segstart && y > x) x = y;
  }
  return x;
}
__device__ __forceinline__ uint32_t seg_or(uint32_t x, int segstart) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, OPA_WAVE);
    if (l - o >= segstart) x |= y;
  }
  return x;
}

template <int MODE>
__global__ void __launch_bounds__(kEncThreads) k_enc(EncParams a) {
  __shared__ uint64_t sS[kEncWindow];
  __shared__ uint64_t red[2][kEncThreads / OPA_WAVE];
  __shared__ int64_t win[3];  // window first index, size, block stream's first range
  __shared__ uint32_t sbad;
  const int tid = threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.x * kEncThreads;
  const int64_t i = i0 + tid;
  const bool valid = i < a.T;
  if (tid == 0) sbad = 0;
  uint32_t bad = 0;
  uint32_t g = a.NOPS + 1;  // sentinel: never flushed
  if (valid) g = a.NOPS;

  if (MODE & 1) {
    const uint16_t st = valid ? a.stream[i] : (uint16_t)0xFFFF;
    const uint64_t q = valid ? a.q[i] : 0;
    const uint16_t s0 = a.stream[i0];
    const bool in0 = valid && st == s0 && s0 < a.NS;
    // smallest and largest query point of the block's main stream
    uint64_t mn = in0 ? q : ~0ull, mx = in0 ? q : 0ull;
    for (int o = OPA_WAVE / 2; o > 0; o >>= 1) {
      const uint64_t y = __shfl_xor(mn, o, OPA_WAVE), z = __shfl_xor(mx, o, OPA_WAVE);
      mn = y < mn ? y : mn;
      mx = z > mx ? z : mx;
    }
    if (lane_id() == 0) {
      red[0][wave_id()] = mn;
      red[1][wave_id()] = mx;
    }
    __syncthreads();
    if (wave_id() == 0) {
      uint64_t qa = ~0ull, qb = 0;
      for (int k = 0; k < kEncThreads / OPA_WAVE; ++k) {
        qa = red[0][k] < qa ? red[0][k] : qa;
        qb = red[1][k] > qb ? red[1][k] : qb;
      }
      int64_t wlo = 0, wn = 0, lo = 0;
      if (s0 < a.NS && qa <= qb) {
        lo = a.rblk[s0];
        const int64_t hi = a.rblk[s0 + 1];
        const int64_t pa = wave_upper_bound(a.cr.s, lo, hi, qa) - 1;
        const int64_t pb = wave_upper_bound(a.cr.s, lo, hi, qb) - 1;
        wlo = pa > lo ? pa : lo;
        wn = pb - wlo + 1;
        if (wn < 0) wn = 0;
      }
      if (lane_id() == 0) {
        win[0] = wlo;
        win[1] = wn;
        win[2] = lo;
      }
    }
    __syncthreads();
    const int64_t wlo = win[0], wn = win[1];
    const bool staged = wn > 0 && wn <= kEncWindow;
    if (staged)
      for (int k = tid; k < wn; k += kEncThreads) sS[k] = a.cr.s[wlo + k];
    __syncthreads();

    int32_t rid = -1;
    if (valid && st < a.NS && q < (1ull << 63)) {
      const int64_t lo = a.rblk[st], hi = a.rblk[st + 1];
      int64_t p;
      if (in0 && wn == 0) {
        p = lo - 1;  // no range of the stream starts at or before the block's queries
      } else if (in0 && staged) {
        int l2 = 0, h2 = (int)wn;
        while (l2 < h2) {
          const int mid = (l2 + h2) >> 1;
          if (sS[mid] <= q) l2 = mid + 1;
          else h2 = mid;
        }
        p = wlo + l2 - 1;
        if (p < lo) p = lo - 1;
      } else {
        p = thread_upper_bound(a.cr.s, lo, hi, q) - 1;
      }
      int64_t j = p;
      int steps = 0;
      while (j >= lo && a.ree[j] < (int64_t)q && steps < kMaxWalk) {
        j = a.npg[j];
        ++steps;
      }
      if (j >= lo && a.ree[j] >= (int64_t)q) rid = (int32_t)j;
    } else if (valid && st >= a.NS) {
      bad++;
    }
    if (valid) a.range_id[i] = rid >= 0 ? (a.cr.perm ? a.cr.perm[rid] : rid) : -1;
    if (rid >= 0) g = a.cr.op[rid];
  } else if (valid) {
    const int32_t r = a.range_id[i];
    if (r >= 0 && r < a.R_in && a.op_in[r] < a.NOPS) g = a.op_in[r];
    else if (r < -1 || r >= a.R_in || r >= 0) bad++;
  }

  if (MODE & 2) {
    const uint32_t d = valid ? a.dur[i] : 0u;
    const int32_t m = valid ? a.match[i] : -1;
    const bool matched = valid && m >= 0 && m < a.P;
    if (valid && (m < -1 || m >= a.P)) bad++;
    const int l = lane_id();
    const uint32_t gp = __shfl_up(g, 1, OPA_WAVE);
    const bool head = l == 0 || g != gp;
    const uint64_t H = __ballot(head);
    const uint64_t le = l == 63 ? ~0ull : ((2ull << l) - 1ull);
    const int segstart = 63 - __clzll(H & le);
    const bool tail = l == 63 || ((H >> (l + 1)) & 1ull);
    const bool flush = tail && g <= a.NOPS;

    const unsigned long long kc = seg_sum<unsigned long long>(valid ? 1ull : 0ull, segstart);
    const unsigned long long tn = seg_sum<unsigned long long>(d, segstart);
    const unsigned long long mc = seg_sum<unsigned long long>(matched ? 1ull : 0ull, segstart);
    const unsigned long long mn = seg_sum<unsigned long long>(matched ? d : 0ull, segstart);
    AccRow *row = flush ? &a.acc[g] : nullptr;
    if (flush) {
      atomicAdd(&row->kc, kc);
      atomicAdd(&row->tns, tn);
      if (mc) {
        atomicAdd(&row->mc, mc);
        atomicAdd(&row->mns, mn);
      }
    }
    const bool any_matched = __ballot(matched) != 0;
    if (any_matched) {
      const float *crow = matched ? a.counters + (int64_t)m * a.rs : nullptr;
      uint32_t nanbits = 0;
#pragma unroll 4
      for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
        const float v = matched ? crow[(int64_t)c * a.cs] : 0.0f;
        if ((a.maxmask >> c) & 1u) {
          const uint32_t k = matched ? f2key(v) : 0u;
          if (matched && v != v) nanbits |= 1u << c;
          const uint32_t km = seg_max(k, segstart);
          if (flush && mc && km) atomicMax(&row->maxk[c], km);
        } else {
          double x = (double)v;
          if ((a.dwmask >> c) & 1u) x *= (double)d;  // m_i * d_i
          x = seg_sum<double>(x, segstart);
          if (flush && mc) atomicAdd(&row->sum[c], x);
        }
      }
      const uint32_t nb = seg_or(nanbits, segstart);
      if (flush && nb) atomicOr(&row->nanmask, nb);
    }
  }
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (tid == 0 && sbad)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)sbad);
}

__global__ void __launch_bounds__(1024) k_agg_finalize(const AccRow *__restrict__ acc, uint32_t G,
                                                       uint32_t NOPS, uint32_t dwmask,
                                                       uint32_t summask, uint32_t maxmask,
                                                       uint32_t absent, opattr_op_row *table,
                                                       opattr_summary *sum) {
  __shared__ unsigned long long red[4][16];
  unsigned long long at_ = 0, un = 0, tot = 0, mt = 0;
  for (uint32_t g = threadIdx.x; g < G; g += 1024) {
    const AccRow &a = acc[g];
    opattr_op_row r;
    r.kernel_count = a.kc;
    r.total_ns = a.tns;
    r.matched_count = a.mc;
    r.matched_ns = a.mns;
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      double v;
      if (((absent >> c) & 1u) || a.mc == 0) v = __longlong_as_double(0x7FF8000000000000ll);
      else if ((maxmask >> c) & 1u)
        v = ((a.nanmask >> c) & 1u) ? __longlong_as_double(0x7FF8000000000000ll)
                                     : (double)key2f(a.maxk[c]);
      else if ((dwmask >> c) & 1u)
        v = a.mns ? a.sum[c] / (double)a.mns : __longlong_as_double(0x7FF8000000000000ll);
      else v = a.sum[c];
      r.value[c] = v;
    }
    table[g] = r;
    tot += a.tns;
    mt += a.mns;
    if (g < NOPS) at_ += a.tns;
    else un += a.tns;
  }
  (void)summask;
  at_ = wave_reduce_add(at_);
  un = wave_reduce_add(un);
  tot = wave_reduce_add(tot);
  mt = wave_reduce_add(mt);
  if (lane_id() == 0) {
    red[0][wave_id()] = at_;
    red[1][wave_id()] = un;
    red[2][wave_id()] = tot;
    red[3][wave_id()] = mt;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    opattr_summary s{};
    for (int k = 0; k < 16; ++k) {
      s.attributed_ns += red[0][k];
      s.unattributed_ns += red[1][k];
      s.total_ns += red[2][k];
      s.matched_ns += red[3][k];
    }
    s.attributed_fraction = s.total_ns ? (double)s.attributed_ns / (double)s.total_ns
                                       : __longlong_as_double(0x7FF8000000000000ll);
    *sum = s;
  }
}

void run_enclose_aggregate(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const opattr_kernels *k = x.k;
  EncParams a{};
  a.T = pl.T;
  a.q = k->query_ns ? k->query_ns : k->start_ns;
  a.stream = k->stream_id;
  a.dur = k->dur_ns;
  a.match = x.match;
  a.NS = x.d->n_streams;
  a.NOPS = x.d->n_ops;
  a.range_id = x.range_id;
  a.diag = x.diag;
  a.cr = x.cr;
  a.rblk = at<int64_t>(x.ws, pl.rblk);
  a.ree = at<int64_t>(x.ws, pl.ree);
  a.npg = at<int32_t>(x.ws, pl.npg);
  const uint32_t G = x.d->n_ops + 1;
  if (x.mode & 2) {
    a.P = x.p->n;
    a.counters = x.p->counters;
    a.rs = x.p->row_stride;
    a.cs = x.p->col_stride;
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      const uint8_t kd = x.agg_kind[c];
      if (kd == OPATTR_AGG_DWMEAN) a.dwmask |= 1u << c;
      else if (kd == OPATTR_AGG_MAX) a.maxmask |= 1u << c;
      else a.summask |= 1u << c;
    }
    a.acc = at<AccRow>(x.ws, pl.acc);
    note(hipMemsetAsync(a.acc, 0, sizeof(AccRow) * G, s));
  }
  if (x.mode == kAggregateOnly) {
    a.R_in = x.r ? x.r->n : 0;
    a.op_in = x.r ? x.r->op_id : nullptr;
  }
  const unsigned nb = (unsigned)((pl.T + kEncThreads - 1) / kEncThreads);
  probe_begin(OPATTR_PROBE_MAIN_PASS, s);
  if (pl.T > 0) {
    if (x.mode == kEncloseOnly) k_enc<1><<<nb, kEncThreads, 0, s>>>(a);
    else if (x.mode == kAggregateOnly) k_enc<2><<<nb, kEncThreads, 0, s>>>(a);
    else k_enc<3><<<nb, kEncThreads, 0, s>>>(a);
  }
  if (x.mode & 2)
    k_agg_finalize<<<1, 1024, 0, s>>>(a.acc, G, a.NOPS, a.dwmask, a.summask, a.maxmask,
                                      x.p->absent_mask, x.table, x.sum);
  probe_end(OPATTR_PROBE_MAIN_PASS, s);
}

}  // namespace opa
