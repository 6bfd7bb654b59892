// Per-operator aggregation (Eq. 1, Sec. 3.8.1) without atomics.
//
// The enclosure pass leaves, per block of launches, runs of consecutive
// launches that share an operator row. Here the runs are
//   1. compacted in launch order,
//   2. counting-sorted by row (tiles of 4096 runs sorted in LDS, per-tile row
//      histograms scanned down the columns; stable, so each row keeps its runs
//      in launch order),
//   3. cut into items of at most 32 runs of one row, each reduced by one
//      workgroup: every thread accumulates its launches in registers (u64
//      counts and ns, fp64 sums of m or m*d, an order-preserving key for the
//      fp32 maximum), then one block reduction writes the item's partial row,
//   4. combined per row in item order by one wave, then finalised (duration-
//      weighted means divided by the matched duration, NaN for absent
//      counters and rows without matched launches).
// Every sum is taken in a fixed order, so results are reproducible.
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kRunsPerItem = 32;

RunSlots run_slots(void *ws, const Plan &pl) {
  RunSlots r;
  r.g = at<uint32_t>(ws, pl.slot_g);
  r.kb = at<uint32_t>(ws, pl.slot_kb);
  r.len = at<uint32_t>(ws, pl.slot_len);
  r.nruns = at<uint32_t>(ws, pl.nruns);
  return r;
}

struct AggWork {
  int64_t T, nencb, ntrt;
  uint32_t G, NOPS;
  RunSlots slots;
  const uint32_t *roff;
  uint32_t *cg, *ckb, *clen;
  int64_t *meta;  // [0] runs, [1] run tiles, [2] items
  uint32_t *rth, *rtch, *gcnt, *goff, *ioff, *skb, *slen;
  AccRow *part;
  // inputs
  const uint32_t *dur;
  const int32_t *match;
  int64_t P;
  const float *counters;
  int64_t rs, cs;
  uint32_t dwmask, maxmask, absent;
  opattr_op_row *table;
  opattr_summary *sum;
};

// 1. compaction: one wave per enclosure block
__global__ void __launch_bounds__(256) k_run_compact(AggWork w) {
  const int64_t b = (int64_t)blockIdx.x * 4 + wave_id();
  if (b == 0 && lane_id() == 0) {
    const int64_t nr = w.meta[0];
    w.meta[1] = (nr + OPA_TILE - 1) / OPA_TILE;
  }
  if (b >= w.nencb) return;
  const uint32_t n = w.slots.nruns[b];
  const uint32_t o = w.roff[b];
  for (uint32_t r = lane_id(); r < n; r += OPA_WAVE) {
    const int64_t src = b * kEncThreads + r;
    w.cg[o + r] = w.slots.g[src];
    w.ckb[o + r] = w.slots.kb[src];
    w.clen[o + r] = w.slots.len[src];
  }
}

__device__ inline void run_tile_keys(const AggWork &w, int64_t base, int64_t nr, uint32_t *A) {
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int l = c * OPA_TILE_THREADS + threadIdx.x;
    const int64_t x = base + l;
    const uint32_t g = x < nr ? w.cg[x] : w.G;
    A[l] = (g << OPA_SLOT_BITS) | (uint32_t)l;
  }
}

// 2a. per-tile row histograms
__global__ void __launch_bounds__(256) k_run_hist(AggWork w) {
  __shared__ TileSmem sm;
  const int64_t nr = w.meta[0];
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  if (base >= nr) return;
  run_tile_keys(w, base, nr, sm.A);
  __syncthreads();
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(w.G));
  write_hist_row(sm.A, w.G, w.rth + (int64_t)blockIdx.x * w.G);
}

// 2b. row offsets of the sorted runs and item offsets (one block)
__global__ void __launch_bounds__(1024) k_row_offsets(AggWork w) {
  __shared__ uint32_t sh[16];
  uint32_t carry = 0, icarry = 0;
  for (uint32_t base = 0; base < w.G; base += 1024) {
    const uint32_t g = base + threadIdx.x;
    const uint32_t c = g < w.G ? w.gcnt[g] : 0u;
    const uint32_t it = (c + kRunsPerItem - 1) / kRunsPerItem;
    uint32_t tot, itot;
    const uint32_t pre = block_excl_scan_add<uint32_t>(c, sh, &tot);
    const uint32_t ipre = block_excl_scan_add<uint32_t>(it, sh, &itot);
    if (g < w.G) {
      w.goff[g] = carry + pre;
      w.ioff[g] = icarry + ipre;
    }
    carry += tot;
    icarry += itot;
  }
  if (threadIdx.x == 0) {
    w.goff[w.G] = carry;
    w.ioff[w.G] = icarry;
    w.meta[2] = icarry;
  }
}

// 2c. stable scatter of the runs into row order
__global__ void __launch_bounds__(256) k_run_scatter(AggWork w) {
  __shared__ TileSmem sm;
  const int64_t nr = w.meta[0];
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  if (base >= nr) return;
  run_tile_keys(w, base, nr, sm.A);
  __syncthreads();
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(w.G));
  const uint32_t *row = w.rth + (int64_t)blockIdx.x * w.G;
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int p = c * OPA_TILE_THREADS + threadIdx.x;
    const uint32_t key = sm.A[p];
    const uint32_t g = key >> OPA_SLOT_BITS;
    if (g >= w.G) continue;
    const int lo = lds_lower_bound(sm.A, OPA_TILE, g << OPA_SLOT_BITS);
    const uint32_t dst = w.goff[g] + row[g] + (uint32_t)(p - lo);
    const int64_t x = base + (key & (OPA_TILE - 1));
    w.skb[dst] = w.ckb[x];
    w.slen[dst] = w.clen[x];
  }
}

__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// last index g in [0, n) with a[g] <= x (a non-decreasing, a[0] <= x)
__device__ __forceinline__ uint32_t last_le(const uint32_t *a, uint32_t n, uint32_t x) {
  uint32_t lo = 0, hi = n;
  while (lo + 1 < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid;
    else hi = mid;
  }
  return lo;
}

// 3. one workgroup per item (grid-stride over items)
__global__ void __launch_bounds__(256) k_reduce(AggWork w) {
  __shared__ uint32_t kb[kRunsPerItem];
  __shared__ uint32_t pre[kRunsPerItem + 1];
  __shared__ unsigned long long ired[4][4];
  __shared__ double fred[4][OPATTR_NUM_COUNTERS];
  __shared__ uint32_t kred[4][OPATTR_NUM_COUNTERS + 1];
  const int64_t nitems = w.meta[2];
  const int tid = threadIdx.x, wv = wave_id(), ln = lane_id();
  for (int64_t item = blockIdx.x; item < nitems; item += gridDim.x) {
    const uint32_t g = last_le(w.ioff, w.G, (uint32_t)item);
    const uint32_t first = w.goff[g] + ((uint32_t)item - w.ioff[g]) * kRunsPerItem;
    const uint32_t end = w.goff[g + 1];
    const int nrun = (int)min((uint32_t)kRunsPerItem, end - first);
    if (wv == 0) {
      const uint32_t len = ln < nrun ? w.slen[first + ln] : 0u;
      if (ln < nrun) kb[ln] = w.skb[first + ln];
      const uint32_t inc = wave_incl_scan_add(len);
      if (ln < kRunsPerItem) pre[ln + 1] = inc;
      if (ln == 0) pre[0] = 0;
    }
    __syncthreads();
    const uint32_t K = pre[nrun];
    unsigned long long kc = 0, tn = 0, mc = 0, mn = 0;
    double f[OPATTR_NUM_COUNTERS];
    uint32_t mk[OPATTR_NUM_COUNTERS];
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      f[c] = 0.0;
      mk[c] = 0u;
    }
    uint32_t nanb = 0;
    for (uint32_t pos = tid; pos < K; pos += 256) {
      int lo = 0, hi = nrun;  // run holding pos: last r with pre[r] <= pos
      while (lo + 1 < hi) {
        const int mid = (lo + hi) >> 1;
        if (pre[mid] <= pos) lo = mid;
        else hi = mid;
      }
      const int64_t k = (int64_t)kb[lo] + (pos - pre[lo]);
      const uint32_t d = w.dur[k];
      const int32_t m = w.match[k];
      kc += 1;
      tn += d;
      if (m >= 0 && m < w.P) {
        mc += 1;
        mn += d;
        const float *row = w.counters + (int64_t)m * w.rs;
        const double dd = (double)d;
#pragma unroll
        for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
          const float v = row[(int64_t)c * w.cs];
          if ((w.maxmask >> c) & 1u) {
            const uint32_t key = f2key(v);
            mk[c] = key > mk[c] ? key : mk[c];
            if (v != v) nanb |= 1u << c;
          } else {
            f[c] += ((w.dwmask >> c) & 1u) ? (double)v * dd : (double)v;  // m_i * d_i
          }
        }
      }
    }
    // block reduction
    kc = wave_reduce_add(kc);
    tn = wave_reduce_add(tn);
    mc = wave_reduce_add(mc);
    mn = wave_reduce_add(mn);
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      f[c] = wave_reduce_add(f[c]);
      uint32_t x = mk[c];
      for (int o = OPA_WAVE / 2; o > 0; o >>= 1) {
        const uint32_t y = __shfl_xor(x, o, OPA_WAVE);
        x = y > x ? y : x;
      }
      mk[c] = x;
    }
    for (int o = OPA_WAVE / 2; o > 0; o >>= 1) nanb |= __shfl_xor(nanb, o, OPA_WAVE);
    if (ln == 0) {
      ired[wv][0] = kc;
      ired[wv][1] = tn;
      ired[wv][2] = mc;
      ired[wv][3] = mn;
#pragma unroll
      for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
        fred[wv][c] = f[c];
        kred[wv][c] = mk[c];
      }
      kred[wv][OPATTR_NUM_COUNTERS] = nanb;
    }
    __syncthreads();
    AccRow *out = w.part + item;
    if (tid < 4) {
      unsigned long long s = 0;
      for (int k2 = 0; k2 < 4; ++k2) s += ired[k2][tid];
      (&out->kc)[tid] = s;
    } else if (tid >= 64 && tid < 64 + OPATTR_NUM_COUNTERS) {
      const int c = tid - 64;
      out->sum[c] = ((fred[0][c] + fred[1][c]) + fred[2][c]) + fred[3][c];
    } else if (tid >= 128 && tid < 128 + OPATTR_NUM_COUNTERS + 1) {
      const int c = tid - 128;
      uint32_t x;
      if (c < OPATTR_NUM_COUNTERS) {
        x = kred[0][c];
        for (int k2 = 1; k2 < 4; ++k2) x = kred[k2][c] > x ? kred[k2][c] : x;
        out->maxk[c] = x;
      } else {
        x = kred[0][c] | kred[1][c] | kred[2][c] | kred[3][c];
        out->nanmask = x;
      }
    }
    __syncthreads();
  }
}

// 4. one wave per operator row: combine its items in order and finalise
__global__ void __launch_bounds__(256) k_combine(AggWork w) {
  const uint32_t g = blockIdx.x * 4 + wave_id();
  if (g >= w.G) return;
  const int ln = lane_id();
  const uint32_t i0 = w.ioff[g], i1 = w.ioff[g + 1];
  unsigned long long kc = 0, tn = 0, mc = 0, mn = 0;
  double f[OPATTR_NUM_COUNTERS];
  uint32_t mk[OPATTR_NUM_COUNTERS];
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    f[c] = 0.0;
    mk[c] = 0u;
  }
  uint32_t nanb = 0;
  for (uint32_t it = i0 + ln; it < i1; it += OPA_WAVE) {
    const AccRow &p = w.part[it];
    kc += p.kc;
    tn += p.tns;
    mc += p.mc;
    mn += p.mns;
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      f[c] += p.sum[c];
      mk[c] = p.maxk[c] > mk[c] ? p.maxk[c] : mk[c];
    }
    nanb |= p.nanmask;
  }
  kc = wave_reduce_add(kc);
  tn = wave_reduce_add(tn);
  mc = wave_reduce_add(mc);
  mn = wave_reduce_add(mn);
  for (int o = OPA_WAVE / 2; o > 0; o >>= 1) nanb |= __shfl_xor(nanb, o, OPA_WAVE);
  double mine = 0.0;
  uint32_t mykey = 0;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    const double s = wave_reduce_add(f[c]);
    uint32_t x = mk[c];
    for (int o = OPA_WAVE / 2; o > 0; o >>= 1) {
      const uint32_t y = __shfl_xor(x, o, OPA_WAVE);
      x = y > x ? y : x;
    }
    if (ln == c) {
      mine = s;
      mykey = x;
    }
  }
  opattr_op_row *row = w.table + g;
  if (ln == 0) {
    row->kernel_count = kc;
    row->total_ns = tn;
    row->matched_count = mc;
    row->matched_ns = mn;
  }
  if (ln < OPATTR_NUM_COUNTERS) {
    const int c = ln;
    const double qnan = __longlong_as_double(0x7FF8000000000000ll);
    double v;
    if (((w.absent >> c) & 1u) || mc == 0) v = qnan;
    else if ((w.maxmask >> c) & 1u) v = ((nanb >> c) & 1u) ? qnan : (double)key2f(mykey);
    else if ((w.dwmask >> c) & 1u) v = mn ? mine / (double)mn : qnan;
    else v = mine;
    row->value[c] = v;
  }
}

// summary over the finished rows (one block)
__global__ void __launch_bounds__(1024) k_summary(AggWork w) {
  __shared__ unsigned long long red[4][16];
  unsigned long long at_ = 0, un = 0, tot = 0, mt = 0;
  for (uint32_t g = threadIdx.x; g < w.G; g += 1024) {
    const unsigned long long t = w.table[g].total_ns;
    tot += t;
    mt += w.table[g].matched_ns;
    if (g < w.NOPS) at_ += t;
    else un += t;
  }
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
    *w.sum = s;
  }
}

void run_aggregate(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  AggWork w{};
  w.T = pl.T;
  w.nencb = pl.nencb;
  w.ntrt = pl.ntrt;
  w.G = pl.G;
  w.NOPS = x.d->n_ops;
  w.slots = run_slots(x.ws, pl);
  w.roff = at<uint32_t>(x.ws, pl.roff);
  w.cg = at<uint32_t>(x.ws, pl.cg);
  w.ckb = at<uint32_t>(x.ws, pl.ckb);
  w.clen = at<uint32_t>(x.ws, pl.clen);
  w.meta = at<int64_t>(x.ws, pl.meta);
  w.rth = at<uint32_t>(x.ws, pl.rth);
  w.rtch = at<uint32_t>(x.ws, pl.rtch);
  w.gcnt = at<uint32_t>(x.ws, pl.gcnt);
  w.goff = at<uint32_t>(x.ws, pl.goff);
  w.ioff = at<uint32_t>(x.ws, pl.ioff);
  w.skb = at<uint32_t>(x.ws, pl.skb);
  w.slen = at<uint32_t>(x.ws, pl.slen);
  w.part = at<AccRow>(x.ws, pl.part);
  w.dur = x.k->dur_ns;
  w.match = x.match;
  w.P = x.p->n;
  w.counters = x.p->counters;
  w.rs = x.p->row_stride;
  w.cs = x.p->col_stride;
  w.absent = x.p->absent_mask;
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    if (x.agg_kind[c] == OPATTR_AGG_DWMEAN) w.dwmask |= 1u << c;
    else if (x.agg_kind[c] == OPATTR_AGG_MAX) w.maxmask |= 1u << c;
  }
  w.table = x.table;
  w.sum = x.sum;

  probe_begin(OPATTR_PROBE_AGGREGATE, s);
  note(hipMemsetAsync(w.gcnt, 0, (size_t)pl.G * 4, s));
  if (pl.T > 0) {
    launch_scan_excl(w.slots.nruns, at<uint32_t>(x.ws, pl.roff), pl.nencb, w.meta, s);
    k_run_compact<<<(unsigned)((pl.nencb + 3) / 4), 256, 0, s>>>(w);
    k_run_hist<<<(unsigned)pl.ntrt, 256, 0, s>>>(w);
    column_scan(w.rth, pl.ntrt, pl.G, w.rtch, w.gcnt, s, w.meta + 1);
  } else {
    note(hipMemsetAsync(w.meta, 0, 3 * sizeof(int64_t), s));
  }
  k_row_offsets<<<1, 1024, 0, s>>>(w);
  if (pl.T > 0) {
    k_run_scatter<<<(unsigned)pl.ntrt, 256, 0, s>>>(w);
    const int64_t max_items = pl.T / kRunsPerItem + pl.G + 1;
    const unsigned grid = (unsigned)(max_items < 16384 ? max_items : 16384);
    k_reduce<<<grid, 256, 0, s>>>(w);
  }
  k_combine<<<(pl.G + 3) / 4, 256, 0, s>>>(w);
  k_summary<<<1, 1024, 0, s>>>(w);
  probe_end(OPATTR_PROBE_AGGREGATE, s);
}

int64_t max_agg_items(int64_t T, uint32_t G) { return T / kRunsPerItem + G + 1; }

}  // namespace opa
