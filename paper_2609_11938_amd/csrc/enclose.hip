// Enclosure (Alg. 2) in one pass over the timeline, emitting the operator
// runs that the aggregation reduces.
//
// Each block takes 256 consecutive launches. The range starts that can matter
// for the block's main stream (those between the block's smallest and largest
// query point) are staged in LDS; the two bounds are found by 64-ary searches
// in which every lane of a wave probes one sample. A launch's innermost range
// is the last range starting at or before its query point, lifted along the
// parent chain while that range ends before the query point.
//
// For the aggregation the block then cuts its launches into runs of equal
// operator row (consecutive launches of one range are one run) and writes one
// (row, first launch, length) record per run into its own slot area; no
// accumulation happens here.
#include "common.h"
#include "impl.h"

namespace opa {

struct EncParams {
  int64_t T;
  const uint64_t *q;  // query_ns or start_ns
  const uint16_t *stream;
  const int32_t *match;
  int64_t P;
  CoreRanges cr;
  const int64_t *rblk;
  const int64_t *ree;
  const int32_t *npg;
  uint32_t NS, NOPS;
  int64_t R_in;           // aggregate-only: input ranges
  const uint32_t *op_in;  // aggregate-only: op ids by input range index
  int32_t *range_id;
  RunSlots runs;
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

template <int MODE>
__global__ void __launch_bounds__(kEncThreads) k_enc(EncParams a) {
  __shared__ uint64_t sS[kEncWindow];
  __shared__ uint64_t red[2][kEncThreads / OPA_WAVE];
  __shared__ int64_t win[3];
  __shared__ uint32_t sg[kEncThreads];
  __shared__ uint32_t rstart[kEncThreads];
  __shared__ uint32_t sh[8];
  __shared__ uint32_t sbad;
  const int tid = threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.x * kEncThreads;
  const int64_t i = i0 + tid;
  const bool valid = i < a.T;
  if (tid == 0) sbad = 0;
  uint32_t bad = 0;
  uint32_t g = a.NOPS;

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
    // runs of equal operator row among the block's launches, in launch order
    if (valid) {
      const int32_t m = a.match[i];
      if (m < -1 || m >= a.P) bad++;  // such a launch aggregates as unmatched
    }
    sg[tid] = valid ? g : 0xFFFFFFFFu;
    __syncthreads();
    const bool head = valid && (tid == 0 || sg[tid - 1] != g);
    uint32_t nr;
    const uint32_t r = block_excl_scan_add<uint32_t>(head ? 1u : 0u, sh, &nr);
    if (head) rstart[r] = (uint32_t)tid;
    __syncthreads();
    const bool tail = valid && (tid == kEncThreads - 1 || sg[tid + 1] != g);
    if (tail) {
      const uint32_t rr = r + (head ? 1u : 0u) - 1u;  // this launch's run
      const uint32_t s0 = rstart[rr];
      const int64_t slot = (int64_t)blockIdx.x * kEncThreads + rr;
      a.runs.g[slot] = g;
      a.runs.kb[slot] = (uint32_t)(i0 + s0);
      a.runs.len[slot] = (uint32_t)(tid - s0 + 1);
    }
    if (tid == 0) a.runs.nruns[blockIdx.x] = nr;
  }
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (tid == 0 && sbad)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)sbad);
}

void run_enclose_aggregate(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const opattr_kernels *k = x.k;
  EncParams a{};
  a.T = pl.T;
  a.q = k->query_ns ? k->query_ns : k->start_ns;
  a.stream = k->stream_id;
  a.match = x.match;
  a.P = x.p ? x.p->n : 0;
  a.NS = x.d->n_streams;
  a.NOPS = x.d->n_ops;
  a.range_id = x.range_id;
  a.diag = x.diag;
  a.cr = x.cr;
  a.rblk = at<int64_t>(x.ws, pl.rblk);
  a.ree = at<int64_t>(x.ws, pl.ree);
  a.npg = at<int32_t>(x.ws, pl.npg);
  a.runs = run_slots(x.ws, pl);
  if (x.mode == kAggregateOnly) {
    a.R_in = x.r ? x.r->n : 0;
    a.op_in = x.r ? x.r->op_id : nullptr;
  }
  const unsigned nb = (unsigned)pl.nencb;
  probe_begin(OPATTR_PROBE_MAIN_PASS, s);
  if (pl.T > 0) {
    if (x.mode == kEncloseOnly) k_enc<1><<<nb, kEncThreads, 0, s>>>(a);
    else if (x.mode == kAggregateOnly) k_enc<2><<<nb, kEncThreads, 0, s>>>(a);
    else k_enc<3><<<nb, kEncThreads, 0, s>>>(a);
  }
  probe_end(OPATTR_PROBE_MAIN_PASS, s);
  if (x.mode & 2) run_aggregate(x, s);
}

}  // namespace opa
