// The attribution's last passes on the segment path of opattr_attribute:
// layer-dedup broadcast (Sec. 3.7) and aggregation (Eq. 1, Sec. 3.8.1) over
// the launches in storage order.
//
// 1. k_f_agg: each lane takes eight consecutive launches. Their matches come
//    first: the matching leaves, by seq rank, the row and name of every
//    eligible launch (mbs, nbs); each launch takes its own entry, and a
//    duplicate the entry of the representative's launch at the same
//    position (the partition record gives the seq offset) when the names
//    agree (else -1 and a dedup error). The lane then adds the launches'
//    durations and counter rows (m or m * d, or the fp32 maximum as an
//    order-preserving key) into a register accumulator. Consecutive
//    launches of one operator row form a run: a run that ends inside a lane
//    is staged in LDS; the piece a lane ends with is carried across the
//    wave by a segmented lane scan. A block keeps up to 128 partial results,
//    sorts them by bucket of operator rows (256 buckets, then the
//    unattributed row on its own) and writes them to its own region with a
//    (count, offset) entry per bucket; anything past that goes to a row
//    accumulator with device-scope atomics. The blocks are taken per XCD in
//    the order k_f_order gives (launch-order windows).
// 2. k_f_comb: one wave per (bucket, share of the blocks) adds the bucket's
//    partial results of those blocks in LDS (each partial read field-wise
//    by 25 lanes) and writes one partial per row; 32 more waves add the
//    unattributed row's partials.
// 3. k_f_rows: one block per bucket adds every share and the row
//    accumulators and writes the bucket's table rows (DW-mean = sum /
//    matched ns, NaN rules) and summary sums; the last block to finish
//    writes the summary and the status.
// Integer fields are exact in any order; fp64 sums are added in an order
// that depends on scheduling (well inside the 1e-9 tolerance); maxima are
// exact.
#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kAPer = 8;                      // launches per lane (aggregation)
constexpr int kAHalf = 8;                      // of them in registers at a time
constexpr int kAThreads = 256;                 // threads per block
constexpr int kASpan = kAPer * kAThreads;      // launches per block
constexpr int kASlots = 32;                    // partial results a wave keeps
constexpr int kABlockCap = kASlots * (kAThreads / OPA_WAVE);  // and a block
constexpr int kFFields = 25;                   // kc, tns, mc, mns, 20 counters, NaN bits
constexpr int kBuckets = 256;                  // buckets of operator rows
// A block's bucket entries: the buckets, then the unattributed row (NOPS) on
// its own: it has a partial in almost every block, which would make its
// bucket's combine waves the last to finish by far.
constexpr int kBktStride = kBuckets + 1;
constexpr int kHot = 32;                       // combine waves of the unattributed row
constexpr int kSplits = 16;                    // shares of the blocks per bucket
constexpr int kPre = 8;                        // bucket entries a combine lane fetches at once
constexpr int kList = 512;                     // partials a combine wave lists in LDS at once
constexpr int kBatch = 8;                      // partial loads per lane in flight
constexpr uint32_t kNoSrc = 0xFFFFFFFFu;
constexpr uint32_t kHash = 256;                // LDS table of a block's rows (> 2 x kept)


static_assert(kABlockCap <= 255, "bucket offsets fit in a byte");
static_assert(kBuckets <= kSumBlocks, "one summary partial per bucket fits the summary workspace");

// kN consecutive 32-bit elements from p[i..), 16-byte vector loads when aligned
template <int kN, typename T>
__device__ __forceinline__ void load_n(const T *p, int64_t i, int nv, T (&o)[kN]) {
  static_assert(sizeof(T) == 4 && kN % 4 == 0, "32-bit elements, whole vectors");
  if (nv == kN && (reinterpret_cast<uintptr_t>(p + i) & 15) == 0) {
    const uint4 *v = reinterpret_cast<const uint4 *>(p + i);
#pragma unroll
    for (int q = 0; q < kN / 4; ++q) {
      const uint4 t = v[q];
      memcpy(reinterpret_cast<char *>(o) + 16 * q, &t, 16);
    }
  } else {
#pragma unroll
    for (int k = 0; k < kN; ++k) o[k] = k < nv ? p[i + k] : T(0);
  }
}

template <int kN, typename T>
__device__ __forceinline__ void store_n(T *p, int64_t i, int nv, const T (&o)[kN]) {
  if (nv == kN && (reinterpret_cast<uintptr_t>(p + i) & 15) == 0) {
    uint4 *v = reinterpret_cast<uint4 *>(p + i);
#pragma unroll
    for (int q = 0; q < kN / 4; ++q) {
      uint4 t;
      memcpy(&t, reinterpret_cast<const char *>(o) + 16 * q, 16);
      v[q] = t;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kN; ++k)
      if (k < nv) p[i + k] = o[k];
  }
}

// ---------------------------------------------------------------------------
// matches
// ---------------------------------------------------------------------------
struct MatchParams {
  int64_t T;
  const uint32_t *seq, *name;
  const int32_t *part;   // NULL: no partitions
  const PartRec *prec;   // the partition records (NULL: no partitions)
  uint32_t NN, NP;
  const int32_t *mbs;    // by seq rank: row of each eligible launch
  const uint32_t *nbs;   // by seq rank: its name
  int32_t *match;        // out
  opattr_diag *diag;
};

// The matches of kN consecutive launches from i (nv of them exist), stored to
// a.match; dedup errors are added to err.
template <int kN>
__device__ __forceinline__ void match_of(const MatchParams &a, int64_t i, int nv,
                                         int32_t (&mt)[kN], uint32_t &err) {
  uint32_t sq[kN], nm[kN];
  int32_t pt[kN];
  load_n<kN>(a.seq, i, nv, sq);
  load_n<kN>(a.name, i, nv, nm);
  if (a.part) load_n<kN>(a.part, i, nv, pt);
  else
#pragma unroll
    for (int k = 0; k < kN; ++k) pt[k] = -1;
  PartRec rc[kN];
#pragma unroll
  for (int k = 0; k < kN; ++k) {
    const bool ok = k < nv && nm[k] < a.NN && (int64_t)sq[k] < a.T && pt[k] >= -1 &&
                    (pt[k] < 0 || (uint32_t)pt[k] < a.NP);
    rc[k] = PartRec{0, ok ? kRecEligible : kRecNone};
    if (ok && pt[k] >= 0) rc[k] = a.prec[pt[k]];
  }
  uint32_t src[kN], dup = 0;
#pragma unroll
  for (int k = 0; k < kN; ++k) {
    const uint32_t hi = rc[k].hi;
    src[k] = kNoSrc;
    if (hi == kRecEligible) {
      src[k] = sq[k];
    } else if (hi != kRecNone) {
      const uint32_t x = sq[k] + (uint32_t)rc[k].delta;
      if (sq[k] < hi && (int64_t)x < a.T) {  // x < T always when seq is dense
        src[k] = x;
        dup |= 1u << k;
      } else {
        err++;
      }
    }
  }
  uint32_t sn[kN];
#pragma unroll
  for (int k = 0; k < kN; ++k) {
    mt[k] = src[k] != kNoSrc ? a.mbs[src[k]] : -1;
    sn[k] = ((dup >> k) & 1u) ? a.nbs[src[k]] : 0u;
  }
#pragma unroll
  for (int k = 0; k < kN; ++k)
    if (((dup >> k) & 1u) && sn[k] != nm[k]) {
      mt[k] = -1;
      err++;
    }
  store_n<kN>(a.match, i, nv, mt);
}

// ---------------------------------------------------------------------------
// 0. processing order of the run reduction's blocks. A block of 2048
// launches in storage order holds one stream's launches over a window of
// launch order; its duplicates read the matches (and the counter rows) of
// the representatives of that window, which every stream's blocks over the
// window read too. The blocks are ordered by the seq rank of their first
// launch (a counting sort into kOrderBuckets windows), and each XCD takes a
// contiguous part of that order, so that the blocks sharing those reads
// run at about the same time on one L2. The order only moves work between
// workgroups: every block still reduces its own launches.
// ---------------------------------------------------------------------------
constexpr int kOrderBuckets = 1024;
constexpr uint32_t kXcds = 8;  // workgroups go round robin over the XCDs in dispatch order

__global__ void __launch_bounds__(kOrderBuckets) k_f_order(const uint32_t *__restrict__ seq,
                                                           int64_t T, int64_t nb,
                                                           uint32_t *order) {
  __shared__ uint32_t hist[kOrderBuckets];
  __shared__ uint32_t sh[kOrderBuckets / OPA_WAVE];
  const int tid = threadIdx.x;
  hist[tid] = 0;
  __syncthreads();
  auto bucket = [&](int64_t b) -> uint32_t {
    const uint64_t q = seq[b * kASpan];
    const uint64_t c = q < (uint64_t)T ? q : (uint64_t)T - 1;  // a broken promise: any window
    return (uint32_t)(c * kOrderBuckets / (uint64_t)T);
  };
  for (int64_t b = tid; b < nb; b += kOrderBuckets) atomicAdd(&hist[bucket(b)], 1u);
  __syncthreads();
  uint32_t tot;
  const uint32_t base = block_excl_scan_add<uint32_t>(hist[tid], sh, &tot);
  __syncthreads();
  hist[tid] = base;
  __syncthreads();
  for (int64_t b = tid; b < nb; b += kOrderBuckets)
    order[atomicAdd(&hist[bucket(b)], 1u)] = (uint32_t)b;
}

// The block workgroup i reduces: dispatch index i runs on XCD i % kXcds,
// and XCD x takes the part of the order after the parts of XCDs 0 .. x-1
// (without an order, block i).
__device__ __forceinline__ int64_t order_slot(const uint32_t *order, uint32_t i, uint32_t n) {
  if (!order) return i;
  const uint32_t x = i % kXcds, t = i / kXcds;
  uint32_t before = 0;
  for (uint32_t y = 0; y < x; ++y) before += (n - y + kXcds - 1) / kXcds;
  return order[before + t];
}

// ---------------------------------------------------------------------------
// 1. runs
// ---------------------------------------------------------------------------
struct AggParams {
  int64_t T;
  MatchParams m;            // the matching's inputs; m.match is written here
  const int32_t *range_id;  // innermost (or walked) range, input index, or -1
  const uint32_t *op_in;    // op id of each input range
  int64_t R_in;
  uint32_t NOPS, rb;        // rb: operator rows per bucket
  AggIn in;
  PartRow *acc;             // [G] row accumulators for what blocks do not keep (zeroed)
  PartRow *parts;           // [blocks][kABlockCap] kept partials, by bucket (row in pad)
  uint16_t *bkt;            // [blocks][kBktStride] offset << 8 | count
  const uint32_t *order;    // [blocks] processing order (k_f_order), or NULL
};

// A partial result staged in LDS: its 25 fields and its row (live 0: merged
// into the neighbouring lane's piece instead).
struct Slot {
  unsigned long long f[kFFields];
  uint32_t g, live;
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// a += partial result of some launches of row g, one lane at a time
// (device-scope atomics; only for what a block cannot keep)
__device__ __forceinline__ void acc_to_table(PartRow *acc, uint32_t g, const Acc &a,
                                             uint32_t mx) {
  PartRow *r = acc + g;
  atomicAdd(&r->kc, a.kc);
  atomicAdd(&r->tns, a.tns);
  if (a.mc == 0) return;  // no counter row reached: every counter field is still zero
  atomicAdd(&r->mc, a.mc);
  atomicAdd(&r->mns, a.mns);
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    if ((mx >> c) & 1u) atomicMax(&r->v[c], a.v[c]);
    else unsafeAtomicAdd(reinterpret_cast<double *>(&r->v[c]), bits2d(a.v[c]));
  }
  if (a.nan) atomicOr(&r->nan, a.nan);
}

// Stage the partial of every lane with want set (row g) in the wave's slots;
// returns the lane's slot, or -1 when the slots are full (then the partial
// goes to the accumulator). Called by the whole wave; n is wave-uniform.
__device__ __forceinline__ int stage_put(bool want, uint32_t g, const Acc &a, Slot *slot, int &n,
                                         PartRow *acc, uint32_t mx) {
  const unsigned long long m = __ballot(want);
  if (!m) return -1;
  const int r = __popcll(m & lanemask_lt());
  int idx = -1;
  if (want) {
    if (n + r < kASlots) {
      idx = n + r;
      Slot *q = slot + idx;
      q->f[0] = a.kc;
      q->f[1] = a.tns;
      q->f[2] = a.mc;
      q->f[3] = a.mns;
#pragma unroll
      for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) q->f[4 + c] = a.v[c];
      q->f[24] = a.nan;
      q->g = g;
      q->live = 1;
    } else {
      acc_to_table(acc, g, a, mx);
    }
  }
  const int tot = n + __popcll(m);
  n = tot < kASlots ? tot : kASlots;
  return idx;
}

// a += the staged partial q (a piece of the same run, after a's launches)
__device__ __forceinline__ void acc_merge_slot(Acc &a, const Slot *q, uint32_t mx) {
  a.kc += q->f[0];
  a.tns += q->f[1];
  a.mc += q->f[2];
  a.mns += q->f[3];
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    const unsigned long long y = q->f[4 + c];
    if ((mx >> c) & 1u) a.v[c] = y > a.v[c] ? y : a.v[c];
    else a.v[c] = d2bits(bits2d(a.v[c]) + bits2d(y));
  }
  a.nan |= (uint32_t)q->f[24];
}

__device__ __forceinline__ uint32_t row_of(const AggParams &a, int32_t rid) {
  uint32_t g = a.NOPS;
  if (rid >= 0 && rid < a.R_in) {
    const uint32_t o = a.op_in[rid];
    g = o < a.NOPS ? o : a.NOPS;
  }
  return g;
}

// The operator rows of kN launches: every gather is issued before the first
// is used (an out-of-range id reads entry 0 and is replaced afterwards), so
// their latencies overlap instead of adding up.
template <int kN>
__device__ __forceinline__ void rows_of(const AggParams &a, const int32_t (&rid)[kN], int nh,
                                        uint32_t (&g)[kN]) {
  if (a.R_in > 0) {
    uint32_t o[kN];
#pragma unroll
    for (int k = 0; k < kN; ++k) o[k] = a.op_in[(rid[k] >= 0 && rid[k] < a.R_in) ? rid[k] : 0];
#pragma unroll
    for (int k = 0; k < kN; ++k) {
      const bool ok = rid[k] >= 0 && rid[k] < a.R_in && o[k] < a.NOPS;
      g[k] = k < nh ? (ok ? o[k] : a.NOPS) : 0xFFFFFFFFu;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kN; ++k) g[k] = k < nh ? a.NOPS : 0xFFFFFFFFu;
  }
}

template <bool DEF>  // DEF: the default aggregation kinds
__global__ void __launch_bounds__(kAThreads) __attribute__((amdgpu_waves_per_eu(3)))
k_f_agg(AggParams a) {
  __shared__ Slot slots[kAThreads / OPA_WAVE][kASlots];
  __shared__ int nslot[kAThreads / OPA_WAVE];
  __shared__ uint32_t hist[kBktStride], spos[kABlockCap];
  __shared__ uint32_t hkey[kHash], hown[kHash];
  __shared__ uint32_t sh[4];
  const int tid = threadIdx.x, ln = lane_id(), w = wave_id();
  const AggIn &in = a.in;
  const uint32_t mx = DEF ? kDefMaxMask : in.maxmask, dw = DEF ? kDefDwMask : in.dwmask;
  const int64_t blk = order_slot(a.order, blockIdx.x, gridDim.x);
  const int64_t ib = blk * kASpan + (int64_t)tid * kAPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kAPer ? a.T - ib : kAPer));
  Slot *wslot = slots[w];
  int nst = 0;      // staged partials of the wave (uniform)
  int fslot = -1;   // the staged first piece of this lane (it continues the previous lane's run)
  uint32_t hm = 0;  // bit k: launch k starts a run (the wave's first launch always does)
  Acc inc;
  acc_zero(inc);
  // the operator row of the launch before the lane's first (the wave's first
  // launch starts a run whatever it is)
  uint32_t gprev = 0xFFFFFFFFu;
  if (ln > 0 && nv > 0) gprev = row_of(a, a.range_id[ib - 1]);
  uint32_t gcur = 0xFFFFFFFFu;
  uint32_t err = 0;  // dedup errors of the lane's launches
#pragma unroll 1
  for (int h = 0; h < kAPer / kAHalf; ++h) {
    const int64_t i0 = ib + h * kAHalf;
    const int nh = nv - h * kAHalf < 0 ? 0 : (nv - h * kAHalf < kAHalf ? nv - h * kAHalf : kAHalf);
    int32_t mt[kAHalf], rid[kAHalf];
    uint32_t du[kAHalf], g[kAHalf];
    match_of<kAHalf>(a.m, i0, nh, mt, err);
    load_n<kAHalf>(in.dur, i0, nh, du);
    load_n<kAHalf>(a.range_id, i0, nh, rid);
    rows_of<kAHalf>(a, rid, nh, g);
#pragma unroll
    for (int k = 0; k < kAHalf; ++k) {
      const int kk = h * kAHalf + k;
      const uint32_t prev = k ? g[k - 1] : gprev;
      if (k < nh && g[k] != prev) hm |= 1u << kk;
    }
    gprev = g[kAHalf - 1];
    if (h == 0) gcur = g[0];
    // launch k is always at position 0 of the arrays: they shift by one per
    // step (a run-time index would move them to scratch memory). The loop
    // is uniform over the wave: staging is cooperative.
#pragma unroll 1
    for (int k = 0; k < kAHalf; ++k) {
      const int kk = h * kAHalf + k;
      const bool cut = kk > 0 && k < nh && ((hm >> kk) & 1u);
      const int idx = stage_put(cut, gcur, inc, wslot, nst, a.acc, mx);
      // the lane's first piece continues the previous lane's run
      if (cut && (hm & 1u) == 0 && (hm & ((1u << kk) - 1u)) == 0) fslot = idx;
      if (cut) {
        acc_zero(inc);
        gcur = g[0];
      }
      if (k < nh) acc_launch(inc, in, mt[0], du[0], mx, dw);
#pragma unroll
      for (int j = 0; j + 1 < kAHalf; ++j) {
        mt[j] = mt[j + 1];
        du[j] = du[j + 1];
        g[j] = g[j + 1];
      }
    }
  }
  // the next lane's first piece belongs to the run this lane ends with
  wave_sync_lds();
  {
    int fi = __shfl_down(fslot, 1, OPA_WAVE);
    if (ln == OPA_WAVE - 1) fi = -1;
    if (fi >= 0) {
      acc_merge_slot(inc, wslot + fi, mx);
      wslot[fi].live = 0;
    }
  }
  wave_sync_lds();
  // the piece each lane ends with, carried across the lanes: a segment
  // starts at every lane whose last piece starts inside it
  const unsigned long long hl = __ballot(hm != 0) | 1ull;
  const unsigned long long upto = ln == 63 ? ~0ull : ((2ull << ln) - 1);
  const int sl = 63 - __clzll(hl & upto);
  acc_seg_scan(inc, sl, mx);
  // the run goes on into the next lane only if that lane has launches and
  // no run start at all
  const uint32_t nvn = __shfl_down((uint32_t)nv, 1, OPA_WAVE);
  const uint32_t hmn = __shfl_down(hm, 1, OPA_WAVE);
  stage_put(nv > 0 && (ln == OPA_WAVE - 1 || nvn == 0 || hmn != 0), gcur, inc, wslot, nst, a.acc,
            mx);
  if (ln == 0) nslot[w] = nst;
  {
    const unsigned long long e = wave_reduce_add((unsigned long long)err);
    if (ln == 0 && e) atomicAdd((unsigned long long *)&a.m.diag->dedup_errors, e);
  }
  for (int q = tid; q < kBktStride; q += kAThreads) hist[q] = 0;
  for (int q = tid; q < kHash; q += kAThreads) {
    hkey[q] = 0u;
    hown[q] = 0xFFFFFFFFu;
  }
  __syncthreads();

  // the block's kept partials of one row are added into the first of them
  // (a busy row, such as the unattributed one, would otherwise reach the
  // combine once per run), then counted by bucket and written in bucket order
  // (an open-addressing table of rows in LDS: the lowest slot of a row owns it)
  bool own = false;
  int hs = -1;
  const Slot *qs = nullptr;
  if (tid < kABlockCap) {
    const int sw = tid / kASlots, sj = tid % kASlots;
    qs = &slots[sw][sj];
    if (sj < nslot[sw] && qs->live) {
      const uint32_t key = qs->g + 1u;
      uint32_t h = (qs->g * 2654435761u) >> 24;
      for (;;) {
        const uint32_t old = atomicCAS(&hkey[h], 0u, key);
        if (old == 0u || old == key) break;
        h = (h + 1u) & (kHash - 1u);
      }
      atomicMin(&hown[h], (uint32_t)tid);
      hs = (int)h;
    }
  }
  __syncthreads();
  if (hs >= 0) {
    const uint32_t first = hown[hs];
    own = first == (uint32_t)tid;
    if (!own) {
      Slot *o = &slots[first / kASlots][first % kASlots];
      atomicAdd(&o->f[0], qs->f[0]);
      atomicAdd(&o->f[1], qs->f[1]);
      atomicAdd(&o->f[2], qs->f[2]);
      atomicAdd(&o->f[3], qs->f[3]);
#pragma unroll
      for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
        if ((mx >> c) & 1u) atomicMax(&o->f[4 + c], qs->f[4 + c]);
        else unsafeAtomicAdd(reinterpret_cast<double *>(&o->f[4 + c]), bits2d(qs->f[4 + c]));
      }
      if ((uint32_t)qs->f[24])
        atomicOr(reinterpret_cast<unsigned int *>(&o->f[24]), (uint32_t)qs->f[24]);
    }
  }
  __syncthreads();
  uint32_t bq = 0xFFFFFFFFu, rk = 0;
  if (own) {
    const uint32_t g = slots[tid / kASlots][tid % kASlots].g;
    bq = g == a.NOPS ? (uint32_t)kBuckets : g / a.rb;
    rk = atomicAdd(&hist[bq], 1u);
  }
  __syncthreads();
  uint32_t cnt = 0, tot;
  if (tid < kBuckets) cnt = hist[tid];
  const uint32_t off = block_excl_scan_add<uint32_t>(tid < kBuckets ? cnt : 0u, sh, &tot);
  const uint32_t hcnt = hist[kBuckets];  // the unattributed row's partial goes last
  if (tid < kBuckets)
    a.bkt[blk * kBktStride + tid] = (uint16_t)((off << 8) | cnt);
  if (tid == 0) a.bkt[blk * kBktStride + kBuckets] = (uint16_t)((tot << 8) | hcnt);
  __syncthreads();
  if (tid < kBuckets) hist[tid] = off;
  if (tid == 0) hist[kBuckets] = tot;
  __syncthreads();
  if (tid < kABlockCap) spos[tid] = bq != 0xFFFFFFFFu ? hist[bq] + rk : 0xFFFFFFFFu;
  __syncthreads();
  // coalesced copy: consecutive threads take consecutive fields
  PartRow *dst = a.parts + blk * kABlockCap;
  for (int x = tid; x < kABlockCap * kFFields; x += kAThreads) {
    const int s = x / kFFields, f = x % kFFields;
    const uint32_t p = spos[s];
    if (p == 0xFFFFFFFFu) continue;
    const Slot *q = &slots[s / kASlots][s % kASlots];
    unsigned long long *d = reinterpret_cast<unsigned long long *>(dst + p);
    if (f < 24) d[f] = q->f[f];
    else d[24] = (unsigned long long)(uint32_t)q->f[24] | ((unsigned long long)q->g << 32);
  }
}

// ---------------------------------------------------------------------------
// 2. per bucket: the kept partials of a share of the blocks, added in LDS
// ---------------------------------------------------------------------------
struct CombParams {
  int64_t nblocks;
  uint32_t rb, G, NOPS;
  uint32_t mx, dw, absent;
  const PartRow *parts;
  const uint16_t *bkt;
  PartRow *split;              // [kBuckets][kSplits][rb]
  PartRow *hot;                // [kHot] the unattributed row's shares
  const PartRow *acc;          // [G] row accumulators (the blocks' overflow)
  opattr_op_row *table;
  unsigned long long *part;    // [kBuckets][4] summary sums per bucket
  // the finalisation, by the last block of the per-row reduction to finish
  uint32_t *done;              // blocks finished (zero at launch)
  opattr_diag *diag;
  const uint8_t *sflag;        // [ns] per-stream crossing flags
  uint32_t ns;
  opattr_summary *sum;
};

__device__ __forceinline__ unsigned long long merge_field(int f, unsigned long long x,
                                                          unsigned long long y, uint32_t mx) {
  if (f < 4) return x + y;
  if (f < 24) return ((mx >> (f - 4)) & 1u) ? (x > y ? x : y) : d2bits(bits2d(x) + bits2d(y));
  return x | y;
}

// t (one field f of an LDS row) += the field's value x
__device__ __forceinline__ void field_add(unsigned long long *t, int f, unsigned long long x,
                                          uint32_t mx) {
  if (f < 4) {
    atomicAdd(t, x);
  } else if (f < 24) {
    if ((mx >> (f - 4)) & 1u) atomicMax(t, x);
    else unsafeAtomicAdd(reinterpret_cast<double *>(t), bits2d(x));
  } else if ((uint32_t)x) {
    atomicOr(reinterpret_cast<unsigned int *>(t), (uint32_t)x);
  }
}

// A wave takes a share of the blocks for one bucket: its lanes fetch the
// blocks' bucket entries eight at a time, list the partial results those
// entries point to in LDS, and then read each partial with 25 lanes (one
// field each, two partials per load instruction, eight loads in flight), so
// that a partial costs two cache lines of requests instead of 25; the fields
// are added into the wave's LDS table of the bucket's rows. The unattributed
// row's waves add whole partials per lane in registers, then across the wave.
template <bool DEF>
__global__ void __launch_bounds__(64) k_f_comb(CombParams a) {
  extern __shared__ __align__(16) unsigned char comb_raw[];
  unsigned long long *tab = reinterpret_cast<unsigned long long *>(comb_raw);  // [rb][kFFields]
  const uint32_t mx = DEF ? kDefMaxMask : a.mx;
  const int ln = lane_id();
  if (blockIdx.x >= (unsigned)(kBuckets * kSplits)) {
    // the unattributed row: a share of the blocks, each lane adding its
    // blocks' partials in registers, then the lanes across the wave
    const int h = (int)blockIdx.x - kBuckets * kSplits;
    const int64_t per = (a.nblocks + kHot - 1) / kHot;
    const int64_t b_lo = (int64_t)h * per, b_hi = b_lo + per < a.nblocks ? b_lo + per : a.nblocks;
    unsigned long long racc[kFFields];
#pragma unroll
    for (int f = 0; f < kFFields; ++f) racc[f] = 0;
    for (int64_t b = b_lo + ln; b < b_hi; b += OPA_WAVE) {
      const uint32_t e = a.bkt[b * kBktStride + kBuckets];
      const uint32_t c = e & 0xFFu, o = e >> 8;
      const unsigned long long *pr =
          reinterpret_cast<const unsigned long long *>(a.parts + b * kABlockCap + o);
#pragma unroll 1
      for (uint32_t p = 0; p < c; ++p, pr += sizeof(PartRow) / 8)
#pragma unroll
        for (int f = 0; f < kFFields; ++f)
          racc[f] = merge_field(f, racc[f], f < 24 ? pr[f] : (pr[f] & 0xFFFFFFFFull), mx);
    }
#pragma unroll
    for (int o = OPA_WAVE / 2; o > 0; o >>= 1)
#pragma unroll
      for (int f = 0; f < kFFields; ++f)
        racc[f] = merge_field(f, racc[f], __shfl_xor(racc[f], o, OPA_WAVE), mx);
    if (ln < kFFields) {
      unsigned long long v = racc[0];
#pragma unroll
      for (int f = 1; f < kFFields; ++f) v = ln == f ? racc[f] : v;
      reinterpret_cast<unsigned long long *>(a.hot + h)[ln] = v;
    }
    return;
  }
  const uint32_t q = blockIdx.x / kSplits, s = blockIdx.x % kSplits;
  const uint32_t rb = a.rb, ne = rb * kFFields;
  for (uint32_t x = ln; x < ne; x += OPA_WAVE) tab[x] = 0;
  wave_sync_lds();
  const int64_t per = (a.nblocks + kSplits - 1) / kSplits;
  const int64_t b_lo = (int64_t)s * per, b_hi = b_lo + per < a.nblocks ? b_lo + per : a.nblocks;
  uint32_t *list = reinterpret_cast<uint32_t *>(tab + ne);  // [kList] partial indices
  const unsigned long long *parts64 = reinterpret_cast<const unsigned long long *>(a.parts);
  const int half = ln >> 5, f = ln & 31;
  for (int64_t b0 = b_lo; b0 < b_hi; b0 += (int64_t)OPA_WAVE * kPre) {
    // the lane's next kPre blocks' entries for the bucket, loads in flight together
    uint32_t ev[kPre], mine = 0;
#pragma unroll
    for (int k = 0; k < kPre; ++k) {
      const int64_t b = b0 + ln + (int64_t)OPA_WAVE * k;
      ev[k] = b < b_hi ? a.bkt[b * kBktStride + q] : 0u;
      mine += ev[k] & 0xFFu;
    }
    const uint32_t incl = wave_incl_scan_add<uint32_t>(mine);
    const uint32_t n = __shfl(incl, OPA_WAVE - 1, OPA_WAVE);
    if (n == 0) continue;
    if (n <= (uint32_t)kList) {
      // the partials listed in LDS, then read by 25 lanes each (two
      // partials per instruction, kBatch instructions in flight) and added
      // field by field
      uint32_t w = incl - mine;
#pragma unroll
      for (int k = 0; k < kPre; ++k) {
        const uint32_t c = ev[k] & 0xFFu;
        const uint32_t x0 = (uint32_t)((b0 + ln + (int64_t)OPA_WAVE * k) * kABlockCap) + (ev[k] >> 8);
        for (uint32_t p = 0; p < c; ++p) list[w++] = x0 + p;
      }
      wave_sync_lds();
      for (uint32_t i = 0; i < n; i += 2 * kBatch) {
        unsigned long long v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          const uint32_t idx = i + 2 * j + half;
          v[j] = (idx < n && f < kFFields)
                     ? parts64[(size_t)list[idx] * (sizeof(PartRow) / 8) + f] : 0ull;
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          const uint32_t g = (uint32_t)(__shfl(v[j], (ln & 32) + 24, OPA_WAVE) >> 32);
          const uint32_t idx = i + 2 * j + half;
          if (idx < n && f < kFFields) field_add(tab + (size_t)(g % rb) * kFFields + f, f, v[j], mx);
        }
      }
    } else {
      // more partials than the list holds (rare): one lane's entry at a
      // time, its partials read two at a time by 25 lanes each
#pragma unroll 1
      for (int k = 0; k < kPre; ++k) {
        uint32_t e = 0;
#pragma unroll
        for (int j = 0; j < kPre; ++j) e = k == j ? ev[j] : e;
        for (uint64_t m = __ballot((e & 0xFFu) != 0); m; m &= m - 1) {
          const int src = __ffsll((unsigned long long)m) - 1;
          const uint32_t es = __shfl(e, src, OPA_WAVE), c = es & 0xFFu;
          const uint64_t x0 = (uint64_t)((b0 + src + (int64_t)OPA_WAVE * k) * kABlockCap) + (es >> 8);
          for (uint32_t p = 0; p < c; p += 2) {
            const uint32_t pp = p + half;
            const unsigned long long v = (pp < c && f < kFFields)
                ? parts64[(x0 + pp) * (sizeof(PartRow) / 8) + f] : 0ull;
            const uint32_t g = (uint32_t)(__shfl(v, (ln & 32) + 24, OPA_WAVE) >> 32);
            if (pp < c && f < kFFields) field_add(tab + (size_t)(g % rb) * kFFields + f, f, v, mx);
          }
        }
      }
    }
    wave_sync_lds();
  }
  unsigned long long *out =
      reinterpret_cast<unsigned long long *>(a.split + ((size_t)q * kSplits + s) * rb);
  for (uint32_t x = ln; x < ne; x += OPA_WAVE) {
    const uint32_t rr = x / kFFields, ff = x % kFFields;
    out[rr * (sizeof(PartRow) / 8) + ff] = tab[x];
  }
}

// ---------------------------------------------------------------------------
// 4. per bucket (one block): the row accumulators plus every share, then the
// bucket's table rows (DW-mean = sum / matched ns, NaN rules) and its summary
// sums (attributed, unattributed, total, matched ns)
// ---------------------------------------------------------------------------
template <bool DEF>
__global__ void __launch_bounds__(256) k_f_rows(CombParams a) {
  extern __shared__ __align__(16) unsigned char rows_raw[];
  unsigned long long *tab = reinterpret_cast<unsigned long long *>(rows_raw);  // [rb][kFFields]
  __shared__ unsigned long long red[4][4];
  const uint32_t mx = DEF ? kDefMaxMask : a.mx, dw = DEF ? kDefDwMask : a.dw;
  const int tid = threadIdx.x, ln = lane_id();
  const uint32_t q = blockIdx.x, rb = a.rb, ne = rb * kFFields;
  // element x = row * 25 + field: its accumulator and all its shares at once
  for (uint32_t x = tid; x < ne; x += blockDim.x) {
    const uint32_t rr = x / kFFields, ff = x % kFFields;
    const uint32_t g = q * rb + rr;
    const unsigned long long *sp =
        reinterpret_cast<const unsigned long long *>(a.split + (size_t)q * kSplits * rb) +
        (size_t)rr * (sizeof(PartRow) / 8) + ff;
    unsigned long long y[kSplits + 1];
    y[kSplits] = g < a.G ? reinterpret_cast<const unsigned long long *>(a.acc + g)[ff] : 0ull;
#pragma unroll
    for (int k = 0; k < kSplits; ++k) y[k] = sp[(size_t)k * rb * (sizeof(PartRow) / 8)];
    unsigned long long v = y[kSplits];
#pragma unroll
    for (int k = 0; k < kSplits; ++k) v = merge_field((int)ff, v, y[k], mx);
    if (g == a.NOPS) {  // the unattributed row's own shares, loads in flight together
      unsigned long long hv[kHot];
#pragma unroll
      for (int h = 0; h < kHot; ++h) hv[h] = reinterpret_cast<const unsigned long long *>(a.hot + h)[ff];
#pragma unroll
      for (int h = 0; h < kHot; ++h) v = merge_field((int)ff, v, hv[h], mx);
    }
    tab[x] = v;
  }
  __syncthreads();
  unsigned long long at_ = 0, un = 0, tot = 0, mt = 0;
  for (uint32_t rr = tid; rr < rb; rr += blockDim.x) {
    const uint32_t g = q * rb + rr;
    if (g >= a.G) break;
    const unsigned long long *f = tab + (size_t)rr * kFFields;
    opattr_op_row *row = a.table + g;
    const unsigned long long kc = f[0], tns = f[1], mc = f[2], mns = f[3];
    const uint32_t nan = (uint32_t)f[24];
    row->kernel_count = kc;
    row->total_ns = tns;
    row->matched_count = mc;
    row->matched_ns = mns;
    const double qnan = __longlong_as_double(0x7FF8000000000000ll);
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      double v;
      if (((a.absent >> c) & 1u) || mc == 0) v = qnan;
      else if ((mx >> c) & 1u) v = ((nan >> c) & 1u) ? qnan : (double)key2f((uint32_t)f[4 + c]);
      else if ((dw >> c) & 1u) v = mns ? bits2d(f[4 + c]) / (double)mns : qnan;
      else v = bits2d(f[4 + c]);
      row->value[c] = v;
    }
    tot += tns;
    mt += mns;
    if (g < a.NOPS) at_ += tns;
    else un += tns;
  }
  at_ = wave_reduce_add(at_);
  un = wave_reduce_add(un);
  tot = wave_reduce_add(tot);
  mt = wave_reduce_add(mt);
  if (ln == 0) {
    red[0][wave_id()] = at_;
    red[1][wave_id()] = un;
    red[2][wave_id()] = tot;
    red[3][wave_id()] = mt;
  }
  __syncthreads();
  if (tid < 4) a.part[q * 4 + tid] = red[tid][0] + red[tid][1] + red[tid][2] + red[tid][3];
  // the last block to finish reads every block's sums: the wave that wrote
  // them makes them visible device-wide before it counts the block done, and
  // in the last block that wave orders the block's reads after the count
  __shared__ uint32_t last;
  if (tid < OPA_WAVE) {
    __threadfence();
    uint32_t l = 0;
    if (tid == 0) l = atomicAdd(a.done, 1u) == gridDim.x - 1 ? 1u : 0u;
    l = __shfl(l, 0);
    if (l) __threadfence();
    if (tid == 0) last = l;
  }
  __syncthreads();
  if (!last) return;
  finish_block(a.diag, a.sflag, a.ns, a.part, (int)gridDim.x, a.sum);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
uint32_t fused_rows_per_bucket(uint32_t G) { return (G + kBuckets - 1) / kBuckets; }

int64_t fused_agg_blocks(int64_t T) { return (T + kASpan - 1) / kASpan; }

size_t fused_parts_bytes(int64_t T) {
  return (size_t)fused_agg_blocks(T) * kABlockCap * sizeof(PartRow);
}

size_t fused_bkt_bytes(int64_t T) { return (size_t)fused_agg_blocks(T) * kBktStride * 2; }

size_t fused_hot_bytes() { return (size_t)kHot * sizeof(PartRow); }

size_t fused_split_bytes(uint32_t G) {
  return (size_t)kBuckets * kSplits * fused_rows_per_bucket(G) * sizeof(PartRow);
}


// the row accumulators, then the per-row reduction's count of finished blocks
size_t fused_acc_bytes(uint32_t G) { return (size_t)G * sizeof(PartRow) + 256; }

void fused_acc_clear(FillJobs &j, void *ws, const Plan &pl) {
  j.add(at<uint32_t>(ws, pl.acc), 0u, (int64_t)(fused_acc_bytes(pl.G) / 4));
}

void run_fused_order(const opattr_kernels *k, void *ws, const Plan &pl, hipStream_t s) {
  const int64_t nb = fused_agg_blocks(pl.T);
  if (nb > 0) k_f_order<<<1, kOrderBuckets, 0, s>>>(k->seq, pl.T, nb, at<uint32_t>(ws, pl.forder));
}

void run_fused_agg(const FusedIn &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const uint32_t rb = fused_rows_per_bucket(pl.G);
  AggParams a{};
  a.T = pl.T;
  MatchParams &m = a.m;
  m.T = pl.T;
  m.seq = x.k->seq;
  m.name = x.k->name_id;
  const bool dd = x.k->part_id && x.d->part_rep && x.d->n_parts > 0;
  m.part = dd ? x.k->part_id : nullptr;
  m.prec = dd ? at<PartRec>(x.ws, pl.prec) : nullptr;
  m.NN = x.d->n_names;
  m.NP = dd ? x.d->n_parts : 0;
  m.mbs = at<int32_t>(x.ws, pl.mbs);
  m.nbs = at<uint32_t>(x.ws, pl.nbs);
  m.match = x.match;
  m.diag = x.diag;
  a.range_id = x.range_id;
  a.op_in = x.r->op_id;
  a.R_in = x.r->n;
  a.NOPS = x.d->n_ops;
  a.rb = rb;
  a.in = *x.in;
  a.acc = at<PartRow>(x.ws, pl.acc);
  a.parts = at<PartRow>(x.ws, pl.fparts);
  a.bkt = at<uint16_t>(x.ws, pl.fbkt);
  const bool def = a.in.maxmask == kDefMaxMask && a.in.dwmask == kDefDwMask;
  const int64_t nb = fused_agg_blocks(pl.T);
  a.order = x.ordered ? at<uint32_t>(x.ws, pl.forder) : nullptr;  // from run_fused_order
  probe_begin(OPATTR_PROBE_AGG_RUNS, s);
  if (nb > 0) {
    if (def) k_f_agg<true><<<(unsigned)nb, kAThreads, 0, s>>>(a);
    else k_f_agg<false><<<(unsigned)nb, kAThreads, 0, s>>>(a);
  }
  probe_end(OPATTR_PROBE_AGG_RUNS, s);
  probe_begin(OPATTR_PROBE_AGGREGATE, s);
  CombParams c{};
  c.nblocks = nb;
  c.rb = rb;
  c.G = pl.G;
  c.NOPS = x.d->n_ops;
  c.mx = a.in.maxmask;
  c.dw = a.in.dwmask;
  c.absent = x.absent;
  c.parts = a.parts;
  c.bkt = a.bkt;
  c.split = at<PartRow>(x.ws, pl.fsplit);
  c.hot = at<PartRow>(x.ws, pl.fhot);
  c.acc = a.acc;
  c.table = x.table;
  c.part = at<unsigned long long>(x.ws, pl.sumpart);
  c.done = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(x.ws) + pl.acc +
                                        (size_t)pl.G * sizeof(PartRow));
  c.diag = x.diag;
  c.sflag = at<uint8_t>(x.ws, pl.sflag);
  c.ns = x.d->n_streams;
  c.sum = x.sum;
  const size_t lds = (size_t)rb * kFFields * 8;
  const size_t lds_comb = lds + (size_t)kList * 4;  // the table, then the partials' list
  if (def) {
    k_f_comb<true><<<kBuckets * kSplits + kHot, 64, lds_comb, s>>>(c);
    k_f_rows<true><<<kBuckets, 256, lds, s>>>(c);
  } else {
    k_f_comb<false><<<kBuckets * kSplits + kHot, 64, lds_comb, s>>>(c);
    k_f_rows<false><<<kBuckets, 256, lds, s>>>(c);
  }
  probe_end(OPATTR_PROBE_AGGREGATE, s);
}

}  // namespace opa
