// The attribution's last passes on the segment path of opattr_attribute:
// layer-dedup broadcast (Sec. 3.7) and aggregation (Eq. 1, Sec. 3.8.1) over
// the launches in storage order.
//
// 1. k_f_match: the matching leaves, by seq rank, the row and name of every
//    eligible launch (mbs, nbs). Each launch takes its own entry; a duplicate
//    takes the entry of the representative's launch at the same position
//    (the partition record gives the seq offset) when the names agree (else
//    -1 and a dedup error).
// 2. k_f_agg: each lane takes sixteen consecutive launches and adds their
//    durations and counter rows (m or m * d, or the fp32 maximum as an
//    order-preserving key) into a register accumulator. Consecutive launches
//    of one operator row form a run: a run that ends inside a lane is staged
//    in LDS; the piece a lane ends with is carried across the wave by a
//    segmented lane scan. A block keeps up to 128 partial results, sorts them
//    by bucket of operator rows (256 buckets) and writes them to its own
//    region with a (count, offset) entry per bucket; anything past that goes
//    to a row accumulator with device-scope atomics.
// 3. k_f_comb: one wave per (bucket, share of the blocks) adds the bucket's
//    partial results of those blocks in LDS and writes one partial per row.
// 4. k_f_rows: every table row from its shares and its accumulator
//    (DW-mean = sum / matched ns, NaN rules), and the summary's block sums.
// Integer fields are exact in any order; fp64 sums are added in an order
// that depends on scheduling (well inside the 1e-9 tolerance); maxima are
// exact.
#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kMPer = 8;                       // launches per thread (matching)
constexpr int kAPer = 16;                      // launches per lane (aggregation)
constexpr int kAHalf = 8;                      // of them in registers at a time
constexpr int kAThreads = 256;                 // threads per block
constexpr int kASpan = kAPer * kAThreads;      // launches per block
constexpr int kASlots = 48;                    // partial results a wave keeps
constexpr int kABlockCap = kASlots * (kAThreads / OPA_WAVE);  // and a block
constexpr int kFFields = 25;                   // kc, tns, mc, mns, 20 counters, NaN bits
constexpr int kBuckets = 256;                  // buckets of operator rows
constexpr int kSplits = 16;                    // shares of the blocks per bucket
constexpr uint32_t kNoSrc = 0xFFFFFFFFu;

static_assert(kAPer == 2 * kAHalf, "two halves per lane");
static_assert(kABlockCap <= 255, "bucket offsets fit in a byte");

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
// 1. matches
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

__global__ void __launch_bounds__(256) k_f_match(MatchParams a) {
  const int64_t ib = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kMPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kMPer ? a.T - ib : kMPer));
  uint32_t sq[kMPer], nm[kMPer];
  int32_t pt[kMPer];
  load_n<kMPer>(a.seq, ib, nv, sq);
  load_n<kMPer>(a.name, ib, nv, nm);
  if (a.part) load_n<kMPer>(a.part, ib, nv, pt);
  else
#pragma unroll
    for (int k = 0; k < kMPer; ++k) pt[k] = -1;
  PartRec rc[kMPer];
#pragma unroll
  for (int k = 0; k < kMPer; ++k) {
    const bool ok = k < nv && nm[k] < a.NN && (int64_t)sq[k] < a.T && pt[k] >= -1 &&
                    (pt[k] < 0 || (uint32_t)pt[k] < a.NP);
    rc[k] = PartRec{0, ok ? kRecEligible : kRecNone};
    if (ok && pt[k] >= 0) rc[k] = a.prec[pt[k]];
  }
  uint32_t src[kMPer], dup = 0, err = 0;
#pragma unroll
  for (int k = 0; k < kMPer; ++k) {
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
  int32_t mt[kMPer];
  uint32_t sn[kMPer];
#pragma unroll
  for (int k = 0; k < kMPer; ++k) {
    mt[k] = src[k] != kNoSrc ? a.mbs[src[k]] : -1;
    sn[k] = ((dup >> k) & 1u) ? a.nbs[src[k]] : 0u;
  }
#pragma unroll
  for (int k = 0; k < kMPer; ++k)
    if (((dup >> k) & 1u) && sn[k] != nm[k]) {
      mt[k] = -1;
      err++;
    }
  store_n<kMPer>(a.match, ib, nv, mt);
  const unsigned long long e = wave_reduce_add((unsigned long long)err);
  if (lane_id() == 0 && e) atomicAdd((unsigned long long *)&a.diag->dedup_errors, e);
}

// ---------------------------------------------------------------------------
// 2. runs
// ---------------------------------------------------------------------------
struct AggParams {
  int64_t T;
  const int32_t *match;
  const int32_t *range_id;  // innermost (or walked) range, input index, or -1
  const uint32_t *op_in;    // op id of each input range
  int64_t R_in;
  uint32_t NOPS, rb;        // rb: operator rows per bucket
  AggIn in;
  PartRow *acc;             // [G] row accumulators for what blocks do not keep (zeroed)
  PartRow *parts;           // [blocks][kABlockCap] kept partials, by bucket (row in pad)
  uint16_t *bkt;            // [blocks][kBuckets] offset << 8 | count
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

template <bool DEF>  // DEF: the default aggregation kinds
__global__ void __launch_bounds__(kAThreads) __attribute__((amdgpu_waves_per_eu(3)))
k_f_agg(AggParams a) {
  __shared__ Slot slots[kAThreads / OPA_WAVE][kASlots];
  __shared__ int nslot[kAThreads / OPA_WAVE];
  __shared__ uint32_t hist[kBuckets], spos[kABlockCap];
  __shared__ uint32_t sh[4];
  const int tid = threadIdx.x, ln = lane_id(), w = wave_id();
  const AggIn &in = a.in;
  const uint32_t mx = DEF ? kDefMaxMask : in.maxmask, dw = DEF ? kDefDwMask : in.dwmask;
  const int64_t ib = (int64_t)blockIdx.x * kASpan + (int64_t)tid * kAPer;
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
#pragma unroll 1
  for (int h = 0; h < 2; ++h) {
    const int64_t i0 = ib + h * kAHalf;
    const int nh = nv - h * kAHalf < 0 ? 0 : (nv - h * kAHalf < kAHalf ? nv - h * kAHalf : kAHalf);
    int32_t mt[kAHalf], rid[kAHalf];
    uint32_t du[kAHalf], g[kAHalf];
    load_n<kAHalf>(a.match, i0, nh, mt);
    load_n<kAHalf>(in.dur, i0, nh, du);
    load_n<kAHalf>(a.range_id, i0, nh, rid);
    // the counter rows of these launches are touched first (two words per
    // row), so that the accumulation below finds them in cache instead of
    // waiting for one row after another
    uint32_t touch = 0;
#pragma unroll
    for (int k = 0; k < kAHalf; ++k)
      if (k < nh && mt[k] >= 0 && (int64_t)mt[k] < in.P) {
        const float *row = in.counters + (int64_t)mt[k] * in.rs;
        touch ^= __float_as_uint(row[0]) ^
                 __float_as_uint(row[(int64_t)(OPATTR_NUM_COUNTERS - 1) * in.cs]);
      }
    if (touch == 0x9E3779B9u && a.T < 0) a.bkt[0] = 0;  // never true: keeps the loads
#pragma unroll
    for (int k = 0; k < kAHalf; ++k) g[k] = k < nh ? row_of(a, rid[k]) : 0xFFFFFFFFu;
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
  for (int q = tid; q < kBuckets; q += kAThreads) hist[q] = 0;
  __syncthreads();

  // the block's kept partials, counted by bucket, then written in bucket
  // order
  uint32_t bq = 0xFFFFFFFFu, rk = 0;
  if (tid < kABlockCap) {
    const int sw = tid / kASlots, sj = tid % kASlots;
    const Slot *q = &slots[sw][sj];
    if (sj < nslot[sw] && q->live) {
      bq = q->g / a.rb;
      rk = atomicAdd(&hist[bq], 1u);
    }
  }
  __syncthreads();
  uint32_t cnt = 0, tot;
  if (tid < kBuckets) cnt = hist[tid];
  const uint32_t off = block_excl_scan_add<uint32_t>(tid < kBuckets ? cnt : 0u, sh, &tot);
  if (tid < kBuckets)
    a.bkt[(int64_t)blockIdx.x * kBuckets + tid] = (uint16_t)((off << 8) | cnt);
  __syncthreads();
  if (tid < kBuckets) hist[tid] = off;
  __syncthreads();
  if (tid < kABlockCap) spos[tid] = bq != 0xFFFFFFFFu ? hist[bq] + rk : 0xFFFFFFFFu;
  __syncthreads();
  // coalesced copy: consecutive threads take consecutive fields
  PartRow *dst = a.parts + (int64_t)blockIdx.x * kABlockCap;
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
// 3. per bucket: the kept partials of a share of the blocks, added in LDS
// ---------------------------------------------------------------------------
struct CombParams {
  int64_t nblocks;
  uint32_t rb;
  const PartRow *parts;
  const uint16_t *bkt;
  PartRow *split;  // [kBuckets][kSplits][rb]
};

// Each lane takes its own blocks (a contiguous share of them per wave) and
// adds their partials of the bucket one after another, so that the loads of
// all lanes are in flight together; rows accumulate in LDS.
template <bool DEF>
__global__ void __launch_bounds__(64) k_f_comb(CombParams a, uint32_t maxmask) {
  extern __shared__ __align__(16) unsigned char comb_raw[];
  unsigned long long *tab = reinterpret_cast<unsigned long long *>(comb_raw);  // [rb][kFFields]
  const uint32_t mx = DEF ? kDefMaxMask : maxmask;
  const int ln = lane_id();
  const uint32_t q = blockIdx.x / kSplits, s = blockIdx.x % kSplits;
  const uint32_t rb = a.rb;
  for (uint32_t x = ln; x < rb * kFFields; x += OPA_WAVE) tab[x] = 0;
  wave_sync_lds();
  const int64_t per = (a.nblocks + kSplits - 1) / kSplits;
  const int64_t b_lo = (int64_t)s * per, b_hi = b_lo + per < a.nblocks ? b_lo + per : a.nblocks;
  for (int64_t b0 = b_lo; b0 < b_hi; b0 += 4 * OPA_WAVE) {
    // this lane's blocks of the round (their bucket entries loaded together)
    uint32_t e[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t b = b0 + j * OPA_WAVE + ln;
      e[j] = b < b_hi ? a.bkt[b * kBuckets + q] : 0u;
    }
#pragma unroll 1
    for (int j = 0; j < 4; ++j) {
      const int64_t b = b0 + j * OPA_WAVE + ln;
      const uint32_t c = e[j] & 0xFFu, o = e[j] >> 8;
      const unsigned long long *pr =
          reinterpret_cast<const unsigned long long *>(a.parts + b * kABlockCap + o);
#pragma unroll 1
      for (uint32_t p = 0; p < c; ++p, pr += sizeof(PartRow) / 8) {
        unsigned long long v[kFFields];
#pragma unroll
        for (int f = 0; f < kFFields; ++f) v[f] = pr[f];
        unsigned long long *t = tab + (size_t)((uint32_t)(v[24] >> 32) % rb) * kFFields;
        atomicAdd(t + 0, v[0]);
        atomicAdd(t + 1, v[1]);
        if (v[2] == 0) continue;  // no matched launch: counter fields are zero
        atomicAdd(t + 2, v[2]);
        atomicAdd(t + 3, v[3]);
#pragma unroll
        for (int c2 = 0; c2 < OPATTR_NUM_COUNTERS; ++c2) {
          if ((mx >> c2) & 1u) atomicMax(t + 4 + c2, v[4 + c2]);
          else unsafeAtomicAdd(reinterpret_cast<double *>(t + 4 + c2), bits2d(v[4 + c2]));
        }
        if ((uint32_t)v[24]) atomicOr(reinterpret_cast<unsigned int *>(t + 24), (uint32_t)v[24]);
      }
    }
  }
  wave_sync_lds();
  unsigned long long *out =
      reinterpret_cast<unsigned long long *>(a.split + ((size_t)q * kSplits + s) * rb);
  for (uint32_t x = ln; x < rb * kFFields; x += OPA_WAVE) {
    const uint32_t r = x / kFFields, ff = x % kFFields;
    out[r * (sizeof(PartRow) / 8) + ff] = tab[x];
  }
}

// ---------------------------------------------------------------------------
// 4. table rows and the summary's block sums (attributed, unattributed,
// total, matched ns)
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_f_rows(const PartRow *__restrict__ acc,
                                                const PartRow *__restrict__ split, uint32_t rb,
                                                uint32_t G, uint32_t NOPS, uint32_t mx,
                                                uint32_t dw, uint32_t absent,
                                                opattr_op_row *table, unsigned long long *part) {
  __shared__ unsigned long long red[4][4];
  unsigned long long at_ = 0, un = 0, tot = 0, mt = 0;
  for (uint32_t g = blockIdx.x * blockDim.x + threadIdx.x; g < G; g += gridDim.x * blockDim.x) {
    Acc x;
    acc_load(x, acc + g);
    const uint32_t q = g / rb, r = g % rb;
#pragma unroll 1
    for (int s = 0; s < kSplits; ++s) {
      Acc y;
      acc_load(y, split + ((size_t)q * kSplits + s) * rb + r);
      acc_merge(x, y, mx);
    }
    opattr_op_row *row = table + g;
    row->kernel_count = x.kc;
    row->total_ns = x.tns;
    row->matched_count = x.mc;
    row->matched_ns = x.mns;
    const double qnan = __longlong_as_double(0x7FF8000000000000ll);
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      double v;
      if (((absent >> c) & 1u) || x.mc == 0) v = qnan;
      else if ((mx >> c) & 1u) v = ((x.nan >> c) & 1u) ? qnan : (double)key2f((uint32_t)x.v[c]);
      else if ((dw >> c) & 1u) v = x.mns ? bits2d(x.v[c]) / (double)x.mns : qnan;
      else v = bits2d(x.v[c]);
      row->value[c] = v;
    }
    tot += x.tns;
    mt += x.mns;
    if (g < NOPS) at_ += x.tns;
    else un += x.tns;
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
  if (threadIdx.x < 4)
    part[blockIdx.x * 4 + threadIdx.x] =
        red[threadIdx.x][0] + red[threadIdx.x][1] + red[threadIdx.x][2] + red[threadIdx.x][3];
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
uint32_t fused_rows_per_bucket(uint32_t G) { return (G + kBuckets - 1) / kBuckets; }

int64_t fused_agg_blocks(int64_t T) { return (T + kASpan - 1) / kASpan; }

size_t fused_parts_bytes(int64_t T) {
  return (size_t)fused_agg_blocks(T) * kABlockCap * sizeof(PartRow);
}

size_t fused_bkt_bytes(int64_t T) { return (size_t)fused_agg_blocks(T) * kBuckets * 2; }

size_t fused_split_bytes(uint32_t G) {
  return (size_t)kBuckets * kSplits * fused_rows_per_bucket(G) * sizeof(PartRow);
}

int fused_sum_blocks(const Plan &pl) {
  const int64_t want = ((int64_t)pl.G + 255) / 256;
  return (int)(want < kSumBlocks ? (want > 0 ? want : 1) : kSumBlocks);
}

void clear_fused_acc(void *ws, const Plan &pl, hipStream_t s) {
  fill_u32(at<uint32_t>(ws, pl.acc), 0u, (int64_t)pl.G * (sizeof(PartRow) / 4), s);
}

void run_fused_match(const FusedIn &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  if (pl.T <= 0) return;
  MatchParams m{};
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
  probe_begin(OPATTR_PROBE_DEDUP, s);
  const int64_t threads = (pl.T + kMPer - 1) / kMPer;
  k_f_match<<<(unsigned)((threads + 255) / 256), 256, 0, s>>>(m);
  probe_end(OPATTR_PROBE_DEDUP, s);
}

void run_fused_agg(const FusedIn &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const uint32_t rb = fused_rows_per_bucket(pl.G);
  AggParams a{};
  a.T = pl.T;
  a.match = x.match;
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
  c.parts = a.parts;
  c.bkt = a.bkt;
  c.split = at<PartRow>(x.ws, pl.fsplit);
  const size_t lds = (size_t)rb * kFFields * 8;
  if (def) k_f_comb<true><<<kBuckets * kSplits, 64, lds, s>>>(c, a.in.maxmask);
  else k_f_comb<false><<<kBuckets * kSplits, 64, lds, s>>>(c, a.in.maxmask);
  k_f_rows<<<fused_sum_blocks(pl), 256, 0, s>>>(a.acc, c.split, rb, pl.G, x.d->n_ops, a.in.maxmask,
                                                 a.in.dwmask, x.absent, x.table,
                                                 at<unsigned long long>(x.ws, pl.sumpart));
  probe_end(OPATTR_PROBE_AGGREGATE, s);
}

}  // namespace opa
