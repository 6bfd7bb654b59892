// Enclosure (Alg. 2) and the first level of the aggregation (Eq. 1), two
// passes over the launches in storage order: the enclosure, which also plans
// the aggregation's items (it needs only the operator row of each launch),
// and the in-place reduction of the runs (which needs the matches).
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
// Plan: a wave with at most kRowCap runs will reduce them in place and emits
// one item (row, partial-row index) per run; a wave with more runs emits
// references (row, first launch, length <= 16) that the per-row reduction
// resolves later. The enclosure pass counts each wave's items and partial
// rows, a scan over the waves turns the counts into bases, and an emission
// pass writes the items in launch order. Reduction: every thread accumulates
// its launches in registers, leaving each run that ends inside it in an LDS
// row, and a segmented scan over the lanes carries the runs that cross
// threads; the rows then go out with coalesced stores at the planned indices.
#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kPer = 8;                         // launches per thread
constexpr int kSpan = kEncThreads * kPer;       // launches per block
constexpr int kRowCap = 32;                     // runs a wave reduces in place

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
  uint8_t *fused;      // optional walk outputs
  int32_t *range_any;
  int32_t *core_id;    // set: the innermost range's core position instead (no kinds)
  const int32_t *wfirst;  // with kinds: each range's walk (first op range, fused)
  const uint8_t *wfused;
  AggIn ag;
  EmitOut em;
  opattr_diag *diag;
  // blocks [nenc, grid) write the range depths instead, 256 ranges a block
  int64_t nenc;
  uint8_t *range_depth;
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

// The operator rows of a thread's launches from input range ids (plan from a
// given range_id array, and the reduction). Counts malformed range ids.
__device__ __forceinline__ uint32_t rows_from_ids(const EncParams &a, int64_t ib, int nv,
                                                  uint32_t (&g)[kPer]) {
  int32_t rin[kPer];
  load_run(a.range_id, ib, nv, rin);
  uint32_t bad = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    g[k] = k < nv ? a.NOPS : 0xFFFFFFFFu;
    if (k >= nv) continue;
    const int32_t r = rin[k];
    if (r >= 0 && r < a.R_in && a.op_in[r] < a.NOPS) g[k] = a.op_in[r];
    else if (r < -1 || r >= a.R_in || r >= 0) bad++;
  }
  return bad;
}

// Piece starts of the references: run starts, and every 16th launch.
__device__ __forceinline__ uint32_t piece_heads(uint32_t hm, int nv) {
  return hm | ((nv > 0 && (lane_id() & 1) == 0) ? 1u : 0u);
}

// Run starts of a thread's launches inside its wave (bit k: launch k starts
// a run; the wave's first launch always does), and the references' piece
// starts (runs cut at every 16th launch as well).
__device__ __forceinline__ void run_heads(const uint32_t (&g)[kPer], int nv, uint32_t &hm,
                                          uint32_t &hp) {
  const int ln = lane_id();
  const uint32_t gl = __shfl_up(g[kPer - 1], 1, OPA_WAVE);
  hm = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const uint32_t prev = k ? g[k - 1] : (ln ? gl : 0xFFFFFFFFu);
    if (k < nv && g[k] != prev) hm |= 1u << k;
  }
  hp = piece_heads(hm, nv);
}

// Items and partial rows of the calling wave (all lanes get them).
__device__ __forceinline__ void wave_counts(uint32_t hm, uint32_t hp, uint32_t &items,
                                            uint32_t &rows) {
  const uint32_t nr = wave_reduce_add((uint32_t)__popc(hm));
  const uint32_t np = wave_reduce_add((uint32_t)__popc(hp));
  const bool rowmode = nr <= (uint32_t)kRowCap;
  items = rowmode ? nr : np;
  rows = rowmode ? nr : 0u;
}

// MODE 1: range ids; MODE 3: range ids and the per-wave item and row counts;
// MODE 2: the counts from a given range_id array.
// six waves per SIMD: the kernel waits on chains of dependent loads, and
// 80 registers (one fewer than it would take) buy a sixth wave without spills
template <int MODE>
__global__ void __launch_bounds__(kEncThreads) __attribute__((amdgpu_waves_per_eu(6)))
k_enclose(EncParams a) {
  __shared__ uint64_t sS[(MODE & 1) ? kEncWindow : 1];
  __shared__ uint64_t red[2][kEncThreads / OPA_WAVE];
  __shared__ int64_t win[2];
  __shared__ uint32_t sbad;
  if ((int64_t)blockIdx.x >= a.nenc) {
    const int64_t x = ((int64_t)blockIdx.x - a.nenc) * kEncThreads + threadIdx.x;
    range_depth_one(a.npg, a.ree, a.cr.st, a.cr.perm, a.cr.n, a.NS, x, a.range_depth, a.diag);
    return;
  }
  const int tid = threadIdx.x, w = wave_id(), ln = lane_id();
  if (tid == 0) sbad = 0;
  if (MODE == 2) __syncthreads();
  const int64_t bid = blockIdx.x;
  const int64_t i0 = bid * kSpan;
  const int64_t ib = i0 + (int64_t)tid * kPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kPer ? a.T - ib : kPer));
  uint32_t bad = 0;
  uint32_t g[kPer];
  if (MODE & 1) {
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

    // Phase 1, the last range starting at or before each query point.
    // Consecutive launches of one stream with non-decreasing query points
    // (the common case) continue from the previous launch: that range only
    // moves forward. Only the staged starts (LDS) are read here when the
    // window holds the stream.
    int32_t pk[kPer], lok[kPer];
    bool have = false;  // the previous launch was searched
    uint16_t sprev = 0;
    uint64_t qprev = 0;
    int32_t pprev = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      pk[k] = -1;
      lok[k] = 0;
      if (k < nv && st[k] < a.NS && q[k] < (1ull << 63)) {
        const int32_t lo = (int32_t)a.rblk[st[k]], hi = (int32_t)a.rblk[st[k] + 1];
        lok[k] = lo;
        const bool win = staged && st[k] == s0;  // the staged starts belong to this stream
        int32_t p;
        if (have && st[k] == sprev && q[k] >= qprev) {
          // forward from the previous launch's range: single steps first
          // (launches close in time), then steps of 2, 4, 8, ... and a
          // bisection of the last one (launches far apart in storage order)
          auto start_of = [&](int64_t j) -> uint64_t {
            const int64_t x = j - wlo;
            return (win && x >= 0 && x < wn) ? sS[x] : a.cr.s[j];
          };
          int64_t lo2 = pprev, hi2 = hi;  // start_of(lo2) <= q (or lo2 = lo - 1)
          int n1 = 0;
          for (; n1 < 4 && lo2 + 1 < hi; ++n1) {
            if (start_of(lo2 + 1) > q[k]) {
              hi2 = lo2 + 1;
              break;
            }
            ++lo2;
          }
          if (n1 == 4) {
            for (int64_t stp = 2; lo2 + stp < hi; stp <<= 1) {
              if (start_of(lo2 + stp) > q[k]) {
                hi2 = lo2 + stp;
                break;
              }
              lo2 += stp;
            }
            while (hi2 - lo2 > 1) {  // every start in [hi2, hi) is past q
              const int64_t mid = lo2 + ((hi2 - lo2) >> 1);
              if (start_of(mid) <= q[k]) lo2 = mid;
              else hi2 = mid;
            }
          }
          p = (int32_t)lo2;
        } else if (st[k] == s0 && wn == 0) {
          p = lo - 1;  // no range of the stream starts at or before the block's queries
        } else if (win) {
          int l2 = 0, h2 = (int)wn;
          while (l2 < h2) {
            const int mid = (l2 + h2) >> 1;
            if (sS[mid] <= q[k]) l2 = mid + 1;
            else h2 = mid;
          }
          p = (int32_t)(wlo + l2 - 1);
          if (p < lo) p = lo - 1;
        } else {
          p = (int32_t)thread_upper_bound(a.cr.s, lo, hi, q[k]) - 1;
        }
        pk[k] = p;
        pprev = p;
        have = true;
        sprev = st[k];
        qprev = q[k];
      } else {
        if (k < nv && st[k] >= a.NS) bad++;
        have = false;
      }
    }
    // Phase 2, the walk up the parent chain while the range ends before the
    // query point, all of the thread's launches in lock step so that their
    // loads (ends, then parents) are in flight together.
    // a launch whose range is the previous launch's takes its end instead of
    // loading it again (a load whose 64 lanes hit 64 lines costs 64 L1
    // requests; consecutive launches mostly share their range)
    // (the previous launch's end was loaded: its range is valid for its own
    // stream, which an index just before a stream's ranges is not)
    int64_t ek[kPer];
    bool same[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      same[k] = k > 0 && pk[k] == pk[k - 1] && pk[k - 1] >= lok[k - 1];
      ek[k] = (pk[k] >= lok[k] && !same[k]) ? a.ree[pk[k]] : 0;
    }
#pragma unroll
    for (int k = 1; k < kPer; ++k)
      if (pk[k] >= lok[k] && same[k]) ek[k] = ek[k - 1];
    for (int step = 0; step < kMaxWalk; ++step) {
      bool act[kPer], any = false;
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        act[k] = pk[k] >= lok[k] && ek[k] < (int64_t)q[k];
        any |= act[k];
      }
      if (!any) break;
#pragma unroll
      for (int k = 0; k < kPer; ++k)
        if (act[k]) pk[k] = a.npg[pk[k]];
#pragma unroll
      for (int k = 0; k < kPer; ++k)
        if (act[k] && pk[k] >= lok[k]) ek[k] = a.ree[pk[k]];
    }
    int32_t ridk[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k)
      ridk[k] = (pk[k] >= lok[k] && ek[k] >= (int64_t)q[k]) ? pk[k] : -1;

    int32_t rout[kPer];
    if (a.core_id) {
      store_run(a.core_id, ib, nv, ridk);
    } else if (!a.cr.kind && !a.fused) {
      // Phase 3 without kinds: the innermost range is the op range; its row
      // and output id for every launch, loads in flight together
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int32_t rid = ridk[k];
        g[k] = k < nv ? (rid >= 0 ? a.cr.op[rid] : a.NOPS) : 0xFFFFFFFFu;
        rout[k] = rid >= 0 ? (a.cr.perm ? a.cr.perm[rid] : rid) : -1;
      }
      if (a.range_any)
#pragma unroll
        for (int k = 0; k < kPer; ++k)
          if (k < nv) a.range_any[ib + k] = rout[k];
      store_run(a.range_id, ib, nv, rout);
    } else {
      // Phase 3 with kinds or fused wanted: Alg. 2's walk outward from the
      // innermost range, once per change of (innermost range, touching)
      int32_t rlast = -1, olast = -1, alast = -1;
      uint32_t glast = 0;
      uint8_t flast = 0;
      bool tlast = false;
      int32_t aout[kPer];
      uint8_t fout[kPer];
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int32_t rid = ridk[k];
        const int64_t slo = lok[k];  // first range of the launch's stream
        // A range that starts at the query point may be preceded, among the
        // ranges containing the point, by ranges that end there without
        // containing it (touching, not nested); any other enclosing range is
        // an ancestor. So the walk depends on the query point only through
        // "the innermost range starts at it", which keys the cache with rid.
        bool touch = false;
        if (rid >= 0 && (a.cr.kind || a.fused)) {
          const int64_t x = rid - wlo;
          const uint64_t sr = (staged && st[k] == s0 && x >= 0 && x < wn) ? sS[x] : a.cr.s[rid];
          touch = sr == q[k];
        }
        if (rid >= 0 && (rid != rlast || touch != tlast)) {
          rlast = rid;
          tlast = touch;
          // the next range outward that contains the query point: the parent,
          // or from a range starting at the point the nearest earlier range in
          // nesting order that ends at or after it
          auto next_out = [&](int64_t j) -> int64_t {
            if (!touch || (uint64_t)a.cr.s[j] != q[k]) return a.npg[j];
            int64_t c = j - 1;
            for (int h = 0; c >= slo && a.ree[c] < (int64_t)q[k] && h < kMaxWalk; ++h) c = a.npg[c];
            return c >= slo ? c : -1;
          };
          // Alg. 2's walk outward from the innermost range: ops collected,
          // skipped kinds passed over, a boundary ends it
          int32_t first = rid;
          flast = 0;
          if (a.cr.kind && !touch) {
            first = a.wfirst[rid];  // the walk from rid, done once per range
            flast = a.wfused[rid];
          } else if (a.cr.kind) {
            first = -1;
            int nops = 0, hops = 0;
            for (int64_t j = rid; j >= 0 && hops < kMaxWalk; j = next_out(j), ++hops) {
              const uint8_t kd = a.cr.kind[j];
              if (kd == OPATTR_KIND_BOUNDARY) break;
              if (kd != OPATTR_KIND_OP) continue;
              if (first < 0) first = (int32_t)j;
              ++nops;
            }
            flast = nops > 1 ? 1 : 0;
          } else if (a.fused) {
            flast = next_out(rid) >= 0 ? 1 : 0;  // every enclosing range is an op
          }
          olast = first >= 0 ? (a.cr.perm ? a.cr.perm[first] : first) : -1;
          glast = first >= 0 ? a.cr.op[first] : a.NOPS;
          alast = a.cr.perm ? a.cr.perm[rid] : rid;
        }
        rout[k] = rid >= 0 ? olast : -1;
        g[k] = k < nv ? (rid >= 0 ? glast : a.NOPS) : 0xFFFFFFFFu;
        aout[k] = rid >= 0 ? alast : -1;
        fout[k] = rid >= 0 ? flast : 0;
      }
      // stored after the walks, so that no store sits between the loads of
      // consecutive launches
      store_run(a.range_id, ib, nv, rout);
      if (a.range_any) store_run(a.range_any, ib, nv, aout);
      if (a.fused)
#pragma unroll
        for (int k = 0; k < kPer; ++k)
          if (k < nv) a.fused[ib + k] = fout[k];
    }
  } else {
    bad += rows_from_ids(a, ib, nv, g);
  }
  if (MODE & 2) {
    uint32_t hm, hp, items, rows;
    run_heads(g, nv, hm, hp);
    wave_counts(hm, hp, items, rows);
    a.em.hmb[bid * kEncThreads + tid] = (uint8_t)hm;
    if (ln == 0) {
      a.em.wi[bid * (kEncThreads / OPA_WAVE) + w] = items;
      a.em.wr[bid * (kEncThreads / OPA_WAVE) + w] = rows;
    }
  }
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (tid == 0 && sbad)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)sbad);
}

// Exclusive scans of the per-wave item and row counts, in place (one block);
// meta[0] / meta[1] get the totals. Each thread takes a contiguous run of
// enclosure blocks (four waves each, one 16-byte load per array) and loads
// them four blocks at a time, so the loads of a batch are in flight
// together.
__global__ void __launch_bounds__(1024) k_wave_scan(EmitOut e, int64_t nblocks) {
  constexpr int kW = kEncThreads / OPA_WAVE;
  static_assert(kW == 4, "one 16-byte load per block");
  constexpr int kBatch = 4;
  __shared__ uint32_t sh[16];
  const uint4 *wi4 = reinterpret_cast<const uint4 *>(e.wi);
  const uint4 *wr4 = reinterpret_cast<const uint4 *>(e.wr);
  const int64_t ch = (nblocks + blockDim.x - 1) / blockDim.x;
  const int64_t lo = (int64_t)threadIdx.x * ch;
  const int64_t hi = lo + ch < nblocks ? lo + ch : nblocks;
  uint32_t si = 0, sr = 0;
  for (int64_t b0 = lo; b0 < hi; b0 += kBatch) {
    uint4 vi[kBatch], vr[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      vi[j] = b0 + j < hi ? wi4[b0 + j] : make_uint4(0, 0, 0, 0);
      vr[j] = b0 + j < hi ? wr4[b0 + j] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      si += vi[j].x + vi[j].y + vi[j].z + vi[j].w;
      sr += vr[j].x + vr[j].y + vr[j].z + vr[j].w;
    }
  }
  uint32_t ti, tr;
  uint32_t ri = block_excl_scan_add<uint32_t>(si, sh, &ti);
  uint32_t rr = block_excl_scan_add<uint32_t>(sr, sh, &tr);
  uint4 *oi = reinterpret_cast<uint4 *>(e.wi);
  uint4 *orr = reinterpret_cast<uint4 *>(e.wr);
  for (int64_t b0 = lo; b0 < hi; b0 += kBatch) {
    uint4 vi[kBatch], vr[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      vi[j] = b0 + j < hi ? wi4[b0 + j] : make_uint4(0, 0, 0, 0);
      vr[j] = b0 + j < hi ? wr4[b0 + j] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (b0 + j >= hi) break;
      uint4 bi, br;
      bi.x = ri;
      bi.y = bi.x + vi[j].x;
      bi.z = bi.y + vi[j].y;
      bi.w = bi.z + vi[j].z;
      ri = bi.w + vi[j].w;
      br.x = rr;
      br.y = br.x + vr[j].x;
      br.z = br.y + vr[j].y;
      br.w = br.z + vr[j].z;
      rr = br.w + vr[j].w;
      oi[b0 + j] = bi;
      orr[b0 + j] = br;
    }
  }
  if (threadIdx.x == 0) {
    e.meta[0] = ti;
    e.meta[1] = tr;
  }
}

// Items of every wave at its scanned bases, in launch order.
__global__ void __launch_bounds__(kEncThreads) k_emit(EncParams a) {
  const int w = wave_id(), ln = lane_id();
  const int64_t wave = (int64_t)blockIdx.x * (kEncThreads / OPA_WAVE) + w;
  const int64_t ib = (int64_t)blockIdx.x * kSpan + (int64_t)threadIdx.x * kPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kPer ? a.T - ib : kPer));
  const uint32_t hm = a.em.hmb[(int64_t)blockIdx.x * kEncThreads + threadIdx.x];
  const uint32_t hp = piece_heads(hm, nv);
  const uint32_t nh = __popc(hm), nhp = __popc(hp);
  const uint32_t hb = wave_incl_scan_add(nh) - nh;
  const uint32_t hpb = wave_incl_scan_add(nhp) - nhp;
  const uint32_t nr_w = __shfl(hb + nh, OPA_WAVE - 1, OPA_WAVE);
  const uint32_t ibase = a.em.wi[wave];
  // the operator rows of the thread's run and piece starts (hp holds hm),
  // all loaded before any item is stored
  int32_t rin[kPer];
  load_run(a.range_id, ib, nv, rin);
  uint32_t gk[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int32_t r = rin[k];
    const bool head = k < nv && ((hp >> k) & 1u);
    gk[k] = (head && r >= 0 && r < a.R_in) ? a.op_in[r] : a.NOPS;
    if (gk[k] >= a.NOPS) gk[k] = a.NOPS;
  }
  if (nr_w <= (uint32_t)kRowCap) {
    // one item per run, written by the launch that starts it
    const uint32_t rbase = a.em.wr[wave];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (!((hm >> k) & 1u)) continue;
      const uint32_t idx = hb + __popc(hm & ((1u << k) - 1u));
      a.em.ig[ibase + idx] = gk[k];
      a.em.ia[ibase + idx] = rbase + idx;
      a.em.ib[ibase + idx] = 0;
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
      a.em.ig[ibase + idx] = gk[k];
      a.em.ia[ibase + idx] = (uint32_t)(ib + k);
      a.em.ib[ibase + idx] = len;
    }
  }
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

// In-place reduction of the planned runs (waves in row mode); the matches of
// every launch are checked here.
template <bool DEF>  // DEF: the default aggregation kinds
__global__ void __launch_bounds__(kEncThreads) __attribute__((amdgpu_waves_per_eu(4)))
k_agg_rows(EncParams a) {
  __shared__ PartRow stage[kEncThreads / OPA_WAVE][kRowCap];
  __shared__ uint32_t sbad;
  const int tid = threadIdx.x, w = wave_id(), ln = lane_id();
  const AggIn &in = a.ag;
  const uint32_t mx = DEF ? kDefMaxMask : in.maxmask, dw = DEF ? kDefDwMask : in.dwmask;
  if (tid == 0) sbad = 0;
  __syncthreads();
  const int64_t bid = blockIdx.x;
  const int64_t ib = bid * kSpan + (int64_t)tid * kPer;
  const int nv = (int)(a.T - ib < 0 ? 0 : (a.T - ib < kPer ? a.T - ib : kPer));
  const uint32_t hm = a.em.hmb[bid * kEncThreads + tid];
  uint32_t mt[kPer];  // profiled row indices (as stored, -1 = unmatched)
  uint32_t du[kPer];
  load_run(reinterpret_cast<const uint32_t *>(in.match), ib, nv, mt);
  load_run(in.dur, ib, nv, du);
  uint32_t bad = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k)
    if (k < nv && ((int32_t)mt[k] < -1 || (int64_t)(int32_t)mt[k] >= in.P))
      bad++;  // aggregates as unmatched
  const uint32_t nh = __popc(hm);
  const uint32_t hb = wave_incl_scan_add(nh) - nh;
  const uint32_t nr_w = __shfl(hb + nh, OPA_WAVE - 1, OPA_WAVE);
  if (nr_w <= (uint32_t)kRowCap) {
    // Each thread accumulates its launches; a run that ends inside the thread
    // goes to its LDS row (the first one of them still lacks the part from
    // earlier threads, added after the scan). The thread's last run is
    // scanned across the lanes.
    PartRow *wst = stage[w];
    Acc inc;
    acc_zero(inc);
    // launch k is always at position 0 of mt / du: the arrays shift by one
    // per step (a run-time index would move them to scratch memory)
#pragma unroll 1
    for (int k = 0; k < nv; ++k) {
      if (k > 0 && ((hm >> k) & 1u)) {
        acc_store(wst + hb + __popc(hm & ((1u << k) - 1u)) - 1u, inc);
        acc_zero(inc);
      }
      acc_launch(inc, in, (int32_t)mt[0], du[0], mx, dw);
#pragma unroll
      for (int j = 0; j + 1 < kPer; ++j) {
        mt[j] = mt[j + 1];
        du[j] = du[j + 1];
      }
    }
    const unsigned long long hl = __ballot(hm != 0) | 1ull;
    const unsigned long long upto = ln == 63 ? ~0ull : ((2ull << ln) - 1);
    const int sl = 63 - __clzll(hl & upto);
    acc_seg_scan(inc, sl, mx);
    // the lane's last run: ends here, or continues into the next lane and
    // (if it ends inside that lane) completes the row that lane left
    const uint32_t nvn = __shfl_down((uint32_t)nv, 1, OPA_WAVE);
    const uint32_t hmn = __shfl_down(hm, 1, OPA_WAVE);
    if (nv > 0) {
      PartRow *r = wst + hb + nh - 1u;
      if (ln == OPA_WAVE - 1 || nvn == 0 || (hmn & 1u)) acc_store(r, inc);
      else if (hmn & 0xFEu) row_add(r, inc, mx);
    }
    // coalesced copy of the wave's rows to the planned indices
    const uint32_t rbase = a.em.wr[bid * (kEncThreads / OPA_WAVE) + w];
    const unsigned long long *src = reinterpret_cast<const unsigned long long *>(wst);
    unsigned long long *dst = reinterpret_cast<unsigned long long *>(a.em.rows + rbase);
    const uint32_t nw = nr_w * (uint32_t)(sizeof(PartRow) / 8);
    for (uint32_t x = ln; x < nw; x += OPA_WAVE) dst[x] = src[x];
  }
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (tid == 0 && sbad)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)sbad);
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
  a.fused = x.fused;
  a.range_any = x.range_any;
  a.diag = x.diag;
  a.cr = x.cr;
  a.rblk = at<int64_t>(x.ws, pl.rblk);
  a.ree = at<int64_t>(x.ws, pl.ree);
  a.npg = at<int32_t>(x.ws, pl.npg);
  // the aggregation reads range ids by input range index
  a.R_in = x.r ? x.r->n : 0;
  a.op_in = x.r ? x.r->op_id : nullptr;
  a.em = emit_out(x.ws, pl);
  a.wfirst = at<int32_t>(x.ws, pl.wfirst);
  a.wfused = at<uint8_t>(x.ws, pl.wfused);
  a.nenc = pl.nencb;
  return a;
}

// per-wave item and row counts (with the enclosure when enclose is set) and
// their scan: all the run reduction needs besides the matches
void plan_counts(const EncArgs &x, bool enclose, hipStream_t s) {
  const Plan &pl = *x.pl;
  const EncParams a = enc_params(x);
  FillJobs clr;
  clr.add(at<uint32_t>(x.ws, pl.gcnt), 0, pl.G);
  if (pl.T <= 0) clr.add(a.em.meta, 0, 8);
  fill_many(clr, s);
  probe_begin(OPATTR_PROBE_MAIN_PASS, s);
  if (pl.T > 0) {
    if (enclose) k_enclose<3><<<(unsigned)pl.nencb, kEncThreads, 0, s>>>(a);
    else k_enclose<2><<<(unsigned)pl.nencb, kEncThreads, 0, s>>>(a);
  }
  probe_end(OPATTR_PROBE_MAIN_PASS, s);
  if (pl.T > 0) k_wave_scan<<<1, 1024, 0, s>>>(a.em, pl.nencb);
}

// the items and their sort by operator row
void plan_emit(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const EncParams a = enc_params(x);
  if (pl.T > 0) k_emit<<<(unsigned)pl.nencb, kEncThreads, 0, s>>>(a);
  plan_items(x, s);
}

void launch_innermost(const CoreRanges &cr, const opattr_kernels *k, const opattr_dims *d,
                      void *ws, const Plan &pl, int32_t *core, opattr_diag *diag, hipStream_t s) {
  EncParams a{};
  a.T = pl.T;
  a.q = k->query_ns ? k->query_ns : k->start_ns;
  a.stream = k->stream_id;
  a.NS = d->n_streams;
  a.NOPS = d->n_ops;
  a.cr = cr;
  a.cr.kind = nullptr;  // the innermost range whatever its kind
  a.rblk = at<int64_t>(ws, pl.rblk);
  a.ree = at<int64_t>(ws, pl.ree);
  a.npg = at<int32_t>(ws, pl.npg);
  a.core_id = core;
  a.diag = diag;
  a.nenc = pl.nencb;
  if (pl.T > 0) k_enclose<1><<<(unsigned)pl.nencb, kEncThreads, 0, s>>>(a);
}

void run_enclose(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  EncParams a = enc_params(x);
  a.nenc = pl.T > 0 ? pl.nencb : 0;
  // the range depths (deferred by resolve_ranges) in blocks of their own
  const int64_t nd = x.depth && pl.R > 0 && x.d->n_streams > 0 ? (pl.R + kEncThreads - 1) / kEncThreads : 0;
  a.range_depth = x.range_depth;
  probe_begin(OPATTR_PROBE_MAIN_PASS, s);
  if (a.nenc + nd > 0) k_enclose<1><<<(unsigned)(a.nenc + nd), kEncThreads, 0, s>>>(a);
  probe_end(OPATTR_PROBE_MAIN_PASS, s);
}

void reduce_runs(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  EncParams a = enc_params(x);
  a.ag = agg_inputs(x);
  probe_begin(OPATTR_PROBE_AGG_RUNS, s);
  if (pl.T > 0) {
    const unsigned nb = (unsigned)pl.nencb;
    if (a.ag.maxmask == kDefMaxMask && a.ag.dwmask == kDefDwMask)
      k_agg_rows<true><<<nb, kEncThreads, 0, s>>>(a);
    else
      k_agg_rows<false><<<nb, kEncThreads, 0, s>>>(a);
  }
  probe_end(OPATTR_PROBE_AGG_RUNS, s);
}

void run_aggregate_all(const EncArgs &x, hipStream_t s) {
  plan_counts(x, false, s);
  plan_emit(x, s);
  reduce_runs(x, s);
  reduce_items(x, s);
}

}  // namespace opa
