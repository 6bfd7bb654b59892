// Per-operator aggregation (Eq. 1, Sec. 3.8.1), second and third levels.
//
// The enclosure pass plans, in launch order, items of one operator row each:
// either a partial row (a run reduced in place once the matches are known)
// or a reference to at most 16 launches. Here the items are
//   1. counting-sorted by row (per-tile row histograms scanned down the
//      columns; stable, so each row keeps its items in launch order); this
//      needs only the rows, so it runs beside the matching,
//   2. reduced in windows of 64 consecutive sorted items, one wave each: a
//      lane loads a partial row or accumulates its referenced launches, then
//      a segmented scan over the lanes by row; a row whose items all lie in
//      the window is finalised there (duration-weighted means divided by the
//      matched duration, NaN for absent counters and rows without matched
//      launches), a row crossing the window's edge leaves a partial for it,
//   3. rows without items, and rows spread over several windows, finalised in
//      a second pass: one wave per spread row, or, for a row spread over
//      many windows (one operator holding most of the launches, e.g. the
//      UNATTRIBUTED row of a workload that is mostly not enclosed), chunks
//      of 256 window partials reduced by a block each and then merged in
//      order by one wave.
// The summary over the table is taken by the finishing kernel. Every sum is
// taken in a fixed order, so results are reproducible.
#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kWinItems = 64;     // sorted items per window (one wave)

// A sorted item in 64 bits: partial-row index or first launch (31 bits, <
// 2^31), reference length (5 bits, 0 for a partial row, else <= 16), and
// its operator row (20 bits, < 2^20).
static_assert(kMaxOps + 1 < (1u << 20), "operator rows fit the item's 20 row bits");
__device__ __forceinline__ unsigned long long item_pack(uint32_t a, uint32_t b, uint32_t g) {
  return (unsigned long long)a | ((unsigned long long)b << 31) | ((unsigned long long)g << 36);
}
constexpr uint32_t kHeavy = 256;  // partials above which a row is reduced in chunks
constexpr int kChunk = 256;       // partials per chunk of a heavy row (one per thread)

EmitOut emit_out(void *ws, const Plan &pl) {
  EmitOut e;
  e.wi = at<uint32_t>(ws, pl.wi);
  e.wr = at<uint32_t>(ws, pl.wr);
  e.hmb = at<uint8_t>(ws, pl.hmb);
  e.ig = at<uint32_t>(ws, pl.ig);
  e.ia = at<uint32_t>(ws, pl.ia);
  e.ib = at<uint32_t>(ws, pl.ib);
  e.rows = at<PartRow>(ws, pl.rows);
  e.meta = at<int64_t>(ws, pl.meta);
  return e;
}

AggIn agg_inputs(const EncArgs &x) {
  AggIn in{};
  in.dur = x.k->dur_ns;
  in.match = x.match;
  in.P = x.p->n;
  in.counters = x.p->counters;
  in.rs = x.p->row_stride;
  in.cs = x.p->col_stride;
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    if (x.agg_kind[c] == OPATTR_AGG_DWMEAN) in.dwmask |= 1u << c;
    else if (x.agg_kind[c] == OPATTR_AGG_MAX) in.maxmask |= 1u << c;
  }
  in.vec4 = in.cs == 1 && (in.rs % 4) == 0 &&
            (reinterpret_cast<uintptr_t>(in.counters) & 15) == 0;
  return in;
}

struct AggWork {
  uint32_t G, NOPS, absent;
  int64_t tcap;  // item tiles of 4096 the histogram table holds
  AggIn in;
  const uint32_t *ig, *ia, *ib;
  const PartRow *rows;
  // [0] items, [1] partial rows, [2] item tiles, [3] heavy-row chunks,
  // [4] listed spread rows, [5] heavy rows
  int64_t *meta;
  uint32_t *ith, *gcnt, *goff;
  uint32_t *multi;          // spread rows, when found by row
  uint32_t *heavy;          // rows over more than kHeavy windows: (row, first chunk) pairs
  unsigned long long *hch;  // chunk slots of the heavy rows: row << 32 | chunk
  PartRow *hpart;           // one partial per chunk slot
  int64_t hcap;             // chunk slots available
  unsigned long long *sit;  // sorted items (item_pack)
  PartRow *part;            // [windows][2]: a continuing row's partial per window
  opattr_op_row *table;
  opattr_summary *sum;
  opattr_diag *diag;
};

// Item tiles hold 1024 items (4 per thread) when the items fit the
// histogram table that way, else 4096 (16 per thread): small tiles give
// more blocks for the usual item counts, and the table is sized for the
// worst case (one item per launch) in 4096-item tiles.
template <int PER>
__device__ __forceinline__ int64_t item_x(int64_t tile, int c) {
  constexpr int kTile = 256 * PER;
  return tile * kTile + wave_id() * (kTile / 4) + c * OPA_WAVE + lane_id();
}

__device__ __forceinline__ bool small_item_tiles(const AggWork &w, int64_t n) {
  return n <= w.tcap * 1024;
}

// 1a. per-tile row histograms of the items (tiles in launch order)
template <int PER>
__device__ inline void item_hist(const AggWork &w, int64_t n, uint16_t *cnt) {
  constexpr int kTile = 256 * PER;
  const int64_t ntiles = (n + kTile - 1) / kTile;
  if (blockIdx.x == 0 && threadIdx.x == 0) w.meta[2] = ntiles;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < 4 * w.G; i += 256) cnt[i] = 0;
    __syncthreads();
    uint32_t key[PER], rank[PER];
#pragma unroll
    for (int c = 0; c < PER; ++c) {
      const int64_t x = item_x<PER>(tile, c);
      key[c] = x < n ? w.ig[x] : w.G;
    }
    wave_rank<PER>(key, w.G, bits_for(w.G), cnt + wave_id() * w.G, rank);
    block_rank_bases(cnt, w.G, w.ith + tile * w.G);
  }
}

__global__ void __launch_bounds__(256) k_item_hist_w(AggWork w) {
  extern __shared__ __align__(16) unsigned char raw[];
  uint16_t *cnt = reinterpret_cast<uint16_t *>(raw);
  const int64_t n = w.meta[0];
  if (small_item_tiles(w, n)) item_hist<4>(w, n, cnt);
  else item_hist<16>(w, n, cnt);
}

// 1b. row offsets of the sorted items (one block; each thread scans a
// contiguous run of rows)
__global__ void __launch_bounds__(1024) k_row_offsets(AggWork w) {
  __shared__ uint32_t sh[16];
  const uint32_t ch = (w.G + blockDim.x - 1) / blockDim.x;
  const uint32_t lo = threadIdx.x * ch;
  const uint32_t hi = lo + ch < w.G ? lo + ch : w.G;
  uint32_t c = 0;
  for (uint32_t g = lo; g < hi; ++g) c += w.gcnt[g];
  uint32_t tot;
  uint32_t run = block_excl_scan_add<uint32_t>(c, sh, &tot);
  for (uint32_t g = lo; g < hi; ++g) {
    w.goff[g] = run;
    run += w.gcnt[g];
  }
  if (threadIdx.x == 0) {
    w.goff[w.G] = tot;
    w.meta[3] = 0;
    w.meta[4] = 0;
    w.meta[5] = 0;
  }
}

// 1c. stable scatter of the items into row order
template <int PER>
__device__ inline void item_scatter(const AggWork &w, int64_t n, uint16_t *cnt) {
  constexpr int kTile = 256 * PER;
  const int64_t ntiles = (n + kTile - 1) / kTile;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < 4 * w.G; i += 256) cnt[i] = 0;
    __syncthreads();
    uint32_t key[PER], rank[PER];
#pragma unroll
    for (int c = 0; c < PER; ++c) {
      const int64_t x = item_x<PER>(tile, c);
      key[c] = x < n ? w.ig[x] : w.G;
    }
    wave_rank<PER>(key, w.G, bits_for(w.G), cnt + wave_id() * w.G, rank);
    block_rank_bases(cnt, w.G, nullptr);
    const uint32_t *row = w.ith + tile * w.G;
    const uint16_t *wb = cnt + wave_id() * w.G;
#pragma unroll
    for (int c = 0; c < PER; ++c) {
      const uint32_t g = key[c];
      if (g >= w.G) continue;
      const int64_t x = item_x<PER>(tile, c);
      w.sit[w.goff[g] + row[g] + wb[g] + rank[c]] = item_pack(w.ia[x], w.ib[x], g);
    }
  }
}

__global__ void __launch_bounds__(256) k_item_scatter_w(AggWork w) {
  extern __shared__ __align__(16) unsigned char raw[];
  uint16_t *cnt = reinterpret_cast<uint16_t *>(raw);
  const int64_t n = w.meta[0];
  if (small_item_tiles(w, n)) item_scatter<4>(w, n, cnt);
  else item_scatter<16>(w, n, cnt);
}

// 1'. many rows: one stable radix sort of (row, item) over the items (the
// sort reads the item count on the device)
__global__ void k_item_keys(AggWork w, uint32_t *k0, uint32_t *v0, int64_t cap) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= cap || x >= w.meta[0]) return;
  k0[x] = w.ig[x];
  v0[x] = (uint32_t)x;
}

// sorted items in place
__global__ void k_item_place(AggWork w, const uint32_t *key, const uint32_t *val,
                             int64_t cap) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= cap || p >= w.meta[0]) return;
  const uint32_t x = val[p];
  w.sit[p] = item_pack(w.ia[x], w.ib[x], (uint32_t)key[p]);
}

// row offsets: goff[g] = the first sorted item of row g or later (the
// item count for g = G)
__global__ void k_row_bounds(AggWork w, const uint32_t *key, int64_t cap) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g > (int64_t)w.G) return;
  const int64_t n = w.meta[0] < cap ? w.meta[0] : cap;
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if ((int64_t)key[mid] < g) lo = mid + 1;
    else hi = mid;
  }
  w.goff[g] = (uint32_t)lo;
  if (g == 0) {
    w.meta[3] = 0;
    w.meta[4] = 0;
    w.meta[5] = 0;
  }
}

// the row's table entry from its combined partial (lane c writes counter c)
__device__ __forceinline__ void write_row(const AggWork &w, uint32_t g, const Acc &acc,
                                          uint32_t mx, uint32_t dw) {
  const int ln = lane_id();
  opattr_op_row *row = w.table + g;
  if (ln == 0) {
    row->kernel_count = acc.kc;
    row->total_ns = acc.tns;
    row->matched_count = acc.mc;
    row->matched_ns = acc.mns;
  }
  if (ln < OPATTR_NUM_COUNTERS) {
    const int c = ln;
    unsigned long long mine = 0;
#pragma unroll
    for (int k = 0; k < OPATTR_NUM_COUNTERS; ++k)
      if (k == c) mine = acc.v[k];
    const double qnan = __longlong_as_double(0x7FF8000000000000ll);
    double v;
    if (((w.absent >> c) & 1u) || acc.mc == 0) v = qnan;
    else if ((mx >> c) & 1u)
      v = ((acc.nan >> c) & 1u) ? qnan : (double)key2f((uint32_t)mine);
    else if ((dw >> c) & 1u) v = acc.mns ? bits2d(mine) / (double)acc.mns : qnan;
    else v = bits2d(mine);
    row->value[c] = v;
  }
}

// the row's table entry from one lane's accumulator
__device__ __forceinline__ void write_row_lane(const AggWork &w, uint32_t g, const Acc &acc,
                                               uint32_t mx, uint32_t dw) {
  opattr_op_row *row = w.table + g;
  row->kernel_count = acc.kc;
  row->total_ns = acc.tns;
  row->matched_count = acc.mc;
  row->matched_ns = acc.mns;
  const double qnan = __longlong_as_double(0x7FF8000000000000ll);
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    double v;
    if (((w.absent >> c) & 1u) || acc.mc == 0) v = qnan;
    else if ((mx >> c) & 1u) v = ((acc.nan >> c) & 1u) ? qnan : (double)key2f((uint32_t)acc.v[c]);
    else if ((dw >> c) & 1u) v = acc.mns ? bits2d(acc.v[c]) / (double)acc.mns : qnan;
    else v = bits2d(acc.v[c]);
    row->value[c] = v;
  }
}

// 2. one wave per window of 64 sorted items
template <bool DEF>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
k_window_reduce(AggWork w) {
  constexpr int kPiece = 16;  // launches of a reference (at most)
  // the matches and durations of the window's references, staged per wave
  __shared__ int32_t s_m[4][kWinItems * kPiece];
  __shared__ uint32_t s_d[4][kWinItems * kPiece];
  const uint32_t mx = DEF ? kDefMaxMask : w.in.maxmask, dw = DEF ? kDefDwMask : w.in.dwmask;
  const int64_t n = w.meta[0];
  const int64_t nwin = (n + kWinItems - 1) / kWinItems;
  const int ln = lane_id();
  int32_t *lm = s_m[wave_id()];
  uint32_t *ld = s_d[wave_id()];
  for (int64_t win = (int64_t)blockIdx.x * 4 + wave_id(); win < nwin;
       win += (int64_t)gridDim.x * 4) {
    const int64_t p = win * kWinItems + ln;
    uint32_t g = 0xFFFFFFFFu, a = 0, b = 0;
    if (p < n) {
      const unsigned long long it = w.sit[p];
      a = (uint32_t)(it & 0x7FFFFFFFu);
      b = (uint32_t)(it >> 31) & 31u;
      g = (uint32_t)(it >> 36);
    }
    // A reference's launches are consecutive: the wave stages them four
    // references at a time, sixteen lanes each, so that its loads of
    // matches and durations are contiguous rather than one line per lane.
    const uint32_t bs = b <= (uint32_t)kPiece ? b : (uint32_t)kPiece;  // staged launches
    const uint32_t incl = wave_incl_scan_add(bs), pre = incl - bs;
    if (__shfl(incl, OPA_WAVE - 1, OPA_WAVE) > 0) {
#pragma unroll 2
      for (int r = 0; r < kWinItems / 4; ++r) {
        const int j = 4 * r + (ln >> 4), k = ln & 15;
        const uint32_t aj = __shfl(a, j, OPA_WAVE), bj = __shfl(bs, j, OPA_WAVE);
        const uint32_t pj = __shfl(pre, j, OPA_WAVE);
        if ((uint32_t)k < bj) {
          lm[pj + k] = w.in.match[aj + k];
          ld[pj + k] = w.in.dur[aj + k];
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    Acc acc;
    acc_zero(acc);
    if (p < n) {
      if (b == 0) {
        acc_load(acc, w.rows + a);
      } else {
        for (uint32_t k = 0; k < b; ++k) {
          const bool st = k < bs;  // always, for references of at most kPiece launches
          acc_launch(acc, w.in, st ? lm[pre + k] : w.in.match[a + k],
                     st ? ld[pre + k] : w.in.dur[a + k], mx, dw);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();  // the staged entries are read before the next window's
    // segmented scan by row (rows are contiguous in the window)
    const uint32_t gp = __shfl_up(g, 1, OPA_WAVE), gn = __shfl_down(g, 1, OPA_WAVE);
    const uint64_t heads = __ballot(ln == 0 || gp != g);
    const uint64_t upto = ln == OPA_WAVE - 1 ? heads : heads & ((2ull << ln) - 1);
    const int sl = 63 - __clzll((long long)upto);
    acc_seg_scan(acc, sl, mx);
    const bool tail = ln == OPA_WAVE - 1 || gn != g;
    if (tail && g != 0xFFFFFFFFu) {
      const uint32_t lo = w.goff[g], hi = w.goff[g + 1];
      const int64_t wlo = win * kWinItems, whi = wlo + kWinItems;
      if ((int64_t)lo >= wlo && (int64_t)hi <= whi) write_row_lane(w, g, acc, mx, dw);
      else if ((int64_t)lo < wlo) acc_store(w.part + 2 * win, acc);  // continued from before
      else acc_store(w.part + 2 * win + 1, acc);                      // continues after
    }
  }
}

// partial j of a row whose items span windows w0 .. w1: the part of w0 it
// continues into, then each later window's continued part
__device__ __forceinline__ const PartRow *row_part(const AggWork &w, int64_t w0, int64_t j) {
  return j == 0 ? w.part + 2 * w0 + 1 : w.part + 2 * (w0 + j);
}

// Spread rows (items over several windows) are found by row when there are
// fewer rows than windows (3a lists them), else by window (3b checks each).
__device__ __forceinline__ bool spread_by_row(const AggWork &w) {
  return (int64_t)w.G < (w.meta[0] + kWinItems - 1) / kWinItems;
}

// 3a. rows without items: zero counts and no values, written by each wave
// over its 64 consecutive rows with coalesced 8-byte stores. A row inside
// one window was written by its window. When spread rows are found by row,
// they are listed here, with one atomic per block (atomics on one address
// serialise across the chip).
template <bool DEF>  // the kinds do not matter here; one instance is used
__global__ void __launch_bounds__(256) k_row_triage(AggWork w) {
  __shared__ uint32_t wcnt[4];
  __shared__ unsigned long long bbase;
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  const int ln = lane_id();
  bool empty = false, spread = false;
  if (g < w.G) {
    const uint32_t lo = w.goff[g], hi = w.goff[g + 1];
    empty = hi == lo;
    spread = !empty && lo / kWinItems != (hi - 1) / kWinItems;
  }
  if (spread_by_row(w)) {  // uniform over the grid
    const unsigned long long sm = __ballot(spread);
    if (ln == 0) wcnt[wave_id()] = (uint32_t)__popcll(sm);
    __syncthreads();
    if (threadIdx.x == 0) {
      const uint32_t n = wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
      bbase = n ? atomicAdd((unsigned long long *)&w.meta[4], (unsigned long long)n) : 0ull;
    }
    __syncthreads();
    if (spread) {
      unsigned long long pos = bbase;
      for (int k = 0; k < wave_id(); ++k) pos += wcnt[k];
      w.multi[pos + __popcll(sm & ((1ull << ln) - 1ull))] = g;
    }
  }
  const unsigned long long em = __ballot(empty);
  if (em) {
    constexpr int kWords = (int)(sizeof(opattr_op_row) / 8);
    static_assert(kWords == 24, "row layout: four counts, then the counter values");
    unsigned long long *dst = reinterpret_cast<unsigned long long *>(w.table + (g - ln));
    for (int x = ln; x < OPA_WAVE * kWords; x += OPA_WAVE) {
      const int r = x / kWords, c = x % kWords;
      if ((em >> r) & 1ull) dst[x] = c < 4 ? 0ull : 0x7FF8000000000000ull;
    }
  }
}

// The spread row g over windows w0 .. w1, by one wave. A row over more than
// kHeavy windows is reduced in chunks of kChunk partials instead: it reserves
// consecutive chunk slots, fills them (row, chunk) and lists itself with the
// first of them.
template <bool DEF>
__device__ __forceinline__ void combine_row(const AggWork &w, uint32_t g, int64_t w0, int64_t w1) {
  const uint32_t mx = DEF ? kDefMaxMask : w.in.maxmask, dw = DEF ? kDefDwMask : w.in.dwmask;
  const int ln = lane_id();
  const uint32_t m = (uint32_t)(w1 - w0 + 1);
  if (m > kHeavy) {
    const uint32_t nch = (m + kChunk - 1) / kChunk;
    uint32_t base = 0;
    if (ln == 0) {
      base = (uint32_t)atomicAdd((unsigned long long *)&w.meta[3], (unsigned long long)nch);
      const uint64_t h = atomicAdd((unsigned long long *)&w.meta[5], 1ull);
      w.heavy[2 * h] = g;
      w.heavy[2 * h + 1] = base;
    }
    base = __shfl(base, 0, OPA_WAVE);
    for (uint32_t c = ln; c < nch; c += OPA_WAVE)
      if ((int64_t)base + c < w.hcap) w.hch[base + c] = ((unsigned long long)g << 32) | c;
    return;
  }
  Acc acc;
  acc_zero(acc);
  for (uint32_t j = ln; j < m; j += OPA_WAVE) {
    Acc b;
    acc_load(b, row_part(w, w0, j));
    acc_merge(acc, b, mx);
  }
  acc_wave_reduce(acc, mx);
  write_row(w, g, acc, mx, dw);
}

// 3b. the spread rows, one wave each: from the list of 3a, or else one wave
// per window: the window whose first item's row began in an earlier window
// and ends in it combines that row (every spread row has exactly one such
// window)
template <bool DEF>
__global__ void __launch_bounds__(256) k_combine(AggWork w) {
  const int64_t nwin = (w.meta[0] + kWinItems - 1) / kWinItems;
  const int64_t wave = (int64_t)blockIdx.x * 4 + wave_id(), nwaves = (int64_t)gridDim.x * 4;
  if (spread_by_row(w)) {
    const int64_t nm = w.meta[4];
    for (int64_t k = wave; k < nm; k += nwaves) {
      const uint32_t g = w.multi[k];
      const uint32_t lo = w.goff[g], hi = w.goff[g + 1];
      combine_row<DEF>(w, g, lo / kWinItems, (hi - 1) / kWinItems);
    }
    return;
  }
  for (int64_t win = wave; win < nwin; win += nwaves) {
    const uint32_t g = (uint32_t)(w.sit[win * kWinItems] >> 36);
    const uint32_t lo = w.goff[g], hi = w.goff[g + 1];
    if ((int64_t)lo >= win * kWinItems || (int64_t)(hi - 1) / kWinItems != win) continue;
    combine_row<DEF>(w, g, lo / kWinItems, win);
  }
}

// 3c. one block per chunk slot: its kChunk partials, one per thread, merged
// in order (lanes, then waves) into the slot's partial
__global__ void __launch_bounds__(kChunk) k_heavy_chunks(AggWork w) {
  const uint32_t mx = w.in.maxmask;
  __shared__ PartRow red[kChunk / OPA_WAVE];
  const int64_t ns = w.meta[3] < w.hcap ? w.meta[3] : w.hcap;
  // the slots are sized so that this cannot happen; if it did, rows would
  // lose partials, so it is reported rather than left silent
  if (blockIdx.x == 0 && threadIdx.x == 0 && w.meta[3] > w.hcap)
    atomicOr(&w.diag->flags, OPATTR_F_LIMIT);
  for (int64_t sl = blockIdx.x; sl < ns; sl += gridDim.x) {
    const unsigned long long e = w.hch[sl];
    const uint32_t g = (uint32_t)(e >> 32), c = (uint32_t)e;
    const uint32_t lo = w.goff[g], hi = w.goff[g + 1];
    const int64_t w0 = lo / kWinItems, w1 = (hi - 1) / kWinItems;
    const int64_t j = (int64_t)c * kChunk + threadIdx.x;
    Acc acc;
    acc_zero(acc);
    if (j < w1 - w0 + 1) acc_load(acc, row_part(w, w0, j));
    acc_wave_reduce(acc, mx);
    __syncthreads();  // red is free (previous slot done)
    if (lane_id() == 0) acc_store(red + wave_id(), acc);
    __syncthreads();
    if (threadIdx.x == 0) {
      Acc t;
      acc_load(t, red);
      for (int k = 1; k < kChunk / OPA_WAVE; ++k) {
        Acc b;
        acc_load(b, red + k);
        acc_merge(t, b, mx);
      }
      acc_store(w.hpart + sl, t);
    }
  }
}

// 3d. one wave per heavy row: its chunk partials in order, and the row
template <bool DEF>
__global__ void __launch_bounds__(256) k_heavy_rows(AggWork w) {
  const uint32_t mx = DEF ? kDefMaxMask : w.in.maxmask, dw = DEF ? kDefDwMask : w.in.dwmask;
  const int64_t nh = w.meta[5];
  const int ln = lane_id();
  for (int64_t h = (int64_t)blockIdx.x * 4 + wave_id(); h < nh; h += (int64_t)gridDim.x * 4) {
    const uint32_t g = w.heavy[2 * h], base = w.heavy[2 * h + 1];
    const uint32_t lo = w.goff[g], hi = w.goff[g + 1];
    const uint32_t m = (uint32_t)((hi - 1) / kWinItems - lo / kWinItems + 1);
    const uint32_t nch = (m + kChunk - 1) / kChunk;
    Acc acc;
    acc_zero(acc);
    for (uint32_t c = ln; c < nch; c += OPA_WAVE) {
      if ((int64_t)base + c >= w.hcap) break;
      Acc b;
      acc_load(b, w.hpart + base + c);
      acc_merge(acc, b, mx);
    }
    acc_wave_reduce(acc, mx);
    write_row(w, g, acc, mx, dw);
  }
}

static AggWork agg_work(const EncArgs &x) {
  const Plan &pl = *x.pl;
  AggWork w{};
  w.G = pl.G;
  w.tcap = pl.ntrt;
  w.NOPS = x.d->n_ops;
  w.absent = x.p->absent_mask;
  w.in = agg_inputs(x);
  w.ig = at<uint32_t>(x.ws, pl.ig);
  w.ia = at<uint32_t>(x.ws, pl.ia);
  w.ib = at<uint32_t>(x.ws, pl.ib);
  w.rows = at<PartRow>(x.ws, pl.rows);
  w.meta = at<int64_t>(x.ws, pl.meta);
  w.ith = at<uint32_t>(x.ws, pl.ith);
  w.gcnt = at<uint32_t>(x.ws, pl.gcnt);
  w.goff = at<uint32_t>(x.ws, pl.goff);
  w.heavy = at<uint32_t>(x.ws, pl.heavy);
  w.multi = at<uint32_t>(x.ws, pl.multi);
  w.hch = at<unsigned long long>(x.ws, pl.hch);
  w.hpart = at<PartRow>(x.ws, pl.hpart);
  w.hcap = pl.hcap;
  w.sit = at<unsigned long long>(x.ws, pl.sit);
  w.part = at<PartRow>(x.ws, pl.part);
  w.table = x.table;
  w.sum = x.sum;
  w.diag = x.diag;
  return w;
}

void plan_items(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  AggWork w = agg_work(x);
  probe_begin(OPATTR_PROBE_ITEM_SORT, s);
  if (pl.G <= kFastKeys) {
    const size_t lds = (size_t)4 * pl.G * sizeof(uint16_t);
    const unsigned tgrid = (unsigned)(pl.ntrt < 1024 ? (pl.ntrt > 0 ? pl.ntrt : 1) : 1024);
    // gcnt (and meta when there are no launches) were cleared before the
    // enclosure pass counted the items
    if (pl.T > 0) {
      k_item_hist_w<<<tgrid, 256, lds, s>>>(w);
      column_scan(w.ith, pl.ntrt, pl.G, at<uint32_t>(x.ws, pl.itch), w.gcnt, s, w.meta + 2);
    }
    k_row_offsets<<<1, 1024, 0, s>>>(w);
    if (pl.T > 0) k_item_scatter_w<<<tgrid, 256, lds, s>>>(w);
  } else {
    const int64_t cap = pl.cap_items;
    uint32_t *k0 = at<uint32_t>(x.ws, pl.isort_k0), *k1 = at<uint32_t>(x.ws, pl.isort_k1);
    uint32_t *v0 = at<uint32_t>(x.ws, pl.isort_v0), *v1 = at<uint32_t>(x.ws, pl.isort_v1);
    bool in1 = false;
    if (cap > 0) {
      k_item_keys<<<(unsigned)((cap + 255) / 256), 256, 0, s>>>(w, k0, v0, cap);
      const int bits = (bits_for_host(pl.G) + 7) & ~7;
      in1 = radix_sort_pairs(k0, v0, k1, v1, cap, 0, bits,
                             at<uint32_t>(x.ws, pl.isort_hist), s, w.meta);
    }
    if (cap > 0)
      k_item_place<<<(unsigned)((cap + 255) / 256), 256, 0, s>>>(w, in1 ? k1 : k0, in1 ? v1 : v0,
                                                                 cap);
    k_row_bounds<<<(pl.G + 1 + 255) / 256, 256, 0, s>>>(w, in1 ? k1 : k0, cap);
  }
  probe_end(OPATTR_PROBE_ITEM_SORT, s);
}

// the rows without items and the listing of spread rows need only the
// sorted items' row offsets, so they can run before the window reduction
void triage_rows(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const AggWork w = agg_work(x);
  k_row_triage<true><<<(pl.G + 255) / 256, 256, 0, s>>>(w);
}

void reduce_items(const EncArgs &x, hipStream_t s, bool triaged) {
  const Plan &pl = *x.pl;
  AggWork w = agg_work(x);
  const bool def = w.in.maxmask == kDefMaxMask && w.in.dwmask == kDefDwMask;
  probe_begin(OPATTR_PROBE_AGGREGATE, s);
  if (pl.T > 0) {
    const int64_t want = (pl.max_windows + 3) / 4;
    const unsigned cgrid = (unsigned)(want < 2048 ? want : 2048);
    if (def) k_window_reduce<true><<<cgrid, 256, 0, s>>>(w);
    else k_window_reduce<false><<<cgrid, 256, 0, s>>>(w);
  }
  const unsigned tg = (pl.G + 255) / 256;
  const int64_t cw = (pl.max_windows + 3) / 4;
  const unsigned cg = (unsigned)(cw < 1024 ? (cw > 0 ? cw : 1) : 1024);
  const unsigned hg = (unsigned)(pl.hcap < 2048 ? pl.hcap : 2048);
  if (!triaged) k_row_triage<true><<<tg, 256, 0, s>>>(w);
  if (def) k_combine<true><<<cg, 256, 0, s>>>(w);
  else k_combine<false><<<cg, 256, 0, s>>>(w);
  k_heavy_chunks<<<hg, kChunk, 0, s>>>(w);
  if (def) k_heavy_rows<true><<<64, 256, 0, s>>>(w);
  else k_heavy_rows<false><<<64, 256, 0, s>>>(w);
  probe_end(OPATTR_PROBE_AGGREGATE, s);
}

}  // namespace opa
