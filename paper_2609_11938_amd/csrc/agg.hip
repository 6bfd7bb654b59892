// Per-operator aggregation (Eq. 1, Sec. 3.8.1), second and third levels.
//
// The enclosure pass plans, in launch order, items of one operator row each:
// either a partial row (a run reduced in place once the matches are known)
// or a reference to at most 16 launches. Here the items are
//   1. counting-sorted by row (per-tile row histograms scanned down the
//      columns; stable, so each row keeps its items in launch order); this
//      needs only the rows, so it runs beside the matching,
//   2. cut into chunks of at most 64 items of one row, each reduced by one
//      wave (a lane loads a partial row or accumulates its referenced
//      launches, then a butterfly reduction),
//   3. finalised (duration-weighted means divided by the matched duration,
//      NaN for absent counters and rows without matched launches): a row of
//      one chunk by the wave that reduced it, a row of several chunks by one
//      wave that combines them in chunk order in a second pass. The summary
//      over the table is taken by the finishing kernel.
// Every sum is taken in a fixed order, so results are reproducible.
#include "accum.h"
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kChunkItems = 64;

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
  int64_t *meta;  // [0] items, [1] partial rows, [2] item tiles, [3] chunks
  uint32_t *ith, *gcnt, *goff, *coff, *cmap;
  unsigned long long *sit;  // sorted items: partial-row index or first launch | length << 32
  PartRow *part;
  opattr_op_row *table;
  opattr_summary *sum;
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

// 1a'. the same with an LDS radix sort per tile, for many rows
__global__ void __launch_bounds__(256) k_item_hist_r(AggWork w) {
  __shared__ TileSmem sm;
  const int64_t n = w.meta[0];
  const int64_t ntiles = (n + OPA_TILE - 1) / OPA_TILE;
  if (blockIdx.x == 0 && threadIdx.x == 0) w.meta[2] = ntiles;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    __syncthreads();
    for (int l = threadIdx.x; l < OPA_TILE; l += 256) {
      const int64_t x = tile * OPA_TILE + l;
      const uint32_t g = x < n ? w.ig[x] : w.G;
      sm.A[l] = (g << OPA_SLOT_BITS) | (uint32_t)l;
    }
    __syncthreads();
    tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(w.G));
    write_hist_row(sm.A, w.G, w.ith + tile * w.G);
  }
}

// 1b. row offsets of the sorted items and chunk offsets (one block; each
// thread scans a contiguous run of rows)
__global__ void __launch_bounds__(1024) k_row_offsets(AggWork w) {
  __shared__ uint32_t sh[16];
  const uint32_t ch = (w.G + blockDim.x - 1) / blockDim.x;
  const uint32_t lo = threadIdx.x * ch;
  const uint32_t hi = lo + ch < w.G ? lo + ch : w.G;
  uint32_t c = 0, cc = 0;
  for (uint32_t g = lo; g < hi; ++g) {
    const uint32_t n = w.gcnt[g];
    c += n;
    cc += (n + kChunkItems - 1) / kChunkItems;
  }
  uint32_t tot, ctot;
  uint32_t run = block_excl_scan_add<uint32_t>(c, sh, &tot);
  uint32_t crun = block_excl_scan_add<uint32_t>(cc, sh, &ctot);
  for (uint32_t g = lo; g < hi; ++g) {
    const uint32_t n = w.gcnt[g];
    w.goff[g] = run;
    w.coff[g] = crun;
    run += n;
    crun += (n + kChunkItems - 1) / kChunkItems;
  }
  if (threadIdx.x == 0) {
    w.goff[w.G] = tot;
    w.coff[w.G] = ctot;
    w.meta[3] = ctot;
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
      w.sit[w.goff[g] + row[g] + wb[g] + rank[c]] = w.ia[x] | ((unsigned long long)w.ib[x] << 32);
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

__global__ void __launch_bounds__(256) k_item_scatter_r(AggWork w) {
  __shared__ TileSmem sm;
  const int64_t n = w.meta[0];
  const int64_t ntiles = (n + OPA_TILE - 1) / OPA_TILE;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    __syncthreads();
    for (int l = threadIdx.x; l < OPA_TILE; l += 256) {
      const int64_t x = tile * OPA_TILE + l;
      const uint32_t g = x < n ? w.ig[x] : w.G;
      sm.A[l] = (g << OPA_SLOT_BITS) | (uint32_t)l;
    }
    __syncthreads();
    tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(w.G));
    const uint32_t *row = w.ith + tile * w.G;
    for (int p = threadIdx.x; p < OPA_TILE; p += 256) {
      const uint32_t key = sm.A[p];
      const uint32_t g = key >> OPA_SLOT_BITS;
      if (g >= w.G) continue;
      const int lo = lds_lower_bound(sm.A, OPA_TILE, g << OPA_SLOT_BITS);
      const int64_t x = tile * OPA_TILE + (key & (OPA_TILE - 1));
      w.sit[w.goff[g] + row[g] + (uint32_t)(p - lo)] =
          w.ia[x] | ((unsigned long long)w.ib[x] << 32);
    }
  }
}

// 1d. chunk -> row map
__global__ void k_chunk_map(AggWork w) {
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= w.G) return;
  const uint32_t c0 = w.coff[g], c1 = w.coff[g + 1];  // read once: cmap may alias
  for (uint32_t c = c0; c < c1; ++c) w.cmap[c] = g;
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

// 2. one wave per chunk of at most 64 items of one row; a row's only chunk
// is finalised right away
template <bool DEF>
__global__ void __launch_bounds__(256) k_chunk_reduce(AggWork w) {
  const uint32_t mx = DEF ? kDefMaxMask : w.in.maxmask, dw = DEF ? kDefDwMask : w.in.dwmask;
  const int64_t nch = w.meta[3];
  const int ln = lane_id();
  for (int64_t ch = (int64_t)blockIdx.x * 4 + wave_id(); ch < nch; ch += (int64_t)gridDim.x * 4) {
    const uint32_t g = w.cmap[ch];
    const uint32_t c0 = w.coff[g];
    const uint32_t p = w.goff[g] + (uint32_t)(ch - c0) * kChunkItems + (uint32_t)ln;
    Acc acc;
    acc_zero(acc);
    if (p < w.goff[g + 1]) {
      const unsigned long long it = w.sit[p];
      const uint32_t a = (uint32_t)it, b = (uint32_t)(it >> 32);
      if (b == 0) {
        acc_load(acc, w.rows + a);
      } else {
        for (uint32_t k = 0; k < b; ++k)
          acc_launch(acc, w.in, w.in.match[a + k], w.in.dur[a + k], mx, dw);
      }
    }
    acc_wave_reduce(acc, mx);
    if (w.coff[g + 1] - c0 == 1) write_row(w, g, acc, mx, dw);
    else if (ln == 0) acc_store(w.part + ch, acc);
  }
}

// 3. one wave per operator row with no or several chunks
template <bool DEF>
__global__ void __launch_bounds__(256) k_combine(AggWork w) {
  const uint32_t mx = DEF ? kDefMaxMask : w.in.maxmask, dw = DEF ? kDefDwMask : w.in.dwmask;
  const uint32_t g = blockIdx.x * 4 + wave_id();
  if (g >= w.G) return;
  const int ln = lane_id();
  const uint32_t c0 = w.coff[g], c1 = w.coff[g + 1];
  if (c1 - c0 == 1) return;  // finalised with its chunk
  Acc acc;
  acc_zero(acc);
  for (uint32_t c = c0 + ln; c < c1; c += OPA_WAVE) {
    Acc b;
    acc_load(b, w.part + c);
    acc_merge(acc, b, mx);
  }
  acc_wave_reduce(acc, mx);
  write_row(w, g, acc, mx, dw);
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
  w.coff = at<uint32_t>(x.ws, pl.coff);
  w.cmap = at<uint32_t>(x.ws, pl.cmap);
  w.sit = at<unsigned long long>(x.ws, pl.sit);
  w.part = at<PartRow>(x.ws, pl.part);
  w.table = x.table;
  w.sum = x.sum;
  return w;
}

void plan_items(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  AggWork w = agg_work(x);
  const bool fast = pl.G <= kFastKeys;
  const size_t lds = (size_t)4 * pl.G * sizeof(uint16_t);
  const unsigned tgrid = (unsigned)(pl.ntrt < 1024 ? (pl.ntrt > 0 ? pl.ntrt : 1) : 1024);
  // gcnt (and meta when there are no launches) were cleared with the
  // look-back states
  probe_begin(OPATTR_PROBE_ITEM_SORT, s);
  if (pl.T > 0) {
    if (fast) k_item_hist_w<<<tgrid, 256, lds, s>>>(w);
    else k_item_hist_r<<<tgrid, 256, 0, s>>>(w);
    column_scan(w.ith, pl.ntrt, pl.G, at<uint32_t>(x.ws, pl.itch), w.gcnt, s, w.meta + 2);
  }
  k_row_offsets<<<1, 1024, 0, s>>>(w);
  if (pl.T > 0) {
    if (fast) k_item_scatter_w<<<tgrid, 256, lds, s>>>(w);
    else k_item_scatter_r<<<tgrid, 256, 0, s>>>(w);
    k_chunk_map<<<(pl.G + 255) / 256, 256, 0, s>>>(w);
  }
  probe_end(OPATTR_PROBE_ITEM_SORT, s);
}

void reduce_items(const EncArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  AggWork w = agg_work(x);
  const bool def = w.in.maxmask == kDefMaxMask && w.in.dwmask == kDefDwMask;
  probe_begin(OPATTR_PROBE_AGGREGATE, s);
  if (pl.T > 0) {
    const int64_t want = (pl.max_chunks + 3) / 4;
    const unsigned cgrid = (unsigned)(want < 2048 ? want : 2048);
    if (def) k_chunk_reduce<true><<<cgrid, 256, 0, s>>>(w);
    else k_chunk_reduce<false><<<cgrid, 256, 0, s>>>(w);
  }
  if (def) k_combine<true><<<(pl.G + 3) / 4, 256, 0, s>>>(w);
  else k_combine<false><<<(pl.G + 3) / 4, 256, 0, s>>>(w);
  probe_end(OPATTR_PROBE_AGGREGATE, s);
}

}  // namespace opa
