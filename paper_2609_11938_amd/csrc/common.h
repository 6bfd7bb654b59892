// Device primitives shared by the opattr kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/opattr.h"

#define OPA_WAVE 64
#define OPA_TILE 4096          // elements per LDS tile (seq tiles, profiled tiles)
#define OPA_TILE_THREADS 256   // 4 waves, 16 elements per thread
#define OPA_TILE_CHUNKS (OPA_TILE / OPA_TILE_THREADS)
#define OPA_SLOT_BITS 12       // log2(OPA_TILE)

static_assert((1 << OPA_SLOT_BITS) == OPA_TILE, "tile size");

namespace opa {

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (OPA_WAVE - 1)); }
__device__ __forceinline__ int wave_id() { return (int)(threadIdx.x / OPA_WAVE); }
__device__ __forceinline__ uint64_t lanemask_lt() {
  return (1ull << lane_id()) - 1ull;
}

// Lanes of the wave holding the same 8-bit digit (match-any built from one
// ballot per bit: the published warp-multisplit peer-mask construction).
__device__ __forceinline__ uint64_t peers8(uint32_t d) {
  uint64_t m = ~0ull;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint64_t v = __ballot((d >> b) & 1u);
    m &= ((d >> b) & 1u) ? v : ~v;
  }
  return m;
}

// Lanes whose keys agree on bits [0, nbits) (nbits uniform across the wave).
__device__ __forceinline__ uint64_t match_any_bits(uint32_t key, int nbits) {
  uint64_t m = ~0ull;
  for (int b = 0; b < nbits; ++b) {
    const uint32_t bit = (key >> b) & 1u;
    const uint64_t v = __ballot(bit);
    m &= bit ? v : ~v;
  }
  return m;
}

// Stable ranking with per-wave counters. The wave owns CH chunks of 64
// elements, visited in order; key[c] is the lane's key in chunk c. On return
// rank[c] = number of earlier elements of the wave with the same key, and
// cnt[k] (this wave's counters in LDS, zeroed by the caller) has grown by the
// wave's count of key k. Keys >= K are skipped; all of them must equal K and
// K < 2^nbits.
template <int CH>
__device__ __forceinline__ void wave_rank(const uint32_t (&key)[CH], uint32_t K, int nbits,
                                          uint16_t *cnt, uint32_t (&rank)[CH]) {
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const uint32_t k = key[c];
    if (__ballot(k < K) == 0) {  // nothing to rank in this chunk
      rank[c] = 0;
      continue;
    }
    const uint64_t pm = match_any_bits(k, nbits);
    const uint32_t lr = (uint32_t)__popcll(pm & lt);
    uint32_t r = 0;
    if (k < K) {
      const uint32_t c0 = cnt[k];
      r = c0 + lr;
      if (lr == 0) cnt[k] = (uint16_t)(c0 + (uint32_t)__popcll(pm));
    }
    rank[c] = r;
  }
}

// After wave_rank over a 4-wave block: turn the per-wave counters cnt[w*K+n]
// into the count of key n in earlier waves, and write the block totals to
// total[n] (if given). Call from all threads; ends with a barrier.
__device__ __forceinline__ void block_rank_bases(uint16_t *cnt, uint32_t K, uint32_t *total) {
  __syncthreads();
  for (uint32_t n = threadIdx.x; n < K; n += blockDim.x) {
    const uint32_t a = cnt[n], b = cnt[K + n], c = cnt[2 * K + n], d = cnt[3 * K + n];
    cnt[n] = 0;
    cnt[K + n] = (uint16_t)a;
    cnt[2 * K + n] = (uint16_t)(a + b);
    cnt[3 * K + n] = (uint16_t)(a + b + c);
    if (total) total[n] = a + b + c + d;
  }
  __syncthreads();
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan_add(T x) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    T y = __shfl_up(x, o, OPA_WAVE);
    if (l >= o) x += y;
  }
  return x;
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan_max(T x) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    T y = __shfl_up(x, o, OPA_WAVE);
    if (l >= o) x = y > x ? y : x;
  }
  return x;
}

template <typename T>
__device__ __forceinline__ T wave_reduce_add(T x) {
#pragma unroll
  for (int o = OPA_WAVE / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, OPA_WAVE);
  return x;
}

// Exclusive scan across a 256-thread block of one value per thread.
// `sh` needs 4 entries. Returns the exclusive prefix; *total gets the sum.
template <typename T>
__device__ __forceinline__ T block_excl_scan_add(T x, T *sh, T *total) {
  T inc = wave_incl_scan_add(x);
  const int w = wave_id(), l = lane_id();
  if (l == OPA_WAVE - 1) sh[w] = inc;
  __syncthreads();
  T base = 0, tot = 0;
  for (int i = 0; i < (int)(blockDim.x / OPA_WAVE); ++i) {
    if (i < w) base += sh[i];
    tot += sh[i];
  }
  __syncthreads();
  if (total) *total = tot;
  return base + inc - x;
}

// Exclusive scan of a[0, n) in place by one block: each thread takes a
// contiguous chunk, so the block synchronises for one scan only. sh needs
// blockDim.x / 64 entries. Returns the total.
__device__ inline uint32_t block_scan_chunked(uint32_t *a, int64_t n, uint32_t *sh) {
  const int64_t ch = (n + blockDim.x - 1) / blockDim.x;
  const int64_t lo = (int64_t)threadIdx.x * ch;
  const int64_t hi = lo + ch < n ? lo + ch : n;
  uint32_t sum = 0;
  for (int64_t i = lo; i < hi; ++i) sum += a[i];
  uint32_t tot;
  uint32_t run = block_excl_scan_add<uint32_t>(sum, sh, &tot);
  for (int64_t i = lo; i < hi; ++i) {
    const uint32_t v = a[i];
    a[i] = run;
    run += v;
  }
  return tot;
}

// Inclusive max-scan across the block; values per thread, block of 256.
template <typename T>
__device__ __forceinline__ T block_incl_scan_max(T x, T *sh) {
  T inc = wave_incl_scan_max(x);
  const int w = wave_id(), l = lane_id();
  if (l == OPA_WAVE - 1) sh[w] = inc;
  __syncthreads();
  T base = inc;
  for (int i = 0; i < w; ++i) base = sh[i] > base ? sh[i] : base;
  __syncthreads();
  return base;
}

// ---------------------------------------------------------------------------
// Stable LDS radix sort of one tile of OPA_TILE 32-bit keys by bits
// [lo_bit, lo_bit + nbits), 8 bits per pass, 256 threads. Element order is
// index order (chunk c, thread t) -> index c*256 + t. `a` holds the keys and
// receives the result; `b` is scratch of the same size; `cnt` needs
// OPA_TILE_CHUNKS * 4 * 256 uint16 entries; `dbase` 256 + 4 uint32 entries.
// ---------------------------------------------------------------------------
struct TileSortSmem {
  uint16_t cnt[OPA_TILE_CHUNKS][OPA_TILE_THREADS / OPA_WAVE][256];
  uint32_t dbase[256];
  uint32_t sh[8];
};

__device__ inline void tile_radix_sort(uint32_t *a, uint32_t *b, TileSortSmem &sm, int lo_bit,
                                       int nbits) {
  const int tid = threadIdx.x, w = wave_id();
  for (int shift = lo_bit; shift < lo_bit + nbits; shift += 8) {
    const int take = (lo_bit + nbits - shift) < 8 ? (lo_bit + nbits - shift) : 8;
    const uint32_t mask = (1u << take) - 1u;
    // per (chunk, wave) digit counts
    for (int i = tid; i < OPA_TILE_CHUNKS * 4 * 256; i += OPA_TILE_THREADS)
      (&sm.cnt[0][0][0])[i] = 0;
    __syncthreads();
    uint32_t lrank[OPA_TILE_CHUNKS];
    uint32_t dig[OPA_TILE_CHUNKS];
#pragma unroll
    for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
      const uint32_t k = a[c * OPA_TILE_THREADS + tid];
      const uint32_t d = (k >> shift) & mask;
      const uint64_t pm = peers8(d);
      dig[c] = d;
      lrank[c] = (uint32_t)__popcll(pm & lanemask_lt());
      if ((pm & lanemask_lt()) == 0) sm.cnt[c][w][d] = (uint16_t)__popcll(pm);
    }
    __syncthreads();
    // thread d scans its digit over (chunk, wave) in index order
    {
      const int d = tid;
      uint32_t run = 0;
      for (int c = 0; c < OPA_TILE_CHUNKS; ++c)
        for (int ww = 0; ww < OPA_TILE_THREADS / OPA_WAVE; ++ww) {
          const uint32_t v = sm.cnt[c][ww][d];
          sm.cnt[c][ww][d] = (uint16_t)run;
          run += v;
        }
      uint32_t tot;
      const uint32_t base = block_excl_scan_add<uint32_t>(run, sm.sh, &tot);
      sm.dbase[d] = base;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
      const uint32_t d = dig[c];
      const uint32_t dst = sm.dbase[d] + sm.cnt[c][w][d] + lrank[c];
      b[dst] = a[c * OPA_TILE_THREADS + tid];
    }
    __syncthreads();
    for (int i = tid; i < OPA_TILE; i += OPA_TILE_THREADS) a[i] = b[i];
    __syncthreads();
  }
}

__device__ __forceinline__ int bits_for(uint32_t v) {  // bits to hold values 0..v
  return v == 0 ? 1 : 32 - __clz(v);
}

// first index in sorted LDS array a[0..n) with a[i] >= x
__device__ __forceinline__ int lds_lower_bound(const uint32_t *a, int n, uint32_t x) {
  int lo = 0, hi = n;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

struct TileSmem {
  uint32_t A[OPA_TILE];
  uint32_t B[OPA_TILE];
  TileSortSmem srt;
  int32_t sh[16];
  uint32_t bad;
};

// hist[tile][n] = eligible launches of name n in the tile (all n < NN)
__device__ inline void write_hist_row(const uint32_t *A, uint32_t NN, uint32_t *row) {
  for (uint32_t n = threadIdx.x; n < NN; n += OPA_TILE_THREADS) {
    const int lo = lds_lower_bound(A, OPA_TILE, n << OPA_SLOT_BITS);
    const int hi = lds_lower_bound(A, OPA_TILE, (n + 1) << OPA_SLOT_BITS);
    row[n] = (uint32_t)(hi - lo);
  }
}

// Diag helpers: device-scope atomics on the caller's record.
__device__ __forceinline__ void diag_flag(opattr_diag *d, uint32_t f) {
  if (d) atomicOr(&d->flags, f);
}
__device__ __forceinline__ void diag_add(unsigned long long *p, unsigned long long v) {
  if (v) atomicAdd(p, v);
}


// blk[s] = first position with stream >= s in st[0..n) (sorted by stream);
// called by one whole wave: each round, the 64 lanes probe 64 evenly spaced
// positions and the range shrinks to the gap where the answer lies.
__device__ inline void stream_block_wave(const uint16_t *st, int64_t n, uint32_t s, int64_t *blk) {
  const int ln = lane_id();
  int64_t lo = 0, hi = n;  // answer in [lo, hi]
  while (hi - lo > OPA_WAVE) {
    const int64_t step = (hi - lo + OPA_WAVE - 1) / OPA_WAVE;
    int64_t p = lo + (int64_t)(ln + 1) * step - 1;
    if (p > hi - 1) p = hi - 1;
    const uint64_t m = __ballot(st[p] >= s);
    if (m == 0) {
      lo = hi;
      break;
    }
    const int f = __ffsll((unsigned long long)m) - 1;  // first probe at or past s
    int64_t pf = lo + (int64_t)(f + 1) * step - 1;
    if (pf > hi - 1) pf = hi - 1;
    lo = f == 0 ? lo : lo + (int64_t)f * step;
    hi = pf;  // st[pf] >= s
  }
  if (hi - lo <= OPA_WAVE && lo < hi) {
    const int64_t p = lo + ln;
    const uint64_t m = __ballot(p < hi && st[p] >= s);
    lo = m ? lo + __ffsll((unsigned long long)m) - 1 : hi;
  }
  if (ln == 0) blk[s] = lo;
}

// The finalisation, by one block of any size: nesting_errors from the
// per-stream crossing flags; with part, the summary from the per-block sums;
// then the flags and the status from every stage's diagnostics
__device__ inline void finish_block(opattr_diag *diag, const uint8_t *sflag, uint32_t ns,
                                    const unsigned long long *part, int nparts,
                                    opattr_summary *sum) {
  __shared__ uint32_t cnt;
  __shared__ unsigned long long tot[4];
  if (threadIdx.x < 4) tot[threadIdx.x] = 0;
  if (threadIdx.x == 0) cnt = 0;
  __syncthreads();
  if (sflag) {
    uint32_t c = 0;
    for (uint32_t s = threadIdx.x; s < ns; s += blockDim.x) c += sflag[s] ? 1u : 0u;
    if (c) atomicAdd(&cnt, c);
  }
  // the per-block sums, one block's four per thread (integer sums: exact in
  // any order)
  if (part) {
    unsigned long long v[4] = {0, 0, 0, 0};
    for (int b = threadIdx.x; b < nparts; b += blockDim.x)
#pragma unroll
      for (int f = 0; f < 4; ++f) v[f] += part[b * 4 + f];
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const unsigned long long x = wave_reduce_add(v[f]);
      if (lane_id() == 0 && x) atomicAdd(&tot[f], x);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0 && part) {
    opattr_summary s{};
    s.attributed_ns = tot[0];
    s.unattributed_ns = tot[1];
    s.total_ns = tot[2];
    s.matched_ns = tot[3];
    s.attributed_fraction = s.total_ns ? (double)s.attributed_ns / (double)s.total_ns
                                       : __longlong_as_double(0x7FF8000000000000ll);
    *sum = s;
  }
  if (threadIdx.x == 0) {
    if (sflag) diag->nesting_errors = cnt;
    uint32_t f = diag->flags;
    if (diag->nesting_errors) f |= OPATTR_F_NOT_NESTED;
    if (diag->bad_records) f |= OPATTR_F_DATA;
    if (diag->dedup_errors) f |= OPATTR_F_DEDUP;
    diag->flags = f;
    int32_t st = 0;
    if (f & OPATTR_F_DATA) st = OPATTR_ERR_DATA;
    else if (f & OPATTR_F_ORDER) st = OPATTR_ERR_ORDER;
    else if (f & OPATTR_F_LIMIT) st = OPATTR_ERR_LIMIT;
    else if (f & OPATTR_F_NOT_NESTED) st = OPATTR_ERR_NOT_NESTED;
    else if (f & OPATTR_F_PARTITION) st = OPATTR_ERR_PARTITION;
    else if (f & OPATTR_F_DEDUP) st = OPATTR_ERR_DEDUP;
    else if ((f & OPATTR_F_COUNT) && diag->strict) st = OPATTR_ERR_COUNT_MISMATCH;
    diag->status = st;
  }
}

// Depth of range x in nesting order (length of its parent chain: 1 for a
// root, 0 for a bad range, ree < 0) into range_depth by input position (perm,
// or x without one); a chain longer than 255 sets the LIMIT flag. Called by
// whole waves.
__device__ inline void range_depth_one(const int32_t *npg, const int64_t *ree, const uint16_t *st,
                                       const int32_t *perm, int64_t n, uint32_t NS, int64_t x,
                                       uint8_t *range_depth, opattr_diag *diag) {
  bool lim = false;
  if (x < n) {
    int d = 0;
    int32_t y = (int32_t)x;
    while (y >= 0 && d <= 255) {
      ++d;
      y = npg[y];
    }
    lim = y >= 0;
    const bool ok = ree[x] >= 0 && st[x] < NS;
    if (range_depth) {
      const int64_t o = perm ? perm[x] : x;
      range_depth[o] = ok ? (uint8_t)(d > 255 ? 255 : d) : 0;
    }
    lim = lim && ok;
  }
  if (__ballot(lim) && lane_id() == 0) atomicOr(&diag->flags, OPATTR_F_LIMIT);
}

}  // namespace opa
