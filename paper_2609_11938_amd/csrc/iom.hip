// Invocation-order matching (Alg. 1) and layer dedup (Sec. 3.7) on the GPU.
//
// Alg. 1 walks the launches in order and hands the i-th launch of a name the
// i-th profiled row of that name. Written data-parallel: the rank of a launch
// among the eligible launches of its name (in seq order) is
//     rank = (launches of the name in earlier seq tiles) + (rank inside the tile)
// and the row is slot[off[name] + rank] when rank < rows(name). Tiles of 4096
// launches in seq order are sorted by name in LDS (stable, so the in-tile rank
// is the distance to the start of the name's run); per-tile name histograms
// are scanned down the columns for the cross-tile part. The profiled side is
// ranked the same way (tiles in replay order) to build the slot table.
#include "common.h"
#include "impl.h"

namespace opa {

// ---------------------------------------------------------------------------
// seq view: sv[rank] = input index of the launch with that rank in seq order
// ---------------------------------------------------------------------------
__global__ void k_seqview_dense(const uint32_t *__restrict__ seq, int64_t T, int32_t *sv,
                                opattr_diag *diag, int validate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= T) return;
  const uint32_t s = seq[i];
  bool bad = false;
  if ((int64_t)s < T) {
    if (validate) bad = atomicCAS(&sv[s], -1, (int32_t)i) != -1;
    else sv[s] = (int32_t)i;
  } else {
    bad = validate != 0;
  }
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1) {
    atomicAdd((unsigned long long *)&diag->order_violations, (unsigned long long)__popcll(m));
    atomicOr(&diag->flags, OPATTR_F_ORDER);
  }
}

__global__ void k_seqview_sorted(const uint64_t *__restrict__ keys, const uint32_t *__restrict__ vals,
                                 int64_t T, int32_t *sv, int32_t *rk, opattr_diag *diag) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= T) return;
  const uint32_t j = vals[p];
  sv[p] = (int32_t)j;
  rk[j] = (int32_t)p;
  if (p > 0 && keys[p] == keys[p - 1]) atomicOr(&diag->flags, OPATTR_F_ORDER);  // seq not unique
}

void build_seq_view(const opattr_kernels *k, const opattr_dims *d, void *ws, const Plan &pl,
                    opattr_diag *diag, bool validate, hipStream_t s) {
  const int64_t T = pl.T;
  if (T <= 0) return;
  int32_t *sv = at<int32_t>(ws, pl.sv);
  const unsigned nb = (unsigned)((T + 255) / 256);
  if (pl.seq_dense) {
    fill_u32(reinterpret_cast<uint32_t *>(sv), 0xFFFFFFFFu, T, s);
    probe_begin(OPATTR_PROBE_SEQ_VIEW, s);
    k_seqview_dense<<<nb, 256, 0, s>>>(k->seq, T, sv, diag, validate ? 1 : 0);
    probe_end(OPATTR_PROBE_SEQ_VIEW, s);
    return;
  }
  probe_begin(OPATTR_PROBE_SEQ_VIEW, s);
  uint64_t *k0 = at<uint64_t>(ws, pl.seqsort_k0), *k1 = at<uint64_t>(ws, pl.seqsort_k1);
  uint32_t *v0 = at<uint32_t>(ws, pl.seqsort_v0), *v1 = at<uint32_t>(ws, pl.seqsort_v1);
  launch_iota(v0, T, s);
  launch_gather_key_u32(k->seq, v0, k0, T, s);
  const bool in1 = radix_sort_pairs(k0, v0, k1, v1, T, 0, 32, at<uint32_t>(ws, pl.rs_hist), s);
  k_seqview_sorted<<<nb, 256, 0, s>>>(in1 ? k1 : k0, in1 ? v1 : v0, T, sv,
                                       at<int32_t>(ws, pl.rk), diag);
  probe_end(OPATTR_PROBE_SEQ_VIEW, s);
}

// ---------------------------------------------------------------------------
// tile loading
// ---------------------------------------------------------------------------
struct TlArgs {
  const int32_t *sv;
  int64_t T;
  const uint32_t *name;
  const int32_t *part;      // NULL when dedup is off
  const int32_t *part_rep;  // NULL when dedup is off
  uint32_t NN, NP;
};

// Fill A[l] with (name << 12 | l) for launches eligible for replay, and
// (NN << 12 | l) otherwise, for the launches of seq ranks base..base+4095.
// lpart[l]: partition of a valid launch (-1 none), -2 for holes and bad ids.
// Returns the number of launches with an id out of range.
__device__ inline uint32_t tl_tile_keys(const TlArgs &a, int64_t base, uint32_t *A, int32_t *lpart,
                                        int32_t *jidx) {
  const int tid = threadIdx.x;
  uint32_t bad = 0;
#pragma unroll 4
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int l = c * OPA_TILE_THREADS + tid;
    const int64_t x = base + l;
    const int32_t j = x < a.T ? a.sv[x] : -1;
    uint32_t key = (a.NN << OPA_SLOT_BITS) | (uint32_t)l;
    int32_t lp = -2;
    if (j >= 0) {
      const uint32_t nm = a.name[j];
      const int32_t pt = a.part ? a.part[j] : -1;
      const bool good = nm < a.NN && pt >= -1 && (pt < 0 || (uint32_t)pt < a.NP);
      if (!good) {
        bad++;
      } else {
        const bool elig = pt < 0 || a.part_rep[pt] == pt;
        if (elig) key = (nm << OPA_SLOT_BITS) | (uint32_t)l;
        lp = pt;
      }
    }
    A[l] = key;
    if (lpart) lpart[l] = lp;
    if (jidx) jidx[l] = j;
  }
  return bad;
}

__global__ void __launch_bounds__(256) k_tl_hist(TlArgs a, uint32_t *tlh, opattr_diag *diag) {
  __shared__ TileSmem sm;
  const int64_t tile = blockIdx.x;
  const int64_t base = tile * OPA_TILE;
  if (threadIdx.x == 0) sm.bad = 0;
  __syncthreads();
  const uint32_t bad = tl_tile_keys(a, base, sm.A, nullptr, nullptr);
  if (bad) atomicAdd(&sm.bad, bad);
  __syncthreads();
  if (threadIdx.x == 0 && sm.bad)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)sm.bad);
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(a.NN));
  write_hist_row(sm.A, a.NN, tlh + tile * a.NN);
}

// ---------------------------------------------------------------------------
// Fast path for up to kFastKeys names: a tile of 4096 launches is owned by
// four waves, each walking 16 chunks of 64 in seq order and ranking names
// with its own LDS counters (wave_rank), so no in-LDS sort is needed.
// Element e of a tile sits in wave e / 1024, chunk (e / 64) % 16, lane e % 64.
// ---------------------------------------------------------------------------
constexpr int kWaveChunks = OPA_TILE / OPA_TILE_THREADS;  // 16 chunks per wave

__device__ __forceinline__ int tile_elem(int c) {
  return wave_id() * (OPA_TILE / 4) + c * OPA_WAVE + lane_id();
}

// One launch of seq rank x: input index j (-1 for holes), ranking key (its
// name if eligible for replay, else NN) and partition (-1 none, -2 hole or
// bad id). Returns 1 if an id is out of range.
__device__ __forceinline__ uint32_t tl_load(const TlArgs &a, int64_t x, uint32_t &key, int32_t &j,
                                            int32_t &lp) {
  j = (x >= 0 && x < a.T) ? a.sv[x] : -1;
  key = a.NN;
  lp = -2;
  if (j < 0) return 0;
  const uint32_t nm = a.name[j];
  const int32_t pt = a.part ? a.part[j] : -1;
  if (nm >= a.NN || pt < -1 || (pt >= 0 && (uint32_t)pt >= a.NP)) return 1;
  if (pt < 0 || a.part_rep[pt] == pt) key = nm;
  lp = pt;
  return 0;
}

// Partition edges of a seq tile. A head (first launch of a maximal run of one
// partition in seq order) stores its rank in pfirst, a tail in plast. With
// verify set, heads and tails instead compare against what is stored: a
// partition with two runs has two heads, only one of which can be stored, so
// the other one marks it non-contiguous.
__device__ inline uint32_t part_edges(const TlArgs &a, const int32_t *lpart, int64_t base,
                                      uint32_t *pfirst, uint32_t *plast, uint8_t *contig,
                                      bool verify) {
  uint32_t nbad = 0;
  for (int e = threadIdx.x; e < OPA_TILE; e += OPA_TILE_THREADS) {
    const int32_t lp = lpart[e];
    if (lp < 0) continue;
    const int64_t x = base + e;
    int32_t prev, next, jj;
    uint32_t kk;
    if (e > 0) prev = lpart[e - 1];
    else tl_load(a, x - 1, kk, jj, prev);
    if (e < OPA_TILE - 1) next = lpart[e + 1];
    else tl_load(a, x + 1, kk, jj, next);
    if (!verify) {
      if (prev != lp) pfirst[lp] = (uint32_t)x;
      if (next != lp) plast[lp] = (uint32_t)x;
    } else {
      const bool bad = (prev != lp && pfirst[lp] != (uint32_t)x) ||
                       (next != lp && plast[lp] != (uint32_t)x);
      if (bad) {
        contig[lp] = 0;
        nbad++;
      }
    }
  }
  return nbad;
}

#define OPA_DYN_LDS(T, name) extern __shared__ __align__(16) unsigned char name##_raw[]; \
  T *name = reinterpret_cast<T *>(name##_raw)

// Partition edges of every seq tile on their own (store, or verify).
__global__ void __launch_bounds__(256) k_part_edges(TlArgs a, uint32_t *pfirst, uint32_t *plast,
                                                    uint8_t *contig, opattr_diag *diag,
                                                    int verify) {
  __shared__ int32_t lpart[OPA_TILE];
  __shared__ uint32_t snc;
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  if (threadIdx.x == 0) snc = 0;
  for (int e = threadIdx.x; e < OPA_TILE; e += OPA_TILE_THREADS) {
    uint32_t k;
    int32_t j, lp;
    tl_load(a, base + e, k, j, lp);
    lpart[e] = lp;
  }
  __syncthreads();
  const uint32_t nb = part_edges(a, lpart, base, pfirst, plast, contig, verify != 0);
  if (nb) atomicAdd(&snc, nb);
  __syncthreads();
  if (threadIdx.x == 0 && snc) atomicOr(&diag->flags, OPATTR_F_PARTITION);
}

__global__ void __launch_bounds__(256) k_tl_hist_w(TlArgs a, uint32_t *tlh, uint32_t *pfirst,
                                                   uint32_t *plast, opattr_diag *diag,
                                                   int want_parts) {
  OPA_DYN_LDS(uint16_t, cnt);
  __shared__ int32_t lpart[OPA_TILE];
  __shared__ uint32_t sbad;
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  for (uint32_t i = threadIdx.x; i < 4 * NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  if (threadIdx.x == 0) sbad = 0;
  __syncthreads();
  uint32_t key[kWaveChunks], rank[kWaveChunks], bad = 0;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int e = tile_elem(c);
    int32_t j, lp;
    bad += tl_load(a, base + e, key[c], j, lp);
    lpart[e] = lp;
  }
  wave_rank<kWaveChunks>(key, NN, bits_for(NN), cnt + wave_id() * NN, rank);
  block_rank_bases(cnt, NN, tlh + tile * NN);
  if (want_parts) part_edges(a, lpart, base, pfirst, plast, nullptr, false);
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (threadIdx.x == 0 && sbad)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)sbad);
}

struct PfArgs {
  const uint32_t *name;
  int64_t P;
  uint32_t NN;
};

__device__ inline uint32_t pf_tile_keys(const PfArgs &a, int64_t base, uint32_t *A) {
  uint32_t bad = 0;
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int l = c * OPA_TILE_THREADS + threadIdx.x;
    const int64_t x = base + l;
    uint32_t n = a.NN;
    if (x < a.P) {
      n = a.name[x];
      if (n >= a.NN) {
        bad++;
        n = a.NN;
      }
    }
    A[l] = (n << OPA_SLOT_BITS) | (uint32_t)l;
  }
  return bad;
}

__global__ void __launch_bounds__(256) k_pf_hist(PfArgs a, uint32_t *pfh, opattr_diag *diag) {
  __shared__ TileSmem sm;
  const int64_t tile = blockIdx.x;
  if (threadIdx.x == 0) sm.bad = 0;
  __syncthreads();
  const uint32_t bad = pf_tile_keys(a, tile * OPA_TILE, sm.A);
  if (bad) atomicAdd(&sm.bad, bad);
  __syncthreads();
  if (threadIdx.x == 0 && sm.bad)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)sm.bad);
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(a.NN));
  write_hist_row(sm.A, a.NN, pfh + tile * a.NN);
}

// ---------------------------------------------------------------------------
// column scans of a [rows][cols] histogram table: exclusive prefix down each
// column, in place, plus the column totals
// ---------------------------------------------------------------------------
// rows_dev (optional): the actual row count, known only on the device
__device__ __forceinline__ int64_t rows_of(int64_t rows, const int64_t *rows_dev) {
  return rows_dev ? (*rows_dev < rows ? *rows_dev : rows) : rows;
}

__global__ void __launch_bounds__(256) k_colsum(const uint32_t *__restrict__ tab, int64_t rows,
                                                uint32_t cols, uint32_t *chs,
                                                const int64_t *rows_dev) {
  __shared__ uint32_t part[4][64];
  rows = rows_of(rows, rows_dev);
  const int l = lane_id(), w = wave_id();
  const uint32_t col = blockIdx.x * 64 + l;
  const int64_t r0 = (int64_t)blockIdx.y * kColChunk + w * (kColChunk / 4);
  if ((int64_t)blockIdx.y * kColChunk >= rows) return;
  uint32_t s = 0;
  if (col < cols)
    for (int i = 0; i < kColChunk / 4; ++i) {
      const int64_t r = r0 + i;
      if (r < rows) s += tab[r * cols + col];
    }
  part[w][l] = s;
  __syncthreads();
  if (w == 0 && col < cols)
    chs[(int64_t)blockIdx.y * cols + col] = part[0][l] + part[1][l] + part[2][l] + part[3][l];
}

__global__ void k_chunkscan(uint32_t *chs, int64_t nch, uint32_t cols, uint32_t *totals,
                            int64_t rows, const int64_t *rows_dev) {
  const uint32_t col = blockIdx.x * blockDim.x + threadIdx.x;
  if (col >= cols) return;
  rows = rows_of(rows, rows_dev);
  const int64_t nc = (rows + kColChunk - 1) / kColChunk;
  if (nc < nch) nch = nc;
  uint32_t run = 0;
  for (int64_t c = 0; c < nch; ++c) {
    const uint32_t v = chs[c * cols + col];
    chs[c * cols + col] = run;
    run += v;
  }
  totals[col] = run;
}

__global__ void __launch_bounds__(256) k_colbase(uint32_t *tab, int64_t rows, uint32_t cols,
                                                 const uint32_t *__restrict__ chs,
                                                 const int64_t *rows_dev) {
  __shared__ uint32_t part[4][64];
  rows = rows_of(rows, rows_dev);
  if ((int64_t)blockIdx.y * kColChunk >= rows) return;
  const int l = lane_id(), w = wave_id();
  const uint32_t col = blockIdx.x * 64 + l;
  const int64_t r0 = (int64_t)blockIdx.y * kColChunk + w * (kColChunk / 4);
  uint32_t v[kColChunk / 4];
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < kColChunk / 4; ++i) {
    const int64_t r = r0 + i;
    v[i] = (col < cols && r < rows) ? tab[r * cols + col] : 0u;
    s += v[i];
  }
  part[w][l] = s;
  __syncthreads();
  if (col >= cols) return;
  uint32_t run = chs[(int64_t)blockIdx.y * cols + col];
  for (int ww = 0; ww < w; ++ww) run += part[ww][l];
#pragma unroll
  for (int i = 0; i < kColChunk / 4; ++i) {
    const int64_t r = r0 + i;
    if (r < rows) tab[r * cols + col] = run;
    run += v[i];
  }
}

void column_scan(uint32_t *tab, int64_t rows, uint32_t cols, uint32_t *chs, uint32_t *totals,
                 hipStream_t s, const int64_t *rows_dev) {
  if (rows <= 0 || cols == 0) return;
  const int64_t nch = (rows + kColChunk - 1) / kColChunk;
  dim3 g((cols + 63) / 64, (unsigned)nch);
  k_colsum<<<g, 256, 0, s>>>(tab, rows, cols, chs, rows_dev);
  k_chunkscan<<<(cols + 255) / 256, 256, 0, s>>>(chs, nch, cols, totals, rows, rows_dev);
  k_colbase<<<g, 256, 0, s>>>(tab, rows, cols, chs, rows_dev);
}

// off[n] = rows of names before n; count validation (Sec. 3.3)
__global__ void __launch_bounds__(1024) k_names(const uint32_t *__restrict__ tlc,
                                                const uint32_t *__restrict__ pfc, uint32_t NN,
                                                uint32_t *off, uint32_t *name_counts,
                                                opattr_diag *diag, int strict) {
  __shared__ uint32_t sh[16];
  __shared__ unsigned long long red[3][16];
  uint32_t carry = 0;
  unsigned long long mism = 0, tlu = 0, pfu = 0;
  for (uint32_t base = 0; base < NN; base += 1024) {
    const uint32_t n = base + threadIdx.x;
    const uint32_t tl = n < NN ? tlc[n] : 0u, pf = n < NN ? pfc[n] : 0u;
    uint32_t tot;
    const uint32_t pre = block_excl_scan_add<uint32_t>(pf, sh, &tot);
    if (n < NN) {
      off[n] = carry + pre;
      if (name_counts) {
        name_counts[2 * (size_t)n] = tl;
        name_counts[2 * (size_t)n + 1] = pf;
      }
      if (tl != pf) {
        mism++;
        if (tl > pf) tlu += tl - pf;
        else pfu += pf - tl;
      }
    }
    carry += tot;
  }
  mism = wave_reduce_add(mism);
  tlu = wave_reduce_add(tlu);
  pfu = wave_reduce_add(pfu);
  if (lane_id() == 0) {
    red[0][wave_id()] = mism;
    red[1][wave_id()] = tlu;
    red[2][wave_id()] = pfu;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long a = 0, b = 0, c = 0;
    for (int i = 0; i < 16; ++i) {
      a += red[0][i];
      b += red[1][i];
      c += red[2][i];
    }
    if (a) {
      atomicAdd(&diag->names_mismatched, (uint32_t)a);
      atomicOr(&diag->flags, OPATTR_F_COUNT);
    }
    if (b) atomicAdd((unsigned long long *)&diag->tl_unmatched, b);
    if (c) atomicAdd((unsigned long long *)&diag->pf_unmatched, c);
    if (strict) diag->strict = 1u;
  }
}

// slot[off[n] + r] = index of the r-th profiled row of name n
__global__ void __launch_bounds__(256) k_pf_slot(PfArgs a, const uint32_t *__restrict__ pfh,
                                                 const uint32_t *__restrict__ off, int32_t *slot) {
  __shared__ TileSmem sm;
  const int64_t tile = blockIdx.x;
  const int64_t base = tile * OPA_TILE;
  pf_tile_keys(a, base, sm.A);
  __syncthreads();
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(a.NN));
  const uint32_t *row = pfh + tile * a.NN;
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int p = c * OPA_TILE_THREADS + threadIdx.x;
    const uint32_t key = sm.A[p];
    const uint32_t n = key >> OPA_SLOT_BITS;
    if (n < a.NN) {
      const int lo = lds_lower_bound(sm.A, OPA_TILE, n << OPA_SLOT_BITS);
      const uint32_t rank = row[n] + (uint32_t)(p - lo);
      slot[off[n] + rank] = (int32_t)(base + (key & (OPA_TILE - 1)));
    }
  }
}

__global__ void __launch_bounds__(256) k_pf_hist_w(PfArgs a, uint32_t *pfh, opattr_diag *diag) {
  OPA_DYN_LDS(uint16_t, cnt);
  __shared__ uint32_t sbad;
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  for (uint32_t i = threadIdx.x; i < 4 * NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  if (threadIdx.x == 0) sbad = 0;
  __syncthreads();
  uint32_t key[kWaveChunks], rank[kWaveChunks], bad = 0;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int64_t x = base + tile_elem(c);
    uint32_t n = NN;
    if (x < a.P) {
      n = a.name[x];
      if (n >= NN) {
        bad++;
        n = NN;
      }
    }
    key[c] = n;
  }
  wave_rank<kWaveChunks>(key, NN, bits_for(NN), cnt + wave_id() * NN, rank);
  block_rank_bases(cnt, NN, pfh + tile * NN);
  if (bad) atomicAdd(&sbad, bad);
  __syncthreads();
  if (threadIdx.x == 0 && sbad)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)sbad);
}

__global__ void __launch_bounds__(256) k_pf_slot_w(PfArgs a, const uint32_t *__restrict__ pfh,
                                                   const uint32_t *__restrict__ off,
                                                   int32_t *slot) {
  OPA_DYN_LDS(uint16_t, cnt);
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  for (uint32_t i = threadIdx.x; i < 4 * NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  __syncthreads();
  uint32_t key[kWaveChunks], rank[kWaveChunks];
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int64_t x = base + tile_elem(c);
    uint32_t n = NN;
    if (x < a.P) {
      n = a.name[x];
      if (n >= NN) n = NN;
    }
    key[c] = n;
  }
  wave_rank<kWaveChunks>(key, NN, bits_for(NN), cnt + wave_id() * NN, rank);
  block_rank_bases(cnt, NN, nullptr);
  const uint32_t *row = pfh + tile * NN;
  const uint16_t *wb = cnt + wave_id() * NN;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const uint32_t n = key[c];
    if (n < NN) {
      const int64_t x = base + tile_elem(c);
      slot[off[n] + row[n] + wb[n] + rank[c]] = (int32_t)x;
    }
  }
}

struct MatchArgs {
  const uint32_t *tlh, *tlc, *pfc, *off;
  const int32_t *slot;
  int32_t *match;
  int32_t *mbs;   // match of dedup-source launches by seq rank (NULL: off)
  uint32_t *nbs;  // their names
  int skip_name;
};

__global__ void __launch_bounds__(256) k_tl_match(TlArgs a, MatchArgs m) {
  __shared__ TileSmem sm;
  __shared__ int32_t jidx[OPA_TILE];
  const int64_t tile = blockIdx.x;
  const int64_t base = tile * OPA_TILE;
  tl_tile_keys(a, base, sm.A, nullptr, jidx);
  __syncthreads();
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(a.NN));
  const uint32_t *row = m.tlh + tile * a.NN;
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int p = c * OPA_TILE_THREADS + threadIdx.x;
    const uint32_t key = sm.A[p];
    const uint32_t n = key >> OPA_SLOT_BITS;
    const int l = (int)(key & (OPA_TILE - 1));
    const int32_t j = jidx[l];
    if (j < 0) continue;
    if (n < a.NN) {
      const int lo = lds_lower_bound(sm.A, OPA_TILE, n << OPA_SLOT_BITS);
      const uint32_t rank = row[n] + (uint32_t)(p - lo);
      const uint32_t rows = m.pfc[n];
      int32_t mt = rank < rows ? m.slot[m.off[n] + rank] : -1;
      if (m.skip_name && m.tlc[n] != rows) mt = -1;
      m.match[j] = mt;
      if (m.mbs && a.part[j] >= 0) {
        m.mbs[base + l] = mt;
        m.nbs[base + l] = n;
      }
    } else {
      m.match[j] = -1;
    }
  }
}

__global__ void __launch_bounds__(256) k_tl_match_w(TlArgs a, MatchArgs m, const uint32_t *pfirst,
                                                    const uint32_t *plast, uint8_t *contig,
                                                    opattr_diag *diag, int want_parts) {
  OPA_DYN_LDS(uint16_t, cnt);
  __shared__ int32_t lpart[OPA_TILE];
  __shared__ uint32_t snc;
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  for (uint32_t i = threadIdx.x; i < 4 * NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  if (threadIdx.x == 0) snc = 0;
  __syncthreads();
  uint32_t key[kWaveChunks], rank[kWaveChunks];
  int32_t jj[kWaveChunks];
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int e = tile_elem(c);
    int32_t lp;
    tl_load(a, base + e, key[c], jj[c], lp);
    lpart[e] = lp;
  }
  wave_rank<kWaveChunks>(key, NN, bits_for(NN), cnt + wave_id() * NN, rank);
  block_rank_bases(cnt, NN, nullptr);
  const uint32_t *row = m.tlh + tile * NN;
  const uint16_t *wb = cnt + wave_id() * NN;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int32_t j = jj[c];
    if (j < 0) continue;
    const uint32_t n = key[c];
    int32_t mt = -1;
    if (n < NN) {
      const uint32_t r = row[n] + wb[n] + rank[c];
      const uint32_t rows = m.pfc[n];
      mt = r < rows ? m.slot[m.off[n] + r] : -1;
      if (m.skip_name && m.tlc[n] != rows) mt = -1;
      const int e = tile_elem(c);
      if (m.mbs && lpart[e] >= 0) {
        m.mbs[base + e] = mt;
        m.nbs[base + e] = n;
      }
    }
    m.match[j] = mt;
  }
  if (want_parts) {
    const uint32_t nb = part_edges(a, lpart, base, const_cast<uint32_t *>(pfirst),
                                   const_cast<uint32_t *>(plast), contig, true);
    if (nb) atomicAdd(&snc, nb);
    __syncthreads();
    if (threadIdx.x == 0 && snc) atomicOr(&diag->flags, OPATTR_F_PARTITION);
  }
}

// bad class-map entries are counted once, with the other bad ids of the match
__global__ void k_rep_check(const int32_t *__restrict__ part_rep, uint32_t NP, opattr_diag *diag) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  const bool bad = q < NP && (part_rep[q] < 0 || (uint32_t)part_rep[q] >= NP);
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)__popcll(m));
}

static TlArgs tl_args(const opattr_kernels *k, const opattr_dims *d, void *ws, const Plan &pl,
                      bool dedup) {
  TlArgs a;
  a.sv = at<int32_t>(ws, pl.sv);
  a.T = pl.T;
  a.name = k->name_id;
  a.part = dedup ? k->part_id : nullptr;
  a.part_rep = dedup ? d->part_rep : nullptr;
  a.NN = d->n_names;
  a.NP = dedup ? d->n_parts : 0;
  return a;
}

static bool has_dedup(const opattr_kernels *k, const opattr_dims *d) {
  return k->part_id && d->part_rep && d->n_parts > 0;
}

void run_match(const IomArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const opattr_kernels *k = x.k;
  const opattr_dims *d = x.d;
  void *ws = x.ws;
  const uint32_t NN = d->n_names;
  const bool dedup = has_dedup(k, d);
  const bool parts = dedup && x.want_dedup;
  const bool fast = NN <= kFastNames, fast_pf = NN <= kFastKeys;
  const size_t lds = (size_t)4 * NN * sizeof(uint16_t);
  uint32_t *tlh = at<uint32_t>(ws, pl.tlh), *pfh = at<uint32_t>(ws, pl.pfh);
  uint32_t *tlc = at<uint32_t>(ws, pl.tlc), *pfc = at<uint32_t>(ws, pl.pfc);
  uint32_t *off = at<uint32_t>(ws, pl.off);
  uint32_t *pfirst = at<uint32_t>(ws, pl.pfirst), *plast = at<uint32_t>(ws, pl.plast);
  uint8_t *contig = at<uint8_t>(ws, pl.contig);
  fill_u32(tlc, 0, NN, s);
  fill_u32(pfc, 0, NN, s);
  if (parts) {
    fill_u32(pfirst, 0xFFFFFFFFu, pl.NP, s);
    fill_u32(plast, 0xFFFFFFFFu, pl.NP, s);
    fill_u8(contig, 1, pl.NP, s);
  }
  if (dedup) k_rep_check<<<(d->n_parts + 255) / 256, 256, 0, s>>>(d->part_rep, d->n_parts, x.diag);
  const TlArgs ta = tl_args(k, d, ws, pl, dedup);
  PfArgs pa;
  pa.name = x.p->name_id;
  pa.P = pl.P;
  pa.NN = NN;
  probe_begin(OPATTR_PROBE_TL_HIST, s);
  if (pl.nt > 0) {
    if (fast) {
      k_tl_hist_w<<<(unsigned)pl.nt, 256, lds, s>>>(ta, tlh, pfirst, plast, x.diag, parts ? 1 : 0);
    } else {
      k_tl_hist<<<(unsigned)pl.nt, 256, 0, s>>>(ta, tlh, x.diag);
      if (parts)
        k_part_edges<<<(unsigned)pl.nt, 256, 0, s>>>(ta, pfirst, plast, contig, x.diag, 0);
    }
  }
  probe_end(OPATTR_PROBE_TL_HIST, s);
  probe_begin(OPATTR_PROBE_PF_HIST, s);
  if (pl.ntp > 0) {
    if (fast_pf) k_pf_hist_w<<<(unsigned)pl.ntp, 256, lds, s>>>(pa, pfh, x.diag);
    else k_pf_hist<<<(unsigned)pl.ntp, 256, 0, s>>>(pa, pfh, x.diag);
  }
  probe_end(OPATTR_PROBE_PF_HIST, s);
  probe_begin(OPATTR_PROBE_COL_SCAN, s);
  column_scan(tlh, pl.nt, NN, at<uint32_t>(ws, pl.tlch), tlc, s, nullptr);
  column_scan(pfh, pl.ntp, NN, at<uint32_t>(ws, pl.pfch), pfc, s, nullptr);
  if (NN)
    k_names<<<1, 1024, 0, s>>>(tlc, pfc, NN, off, x.name_counts, x.diag,
                               x.policy == OPATTR_MISMATCH_STRICT ? 1 : 0);
  probe_end(OPATTR_PROBE_COL_SCAN, s);
  probe_begin(OPATTR_PROBE_PF_SLOT, s);
  if (pl.ntp > 0) {
    if (fast_pf) k_pf_slot_w<<<(unsigned)pl.ntp, 256, lds, s>>>(pa, pfh, off, at<int32_t>(ws, pl.slot));
    else k_pf_slot<<<(unsigned)pl.ntp, 256, 0, s>>>(pa, pfh, off, at<int32_t>(ws, pl.slot));
  }
  probe_end(OPATTR_PROBE_PF_SLOT, s);
  MatchArgs ma;
  ma.tlh = tlh;
  ma.tlc = tlc;
  ma.pfc = pfc;
  ma.off = off;
  ma.slot = at<int32_t>(ws, pl.slot);
  ma.match = x.match;
  ma.mbs = parts ? at<int32_t>(ws, pl.mbs) : nullptr;
  ma.nbs = parts ? at<uint32_t>(ws, pl.nbs) : nullptr;
  ma.skip_name = x.policy == OPATTR_MISMATCH_SKIP_NAME ? 1 : 0;
  probe_begin(OPATTR_PROBE_TL_MATCH, s);
  if (pl.nt > 0) {
    if (fast) {
      k_tl_match_w<<<(unsigned)pl.nt, 256, lds, s>>>(ta, ma, pfirst, plast, contig, x.diag,
                                                     parts ? 1 : 0);
    } else {
      k_tl_match<<<(unsigned)pl.nt, 256, 0, s>>>(ta, ma);
      if (parts)
        k_part_edges<<<(unsigned)pl.nt, 256, 0, s>>>(ta, pfirst, plast, contig, x.diag, 1);
    }
  }
  probe_end(OPATTR_PROBE_TL_MATCH, s);
}

// ---------------------------------------------------------------------------
// layer dedup
// ---------------------------------------------------------------------------
struct DedupArgs {
  int64_t T;
  const uint32_t *seq;
  const int32_t *rk;  // NULL when seq is dense
  const uint32_t *name;
  const int32_t *part;
  const int32_t *part_rep;
  uint32_t NN, NP;
  const uint32_t *pfirst, *plast;
  const uint8_t *contig;
  int32_t *mbs;
  uint32_t *nbs;
  int32_t *match;
  opattr_diag *diag;
};

__device__ __forceinline__ int64_t rank_of(const DedupArgs &a, int64_t i) {
  if (a.rk) return a.rk[i];
  const uint32_t s = a.seq[i];
  return (int64_t)s < a.T ? (int64_t)s : -1;
}

// dedup sources from a given match array (standalone broadcast call)
__global__ void k_src_fill(DedupArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.T) return;
  const int32_t pt = a.part[i];
  const uint32_t nm = a.name[i];
  if (pt < 0 || (uint32_t)pt >= a.NP || nm >= a.NN || a.part_rep[pt] != pt) return;
  const int64_t r = rank_of(a, i);
  if (r < 0) return;
  a.mbs[r] = a.match[i];
  a.nbs[r] = nm;
}

__global__ void k_dedup(DedupArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool err = false;
  if (i < a.T) {
    const int32_t pt = a.part[i];
    const uint32_t nm = a.name[i];
    if (pt >= 0 && (uint32_t)pt < a.NP && nm < a.NN) {
      const int32_t r = a.part_rep[pt];
      if (r >= 0 && (uint32_t)r < a.NP && r != pt) {
        // a duplicate: inherit from the representative's launch at the same
        // position of its partition
        const uint32_t f = a.pfirst[r];
        bool ok = a.contig[pt] && a.part_rep[r] == r && f != 0xFFFFFFFFu && a.contig[r];
        const int64_t rk = rank_of(a, i);
        ok = ok && rk >= 0;
        int32_t mt = -1;
        if (ok) {
          const uint32_t pos = (uint32_t)(rk - (int64_t)a.pfirst[pt]);
          ok = pos < a.plast[r] - f + 1u;
          if (ok) {
            const uint32_t src = f + pos;
            ok = a.nbs[src] == nm;
            if (ok) mt = a.mbs[src];
          }
        }
        a.match[i] = mt;
        err = !ok;
      }
    }
  }
  const uint64_t m = __ballot(err);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
    atomicAdd((unsigned long long *)&a.diag->dedup_errors, (unsigned long long)__popcll(m));
}

void run_dedup(const opattr_kernels *k, const opattr_dims *d, int32_t *match, opattr_diag *diag,
               void *ws, const Plan &pl, bool stats_ready, hipStream_t s) {
  if (!has_dedup(k, d) || pl.T <= 0) return;
  DedupArgs a;
  a.T = pl.T;
  a.seq = k->seq;
  a.rk = pl.seq_dense ? nullptr : at<int32_t>(ws, pl.rk);
  a.name = k->name_id;
  a.part = k->part_id;
  a.part_rep = d->part_rep;
  a.NN = d->n_names;
  a.NP = d->n_parts;
  uint32_t *pfirst = at<uint32_t>(ws, pl.pfirst), *plast = at<uint32_t>(ws, pl.plast);
  uint8_t *contig = at<uint8_t>(ws, pl.contig);
  a.pfirst = pfirst;
  a.plast = plast;
  a.contig = contig;
  a.mbs = at<int32_t>(ws, pl.mbs);
  a.nbs = at<uint32_t>(ws, pl.nbs);
  a.match = match;
  a.diag = diag;
  const unsigned nb = (unsigned)((pl.T + 255) / 256);
  probe_begin(OPATTR_PROBE_DEDUP, s);
  if (!stats_ready) {
    const TlArgs ta = tl_args(k, d, ws, pl, true);
    fill_u32(pfirst, 0xFFFFFFFFu, pl.NP, s);
    fill_u32(plast, 0xFFFFFFFFu, pl.NP, s);
    fill_u8(contig, 1, pl.NP, s);
    k_part_edges<<<(unsigned)pl.nt, 256, 0, s>>>(ta, pfirst, plast, contig, diag, 0);
    k_part_edges<<<(unsigned)pl.nt, 256, 0, s>>>(ta, pfirst, plast, contig, diag, 1);
    k_src_fill<<<nb, 256, 0, s>>>(a);
  }
  k_dedup<<<nb, 256, 0, s>>>(a);
  probe_end(OPATTR_PROBE_DEDUP, s);
}

}  // namespace opa
