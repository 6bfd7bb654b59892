// Invocation-order matching (Alg. 1) and layer dedup (Sec. 3.7) on the GPU.
//
// Alg. 1 walks the launches in order and hands the i-th launch of a name the
// i-th profiled row of that name. Written data-parallel: the rank of a launch
// among the eligible launches of its name (in seq order) is
//     rank = (launches of the name in earlier seq tiles) + (rank inside the tile)
// and the row is slot[off[name] + rank] when rank < rows(name). Seq tiles hold
// 4096 launches; per-tile name histograms are scanned down the columns for the
// cross-tile part. The profiled side is ranked the same way (tiles in replay
// order) to build the slot table.
//
// Fast path (at most 4096 names): a histogram kernel ranks every tile once
// with per-wave LDS counters and leaves each launch's in-tile rank and key by
// seq position; a lookup kernel then gives eligible launches their row and
// duplicates the row of the representative's launch at the same position of
// the representative partition. With more names an LDS radix sort ranks the
// tiles and a separate kernel broadcasts to duplicates.
//
// Seq tiles are read through a launch-order view (sv[seq] = input index), or,
// when the kernels are promised stream-major with dense seq, straight from one
// storage segment per stream (no view is built).
#include "common.h"
#include "impl.h"

namespace opa {

constexpr int kWaveChunks = OPA_TILE / OPA_TILE_THREADS;  // 16 chunks of 64 per wave
constexpr int kMaxSegStreams = OPA_WAVE;

// ---------------------------------------------------------------------------
// launch-order view: sv[rank] = input index of the launch with that rank
// ---------------------------------------------------------------------------
__global__ void k_seqview_dense(const uint32_t *__restrict__ seq, int64_t T, int32_t *sv,
                                opattr_diag *diag, int validate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= T) return;
  const uint32_t s = seq[i];
  const bool bad = (int64_t)s >= T && validate;
  if ((int64_t)s < T) sv[s] = (int32_t)i;
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1) {
    atomicAdd((unsigned long long *)&diag->order_violations, (unsigned long long)__popcll(m));
    atomicOr(&diag->flags, OPATTR_F_ORDER);
  }
}

// Under OPATTR_VALIDATE, after the scatter: a seq value that two launches
// hold keeps only one of them in the view, and the other finds itself
// missing there (no atomics: each launch reads its own slot back).
__global__ void k_seqview_check(const uint32_t *__restrict__ seq, int64_t T,
                                const int32_t *__restrict__ sv, opattr_diag *diag) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (i < T) {
    const uint32_t s = seq[i];
    bad = (int64_t)s < T && sv[s] != (int32_t)i;
  }
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1) {
    atomicAdd((unsigned long long *)&diag->order_violations, (unsigned long long)__popcll(m));
    atomicOr(&diag->flags, OPATTR_F_ORDER);
  }
}

__global__ void k_seqview_sorted(const uint32_t *__restrict__ keys, const uint32_t *__restrict__ vals,
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
  // the segment path reads tiles without the view (and checks the density
  // of seq in them)
  if (T <= 0 || pl.seg) return;
  int32_t *sv = at<int32_t>(ws, pl.sv);
  const unsigned nb = (unsigned)((T + 255) / 256);
  if (pl.seq_dense) {
    fill_u32(reinterpret_cast<uint32_t *>(sv), 0xFFFFFFFFu, T, s);  // positions no launch claims
    probe_begin(OPATTR_PROBE_SEQ_VIEW, s);
    k_seqview_dense<<<nb, 256, 0, s>>>(k->seq, T, sv, diag, validate ? 1 : 0);
    if (validate) k_seqview_check<<<nb, 256, 0, s>>>(k->seq, T, sv, diag);
    probe_end(OPATTR_PROBE_SEQ_VIEW, s);
    return;
  }
  probe_begin(OPATTR_PROBE_SEQ_VIEW, s);
  uint32_t *k0 = at<uint32_t>(ws, pl.seqsort_k0), *k1 = at<uint32_t>(ws, pl.seqsort_k1);
  uint32_t *v0 = at<uint32_t>(ws, pl.seqsort_v0), *v1 = at<uint32_t>(ws, pl.seqsort_v1);
  launch_key_pairs(k->seq, k0, v0, T, s);
  const bool in1 = radix_sort_pairs(k0, v0, k1, v1, T, 0, 32, at<uint32_t>(ws, pl.rs_hist), s);
  k_seqview_sorted<<<nb, 256, 0, s>>>(in1 ? k1 : k0, in1 ? v1 : v0, T, sv,
                                       at<int32_t>(ws, pl.rk), diag);
  probe_end(OPATTR_PROBE_SEQ_VIEW, s);
}

// ---------------------------------------------------------------------------
// tile elements
// ---------------------------------------------------------------------------
struct TlArgs {
  const int32_t *sv;
  int64_t T;
  const uint32_t *name;
  const int32_t *part;      // NULL when dedup is off
  const int32_t *part_rep;  // NULL when dedup is off
  uint32_t NN, NP;
  // segment path
  const uint32_t *seq;
  const uint32_t *bnd;  // [tiles + 1][NS]
  const int64_t *kblk;  // [NS + 1]
  uint32_t NS;
  opattr_diag *vdiag;   // under OPATTR_VALIDATE: the density check reports here (else NULL)
};

// Element e of a tile sits in wave e / 1024, chunk (e / 64) % 16, lane e % 64.
__device__ __forceinline__ int tile_elem(int c) {
  return wave_id() * (OPA_TILE / 4) + c * OPA_WAVE + lane_id();
}

// Ranking key of launch j (its name if eligible for replay -- no partition,
// or a partition that is its own class representative -- else NN) and
// partition (-1 none, -2 bad id). Returns 1 if an id is out of range.
__device__ __forceinline__ uint32_t tl_classify(const TlArgs &a, int64_t j, uint32_t &key,
                                                int32_t &lp) {
  key = a.NN;
  lp = -2;
  const uint32_t nm = a.name[j];
  const int32_t pt = a.part ? a.part[j] : -1;
  if (nm >= a.NN || pt < -1 || (pt >= 0 && (uint32_t)pt >= a.NP)) return 1;
  if (pt < 0 || a.part_rep[pt] == pt) key = nm;
  lp = pt;
  return 0;
}

// The launch of seq rank x through the view: input index j (-1 for holes),
// key and partition as above (NN and -2 for holes).
__device__ __forceinline__ uint32_t tl_load(const TlArgs &a, int64_t x, uint32_t &key, int32_t &j,
                                            int32_t &lp) {
  j = (x >= 0 && x < a.T) ? a.sv[x] : -1;
  key = a.NN;
  lp = -2;
  if (j < 0) return 0;
  return tl_classify(a, j, key, lp);
}

__device__ __forceinline__ int32_t tl_lp(const TlArgs &a, int64_t x) {
  uint32_t k;
  int32_t j, lp;
  tl_load(a, x, k, j, lp);
  return lp;
}

// Segment table of a seq tile (segment path) and the partitions of the
// launches just before and after the tile.
struct SegTable {
  uint32_t lo[kMaxSegStreams], pre[kMaxSegStreams + 1];
  int32_t edge[2];
};

// One seq tile in LDS, by position in the tile.
struct TileData {
  uint16_t key[OPA_TILE];  // ranking key (NN: not eligible, or no launch)
  int32_t lp[OPA_TILE];    // partition (-1 none, -2 no launch or bad id)
  SegTable sg;
  uint32_t bad;
  uint32_t occ[OPA_TILE / 32];  // density check: positions taken
  uint32_t placed, twice;       // density check: launches placed, on a taken position
};

// Fill TileData for seq tile t through the view. Ends with a barrier;
// returns this thread's bad-id count.
__device__ inline uint32_t view_tile(const TlArgs &a, int64_t t, TileData &sm) {
  const int64_t base = t * OPA_TILE;
  uint32_t bad = 0;
#pragma unroll 4
  for (int c = 0; c < kWaveChunks; ++c) {
    const int e = c * OPA_TILE_THREADS + threadIdx.x;
    uint32_t key;
    int32_t j, lp;
    bad += tl_load(a, base + e, key, j, lp);
    sm.key[e] = (uint16_t)key;
    sm.lp[e] = lp;
  }
  if (threadIdx.x == 0) sm.sg.edge[0] = tl_lp(a, base - 1);
  if (threadIdx.x == OPA_WAVE) sm.sg.edge[1] = tl_lp(a, base + OPA_TILE);
  __syncthreads();
  return bad;
}

// ---------------------------------------------------------------------------
// Segment path (kernels stream-major, seq dense): seq tile t holds, for every
// stream s, the storage range [bnd[t][s], bnd[t+1][s]) -- the launches of s
// whose seq falls in the tile -- so a tile is read with coalesced loads and no
// launch-order view is built. Every bound is clamped, so a broken promise
// gives wrong tiles, never an access out of bounds.
// ---------------------------------------------------------------------------

// bnd[t * NS + s] = first launch of stream s with seq >= t * 4096, t in [0, nt].
// Interpolation search (a stream's launches spread evenly over seq in
// practice), alternating with bisection so that a skewed stream still takes
// at most about twice the steps of a binary search.
__global__ void k_tile_bounds(const uint32_t *__restrict__ seq, const int64_t *__restrict__ kblk,
                              uint32_t NS, int64_t nt, uint32_t *bnd) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (nt + 1) * NS) return;
  const int64_t t = id / NS;
  const uint32_t s = (uint32_t)(id - t * NS);
  const int64_t lo = kblk[s], hi = kblk[s + 1];
  const uint64_t x = (uint64_t)t * OPA_TILE;
  int64_t ans;
  if (lo >= hi) {
    ans = lo;
  } else {
    int64_t a = lo, b = hi - 1;
    uint64_t va = seq[a], vb = seq[b];
    if (va >= x) {
      ans = lo;
    } else if (vb < x) {
      ans = hi;
    } else {
      // seq[a] < x <= seq[b]
      bool interp = true;
      while (b - a > 1) {
        int64_t m;
        if (interp && vb > va) {
          const uint64_t off = (x - va) * (uint64_t)(b - a) / (vb - va);
          m = a + (int64_t)off;
          if (m <= a) m = a + 1;
          if (m >= b) m = b - 1;
        } else {
          m = a + ((b - a) >> 1);
        }
        interp = !interp;
        const uint64_t vm = seq[m];
        if (vm < x) {
          a = m;
          va = vm;
        } else {
          b = m;
          vb = vm;
        }
      }
      ans = b;
    }
  }
  bnd[id] = (uint32_t)ans;
}

// Segment table of tile t in sm.lo / sm.pre (wave 0; the caller
// synchronises).
__device__ inline void seg_table(const TlArgs &a, int64_t t, SegTable &sm) {
  const int ln = lane_id();
  const uint64_t T = (uint64_t)a.T;
  if (wave_id() != 0) return;
  uint32_t lo = 0, len = 0;
  if ((uint32_t)ln < a.NS) {
    uint64_t l = a.bnd[t * a.NS + ln], h = a.bnd[(t + 1) * a.NS + ln];
    l = l < T ? l : T;
    h = h < T ? h : T;
    lo = (uint32_t)l;
    len = h > l ? (uint32_t)(h - l) : 0u;
    len = len < OPA_TILE ? len : OPA_TILE;
  }
  const uint32_t inc = wave_incl_scan_add(len);
  sm.lo[ln] = lo;
  sm.pre[ln] = inc - len;
  if (ln == OPA_WAVE - 1) sm.pre[OPA_WAVE] = inc;
}

// The launches with seq base - 1 (wave 1) and base + 4096 (wave 2) are the
// last launch before, or the first launch of, some stream's segment. Lane s
// of those waves holds its stream's candidate (or -1); the caller loads the
// candidate's ids with the tile's own loads and keeps the first candidate
// whose seq matches.
__device__ __forceinline__ int64_t edge_candidate(const TlArgs &a, int64_t t) {
  const int ln = lane_id(), w = wave_id();
  if (w != 1 && w != 2) return -1;
  const int64_t base = t * OPA_TILE;
  const uint64_t T = (uint64_t)a.T;
  const int side = w - 1;
  const uint64_t want = side ? (uint64_t)base + OPA_TILE : (uint64_t)base - 1;
  int64_t c = -1;
  if ((uint32_t)ln < a.NS && (side ? want < T : base > 0)) {
    const int64_t b = a.bnd[(t + side) * a.NS + ln];
    const int64_t s0 = a.kblk[ln], s1 = a.kblk[ln + 1];
    c = side ? b : b - 1;
    if (c < s0 || c >= s1 || c < 0 || (uint64_t)c >= T) c = -1;
  }
  return c;
}

// Input index of each of the thread's elements c * 256 + tid of tile t's
// segment order (or -1). They ascend by 256, so their segment only moves
// forward: a step per segment boundary passed instead of a search for each.
template <int kN>
__device__ __forceinline__ void seg_elems(const SegTable &sm, int64_t T, int32_t (&ii)[kN]) {
  const uint32_t total = sm.pre[OPA_WAVE] < OPA_TILE ? sm.pre[OPA_WAVE] : OPA_TILE;
  int sgi = 0;  // last segment with pre <= e
#pragma unroll
  for (int c = 0; c < kN; ++c) {
    const uint32_t e = (uint32_t)(c * OPA_TILE_THREADS + threadIdx.x);
    ii[c] = -1;
    if (e < total) {
      while (sgi < OPA_WAVE - 1 && sm.pre[sgi + 1] <= e) ++sgi;
      const int64_t i = (int64_t)sm.lo[sgi] + (e - sm.pre[sgi]);
      ii[c] = i < T ? (int32_t)i : -1;
    }
  }
}

// Fill TileData for seq tile t from its segments. Ends with a barrier. The
// loads come in two batches for all elements at once: seq rank, name and
// partition; then the partitions' class representatives.
__device__ inline uint32_t seg_tile(const TlArgs &a, int64_t t, TileData &sm) {
  const int tid = threadIdx.x;
  const int64_t base = t * OPA_TILE;
  for (int x = tid; x < OPA_TILE; x += OPA_TILE_THREADS) {
    sm.key[x] = (uint16_t)a.NN;
    sm.lp[x] = -2;
  }
  if (a.vdiag) {
    for (int x = tid; x < OPA_TILE / 32; x += OPA_TILE_THREADS) sm.occ[x] = 0;
    if (tid == 0) sm.placed = sm.twice = 0;
  }
  seg_table(a, t, sm.sg);
  const int64_t ec = edge_candidate(a, t);
  __syncthreads();
  int32_t ii[kWaveChunks];
  uint32_t sq[kWaveChunks], nm[kWaveChunks];
  int32_t pt[kWaveChunks];
  seg_elems<kWaveChunks>(sm.sg, a.T, ii);
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    sq[c] = ii[c] >= 0 ? a.seq[ii[c]] : 0u;
    nm[c] = ii[c] >= 0 ? a.name[ii[c]] : a.NN;
    pt[c] = (ii[c] >= 0 && a.part) ? a.part[ii[c]] : -1;
  }
  uint64_t esq = 0;
  uint32_t enm = a.NN;
  int32_t ept = -2;
  if (ec >= 0) {
    esq = a.seq[ec];
    enm = a.name[ec];
    ept = a.part ? a.part[ec] : -1;
  }
  // class representatives, and the key / partition of every element
  uint32_t bad = 0;
  int32_t rp[kWaveChunks];
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const bool ok = nm[c] < a.NN && pt[c] >= -1 && (pt[c] < 0 || (uint32_t)pt[c] < a.NP);
    rp[c] = (ii[c] >= 0 && ok && pt[c] >= 0) ? a.part_rep[pt[c]] : -1;
  }
  const bool eok = enm < a.NN && ept >= -1 && (ept < 0 || (uint32_t)ept < a.NP);
  uint32_t placed = 0, twice = 0;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    if (ii[c] < 0) continue;
    const int64_t x = (int64_t)sq[c] - base;
    if (x < 0 || x >= OPA_TILE || base + x >= a.T) continue;  // a broken promise: left out
    if (a.vdiag) {
      placed++;
      const uint32_t bit = 1u << (x & 31);
      if (atomicOr(&sm.occ[x >> 5], bit) & bit) twice++;
    }
    const bool ok = nm[c] < a.NN && pt[c] >= -1 && (pt[c] < 0 || (uint32_t)pt[c] < a.NP);
    if (!ok) {
      bad++;
      continue;
    }
    sm.key[x] = (uint16_t)((pt[c] < 0 || rp[c] == pt[c]) ? nm[c] : a.NN);
    sm.lp[x] = pt[c];
  }
  // edges: the first stream whose candidate has the wanted seq rank
  const int w = wave_id();
  if (w == 1 || w == 2) {
    const int side = w - 1;
    const uint64_t want = side ? (uint64_t)base + OPA_TILE : (uint64_t)base - 1;
    const uint64_t m = __ballot(ec >= 0 && esq == want);
    const int src = m ? __ffsll((unsigned long long)m) - 1 : 0;
    const int32_t lp = eok ? ept : -2;
    const int32_t got = __shfl(lp, src, OPA_WAVE);
    if (lane_id() == 0) sm.sg.edge[side] = m ? got : -2;
  }
  if (a.vdiag) {
    placed = (uint32_t)wave_reduce_add((unsigned long long)placed);
    twice = (uint32_t)wave_reduce_add((unsigned long long)twice);
    if (lane_id() == 0 && (placed || twice)) {
      atomicAdd(&sm.placed, placed);
      atomicAdd(&sm.twice, twice);
    }
  }
  __syncthreads();
  // Density (under OPATTR_VALIDATE): with seq sorted on every stream (checked
  // on its own), the tiles take each launch at most once, so seq is a
  // permutation of [0, n) exactly when every tile's positions are each taken
  // once. Counted: launches on a taken position, plus positions left free.
  if (a.vdiag && tid == 0) {
    const int64_t len = a.T - base < OPA_TILE ? a.T - base : OPA_TILE;
    const int64_t fresh = (int64_t)sm.placed - sm.twice;
    const uint64_t v = (uint64_t)sm.twice + (uint64_t)(len - fresh);
    if (v) {
      atomicAdd((unsigned long long *)&a.vdiag->order_violations, (unsigned long long)v);
      atomicOr(&a.vdiag->flags, OPATTR_F_ORDER);
    }
  }
  return bad;
}

// ---------------------------------------------------------------------------
// Partition edges. A head (first launch of a maximal run of one partition in
// seq order) stores its rank in pfirst and counts itself in pheads, a tail
// stores its rank in plast. A partition is one contiguous run exactly when it
// has one head, and then [pfirst, plast] is that run.
// ---------------------------------------------------------------------------
__device__ inline void part_edges(const int32_t *lpart, int64_t base, int32_t lp_before,
                                  int32_t lp_after, uint32_t *pfirst, uint32_t *plast,
                                  uint32_t *pheads) {
  for (int e = threadIdx.x; e < OPA_TILE; e += OPA_TILE_THREADS) {
    const int32_t lp = lpart[e];
    if (lp < 0) continue;
    const int64_t x = base + e;
    const int32_t prev = e > 0 ? lpart[e - 1] : lp_before;
    const int32_t next = e < OPA_TILE - 1 ? lpart[e + 1] : lp_after;
    if (prev != lp) {
      pfirst[lp] = (uint32_t)x;
      atomicAdd(&pheads[lp], 1u);
    }
    if (next != lp) plast[lp] = (uint32_t)x;
  }
}

// partition edges of every seq tile on their own (view path)
__global__ void __launch_bounds__(256) k_part_edges(TlArgs a, uint32_t *pfirst, uint32_t *plast,
                                                    uint32_t *pheads) {
  __shared__ TileData sm;
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  view_tile(a, blockIdx.x, sm);
  part_edges(sm.lp, base, sm.sg.edge[0], sm.sg.edge[1], pfirst, plast, pheads);
}

// The record of every partition (PartRec, see impl.h); also raises
// PARTITION for every partition seen in more than one run.

__global__ void k_part_prep(const int32_t *__restrict__ part_rep, uint32_t NP,
                            const uint32_t *__restrict__ pfirst, const uint32_t *__restrict__ plast,
                            const uint32_t *__restrict__ pheads, PartRec *prec,
                            opattr_diag *diag) {
  const uint32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  bool nc = false;
  if (p < NP) {
    nc = pheads[p] > 1;
    if (prec) {
      const int32_t r = part_rep[p];
      PartRec q{0, kRecNone};
      if (r == (int32_t)p) {
        q.hi = kRecEligible;
      } else if (r >= 0 && (uint32_t)r < NP) {
        q.hi = 0;
        const uint32_t f = pfirst[r];
        if (pheads[p] == 1u && pheads[r] == 1u && part_rep[r] == r && f != 0xFFFFFFFFu) {
          q.delta = (int32_t)(f - pfirst[p]);
          const uint64_t hi = (uint64_t)pfirst[p] + (plast[r] - f + 1u);
          q.hi = (uint32_t)(hi < 0x7FFFFFFFull ? hi : 0x7FFFFFFFull);  // seq ranks are < 2^31
        }
      }
      prec[p] = q;
    }
  }
  if (__ballot(nc) && lane_id() == 0) atomicOr(&diag->flags, OPATTR_F_PARTITION);
}

// bad class-map entries are counted once, with the other bad ids of the match
__global__ void k_rep_check(const int32_t *__restrict__ part_rep, uint32_t NP, opattr_diag *diag) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  const bool bad = q < NP && (part_rep[q] < 0 || (uint32_t)part_rep[q] >= NP);
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)__popcll(m));
}

// The matching's first launch on the segment path, three jobs in one grid
// by block ranges: [0, nf) the clears (fill jobs), [nf, nf + nr) the class
// map's range check, then one wave per stream s = 0..NS for the storage
// block of the stream (kblk).
struct ProArgs {
  FillJobs fill;
  int nf, nr;
  const int32_t *part_rep;  // the class map (nr = 0: none)
  uint32_t NP;
  opattr_diag *diag;
  const uint16_t *st;
  int64_t T;
  uint32_t NS;
  int64_t *kblk;
};

__global__ void __launch_bounds__(256) k_seg_prologue(ProArgs a) {
  const int b = blockIdx.x;
  if (b < a.nf) {
    const int64_t stride = (int64_t)a.nf * blockDim.x;
    for (int q = 0; q < a.fill.count; ++q)
      for (int64_t i = (int64_t)b * blockDim.x + threadIdx.x; i < a.fill.n[q]; i += stride)
        a.fill.p[q][i] = a.fill.v[q];
  } else if (b < a.nf + a.nr) {
    const uint32_t q = (uint32_t)(b - a.nf) * blockDim.x + threadIdx.x;
    const bool bad = q < a.NP && (a.part_rep[q] < 0 || (uint32_t)a.part_rep[q] >= a.NP);
    const uint64_t m = __ballot(bad);
    if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
      atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)__popcll(m));
  } else {
    const uint32_t sw = (uint32_t)(b - a.nf - a.nr) * (blockDim.x / OPA_WAVE) + wave_id();
    if (sw <= a.NS) stream_block_wave(a.st, a.T, sw, a.kblk);
  }
}

#define OPA_DYN_LDS(T, name) extern __shared__ __align__(16) unsigned char name##_raw[]; \
  T *name = reinterpret_cast<T *>(name##_raw)

// ---------------------------------------------------------------------------
// Fast path, histogram kernel: per seq tile, the per-name counts of eligible
// launches (tlh row), each launch's key and in-tile rank by seq position
// (kr = key << 16 | rank), and the partition edges.
// ---------------------------------------------------------------------------
struct HistOut {
  uint32_t *tlh;
  uint32_t *kr;
  uint32_t *pfirst, *plast, *pheads;  // pheads NULL: no partitions
  opattr_diag *diag;
};

template <bool SEG>
__global__ void __launch_bounds__(256) k_tl_hist_w(TlArgs a, HistOut o) {
  OPA_DYN_LDS(uint16_t, cnt);
  __shared__ TileData sm;
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  for (uint32_t i = threadIdx.x; i < 4 * NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  if (threadIdx.x == 0) sm.bad = 0;
  const uint32_t bad = SEG ? seg_tile(a, tile, sm) : view_tile(a, tile, sm);
  uint32_t key[kWaveChunks], rank[kWaveChunks];
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) key[c] = sm.key[tile_elem(c)];
  wave_rank<kWaveChunks>(key, NN, bits_for(NN), cnt + wave_id() * NN, rank);
  block_rank_bases(cnt, NN, o.tlh + tile * NN);
  const uint16_t *wb = cnt + wave_id() * NN;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int e = tile_elem(c);
    if (base + e >= a.T) continue;
    const uint32_t r = key[c] < NN ? (uint32_t)(wb[key[c]] + rank[c]) : 0u;
    o.kr[base + e] = (key[c] << 16) | r;
  }
  if (o.pheads) part_edges(sm.lp, base, sm.sg.edge[0], sm.sg.edge[1], o.pfirst, o.plast, o.pheads);
  if (bad) atomicAdd(&sm.bad, bad);
  __syncthreads();
  if (threadIdx.x == 0 && sm.bad)
    atomicAdd((unsigned long long *)&o.diag->bad_records, (unsigned long long)sm.bad);
}

// ---------------------------------------------------------------------------
// Fast path, lookup kernel: every launch of a seq tile gets its match.
// Eligible: slot[off[n] + rank] with rank = (tile prefix) + (in-tile rank).
// Duplicate (partition p with class representative r != p): the launch at
// the same position of r, if both partitions are one run each and the names
// agree, lends its rank (the rank decides the row, so the source's match need
// not exist yet); otherwise -1 and a dedup error.
// ---------------------------------------------------------------------------
struct LookArgs {
  const uint32_t *tlh;  // exclusive prefix of each name down the tiles
  const uint32_t *tlc, *pfc, *off;
  const int32_t *slot;
  const uint32_t *kr;   // key << 16 | in-tile rank, by seq rank
  const PartRec *prec;  // NULL: no dedup broadcast (duplicates get -1)
  int32_t *match;
  int skip_name;
  opattr_diag *diag;
};

// Loads come in batches for all of a thread's elements at once: ids; the
// partition record; the source launch's key and in-tile rank, the name's
// prefix in the source tile and the name's rows; the row itself.
template <bool SEG>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
k_tl_look(TlArgs a, LookArgs m) {
  __shared__ SegTable sm;
  __shared__ int32_t sii[OPA_TILE];  // input index of each element (kept out of registers)
  __shared__ unsigned long long serr;
  const int tid = threadIdx.x;
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  constexpr uint32_t kNone = 0xFFFFFFFFu;
  if (tid == 0) serr = 0;
  if (SEG) seg_table(a, tile, sm);
  __syncthreads();
  // batch 1: input index, seq rank, name and partition of each element
  int32_t ii[kWaveChunks];
  uint32_t xs[kWaveChunks], nm[kWaveChunks];
  int32_t pt[kWaveChunks];
  if (SEG) {
    seg_elems<kWaveChunks>(sm, a.T, ii);
  } else {
#pragma unroll
    for (int c = 0; c < kWaveChunks; ++c) {
      const uint32_t e = (uint32_t)(c * OPA_TILE_THREADS + tid);
      ii[c] = base + e < a.T ? a.sv[base + e] : -1;
    }
  }
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const uint32_t e = (uint32_t)(c * OPA_TILE_THREADS + tid);
    xs[c] = SEG ? (ii[c] >= 0 ? a.seq[ii[c]] : 0u) : (uint32_t)(base + e);
    nm[c] = ii[c] >= 0 ? a.name[ii[c]] : NN;
    pt[c] = (ii[c] >= 0 && a.part) ? a.part[ii[c]] : -1;
  }
  // batch 2: how each launch finds its row
  PartRec rc[kWaveChunks];
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    if (SEG && (int64_t)xs[c] >= a.T) ii[c] = -1;  // a broken promise: left out
    sii[c * OPA_TILE_THREADS + tid] = ii[c];
    const bool good = nm[c] < NN && pt[c] >= -1 && (pt[c] < 0 || (uint32_t)pt[c] < a.NP);
    rc[c] = PartRec{0, kRecNone};
    if (!good || ii[c] < 0) continue;
    if (pt[c] < 0) rc[c].hi = kRecEligible;
    else if (m.prec) rc[c] = m.prec[pt[c]];
    else if (a.part_rep[pt[c]] == pt[c]) rc[c].hi = kRecEligible;
  }
  // batch 3: the seq rank whose rank gives the row (own, or the launch at the
  // same position of the representative partition), its key and in-tile
  // rank, the name's prefix in that tile, and the name's rows
  uint32_t kr[kWaveChunks], pre[kWaveChunks], rows[kWaveChunks], ro[kWaveChunks];
  uint32_t dup = 0, err = 0;  // bit c: element c is a duplicate
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    uint32_t src = kNone;
    const uint32_t hi = rc[c].hi;
    if (hi == kRecEligible) {
      src = xs[c];
    } else if (hi != kRecNone) {
      if (xs[c] < hi) {
        src = xs[c] + (uint32_t)rc[c].delta;
        dup |= 1u << c;
      } else {
        err++;
      }
    }
    kr[c] = kNone;
    pre[c] = rows[c] = ro[c] = 0;
    if (src != kNone) {
      kr[c] = m.kr[src];
      pre[c] = m.tlh[(int64_t)(src >> OPA_SLOT_BITS) * NN + nm[c]];
      rows[c] = m.pfc[nm[c]];
      ro[c] = m.off[nm[c]];
      if (m.skip_name && m.tlc[nm[c]] != rows[c]) rows[c] = 0;  // the name is left out
    }
  }
  // batch 4: rows; a duplicate needs the representative's launch at its
  // position to have the same name
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int32_t i = sii[c * OPA_TILE_THREADS + tid];
    if (i < 0) continue;
    int32_t mt = -1;
    if (kr[c] != kNone) {
      if (((dup >> c) & 1u) && (kr[c] >> 16) != nm[c]) {
        err++;
      } else {
        const uint32_t r = pre[c] + (kr[c] & 0xFFFFu);
        if (r < rows[c]) mt = m.slot[ro[c] + r];
      }
    }
    m.match[i] = mt;
  }
  const unsigned long long e = wave_reduce_add((unsigned long long)err);
  if (lane_id() == 0 && e) atomicAdd(&serr, e);
  __syncthreads();
  if (tid == 0 && serr) atomicAdd((unsigned long long *)&m.diag->dedup_errors, serr);
}

// ---------------------------------------------------------------------------
// Bucket path (segment tiles, the fused attribution): the matching stops at
// the eligible launches. Per seq tile, a first pass counts the eligible
// launches of each name (the tile histogram) and writes them, in seq order,
// to the tile's bucket as (name, position). After the column scan a second
// pass ranks the buckets only -- a small fraction of the launches when most
// of them are layer duplicates -- and leaves, by seq rank, each eligible
// launch's row (mbs) and name (nbs). Every launch then finds its match in
// the fused aggregation pass over storage order: its own entry, or, for a
// duplicate, the entry of the representative's launch at its position.
// ---------------------------------------------------------------------------
struct BucketOut {
  uint32_t *tlh;                      // [tiles][NN] eligible launches per name
  uint32_t *rec;                      // [tiles][4096] name << 12 | position, in seq order
  uint32_t *cnt;                      // [tiles] bucket sizes
  uint32_t *pfirst, *plast, *pheads;  // pheads NULL: no partitions
  opattr_diag *diag;
};

__global__ void __launch_bounds__(256) k_f_pass1(TlArgs a, BucketOut o) {
  OPA_DYN_LDS(uint32_t, cnt);
  __shared__ TileData sm;
  __shared__ uint32_t sh[4];
  const int tid = threadIdx.x;
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = a.NN;
  for (uint32_t i = tid; i < NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  if (tid == 0) sm.bad = 0;
  const uint32_t bad = seg_tile(a, tile, sm);
  // this thread's 16 consecutive positions: counts, then the bucket in order
  constexpr int kPos = OPA_TILE / OPA_TILE_THREADS;
  const int e0 = tid * kPos;
  uint32_t key[kPos];
  uint32_t ne = 0;
#pragma unroll
  for (int k = 0; k < kPos; ++k) {
    key[k] = sm.key[e0 + k];
    if (key[k] < NN) {
      ne++;
      atomicAdd(&cnt[key[k]], 1u);
    }
  }
  uint32_t tot;
  uint32_t j = block_excl_scan_add<uint32_t>(ne, sh, &tot);
  uint32_t *rec = o.rec + base;
#pragma unroll
  for (int k = 0; k < kPos; ++k)
    if (key[k] < NN) rec[j++] = (key[k] << OPA_SLOT_BITS) | (uint32_t)(e0 + k);
  if (tid == 0) o.cnt[tile] = tot;
  __syncthreads();
  for (uint32_t n = tid; n < NN; n += OPA_TILE_THREADS) o.tlh[tile * NN + n] = cnt[n];
  if (o.pheads) part_edges(sm.lp, base, sm.sg.edge[0], sm.sg.edge[1], o.pfirst, o.plast, o.pheads);
  if (bad) atomicAdd(&sm.bad, bad);
  __syncthreads();
  if (tid == 0 && sm.bad)
    atomicAdd((unsigned long long *)&o.diag->bad_records, (unsigned long long)sm.bad);
}

// count validation (Sec. 3.3): per name, eligible launches against rows;
// run by one block of up to 1024 threads
__device__ void names_check(const uint32_t *__restrict__ tlc, const uint32_t *__restrict__ pfc,
                            uint32_t NN, uint32_t *name_counts, opattr_diag *diag, int strict) {
  __shared__ unsigned long long red[3][16];
  unsigned long long mism = 0, tlu = 0, pfu = 0;
  for (uint32_t n = threadIdx.x; n < NN; n += blockDim.x) {
    const uint32_t tl = tlc[n], pf = pfc[n];
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
    for (uint32_t i = 0; i < blockDim.x / OPA_WAVE; ++i) {
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

__global__ void __launch_bounds__(1024) k_names(const uint32_t *__restrict__ tlc,
                                                const uint32_t *__restrict__ pfc, uint32_t NN,
                                                uint32_t *name_counts, opattr_diag *diag,
                                                int strict) {
  names_check(tlc, pfc, NN, name_counts, diag, strict);
}

struct RankArgs {
  const uint32_t *rec, *cnt;  // the buckets
  const uint32_t *tlh;        // exclusive prefix of each name down the tiles
  const uint32_t *tlc, *pfc, *off;
  const int32_t *slot;
  int32_t *mbs;   // by seq rank: the row of each eligible launch (-1 none)
  uint32_t *nbs;  // by seq rank: its name
  uint32_t NN;
  int skip_name;
  // the count validation, by the block after the last tile (NN > 0)
  int64_t ntiles;
  uint32_t *name_counts;
  opattr_diag *diag;
  int strict;
};

// rank = (eligible launches of the name in earlier tiles) + (rank in the
// bucket, which is in seq order); row = slot[off[name] + rank] while the
// name has rows left (Alg. 1)
__global__ void __launch_bounds__(256) k_f_pass2(RankArgs m) {
  OPA_DYN_LDS(uint16_t, cnt);
  const int64_t tile = blockIdx.x, base = tile * OPA_TILE;
  const uint32_t NN = m.NN;
  if (tile >= m.ntiles) {
    names_check(m.tlc, m.pfc, NN, m.name_counts, m.diag, m.strict);
    return;
  }
  const uint32_t n = m.cnt[tile];
  if (n == 0) return;
  for (uint32_t i = threadIdx.x; i < 4 * NN; i += OPA_TILE_THREADS) cnt[i] = 0;
  __syncthreads();
  uint32_t key[kWaveChunks], pos[kWaveChunks], rank[kWaveChunks];
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const int e = tile_elem(c);
    const uint32_t r = (uint32_t)e < n ? m.rec[base + e] : (NN << OPA_SLOT_BITS);
    key[c] = r >> OPA_SLOT_BITS;
    pos[c] = r & (OPA_TILE - 1);
  }
  wave_rank<kWaveChunks>(key, NN, bits_for(NN), cnt + wave_id() * NN, rank);
  block_rank_bases(cnt, NN, nullptr);
  const uint16_t *wb = cnt + wave_id() * NN;
  const uint32_t *pre = m.tlh + tile * NN;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const uint32_t k = key[c];
    if (k >= NN) continue;
    const uint32_t r = pre[k] + wb[k] + rank[c];
    uint32_t rows = m.pfc[k];
    if (m.skip_name && m.tlc[k] != rows) rows = 0;  // the name is left out
    m.mbs[base + pos[c]] = r < rows ? m.slot[m.off[k] + r] : -1;
    m.nbs[base + pos[c]] = k;
  }
}

// ---------------------------------------------------------------------------
// Radix path (more names than the LDS counters hold)
// ---------------------------------------------------------------------------
// A[l] = (key << 12 | l) for the launches of seq ranks base..base+4095
// through the view; jidx[l] = input index (-1 holes). Returns bad-id count.
__device__ inline uint32_t tl_tile_keys(const TlArgs &a, int64_t base, uint32_t *A, int32_t *jidx) {
  const int tid = threadIdx.x;
  uint32_t bad = 0;
#pragma unroll 4
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int l = c * OPA_TILE_THREADS + tid;
    uint32_t key;
    int32_t j, lp;
    bad += tl_load(a, base + l, key, j, lp);
    A[l] = (key << OPA_SLOT_BITS) | (uint32_t)l;
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
  const uint32_t bad = tl_tile_keys(a, base, sm.A, nullptr);
  if (bad) atomicAdd(&sm.bad, bad);
  __syncthreads();
  if (threadIdx.x == 0 && sm.bad)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)sm.bad);
  tile_radix_sort(sm.A, sm.B, sm.srt, OPA_SLOT_BITS, bits_for(a.NN));
  write_hist_row(sm.A, a.NN, tlh + tile * a.NN);
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
  tl_tile_keys(a, base, sm.A, jidx);
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

// ---------------------------------------------------------------------------
// profiled rows: per-tile name histograms and the slot table
// ---------------------------------------------------------------------------
struct PfArgs {
  const uint32_t *name;
  int64_t P;
  uint32_t NN;
};

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
    if (n < NN) slot[off[n] + row[n] + wb[n] + rank[c]] = (int32_t)(base + tile_elem(c));
  }
}

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

// With few chunks, each block sums the chunk totals before its own (at most
// kFewChunks - 1 per column) instead of a separate scan over the chunks;
// the blocks of the last chunk write the column totals.
constexpr int64_t kFewChunks = 64;

__global__ void __launch_bounds__(256) k_colbase_few(uint32_t *tab, int64_t rows, uint32_t cols,
                                                     const uint32_t *__restrict__ chs,
                                                     uint32_t *totals, const int64_t *rows_dev) {
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
  uint32_t base = 0;
  if (col < cols) {
    const int64_t nb = blockIdx.y;  // chunks before this one
    for (int64_t c0 = 0; c0 < nb; c0 += 8) {
      uint32_t t[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) t[j] = c0 + j < nb ? chs[(c0 + j) * cols + col] : 0u;
#pragma unroll
      for (int j = 0; j < 8; ++j) base += t[j];
    }
  }
  __syncthreads();
  if (col >= cols) return;
  uint32_t run = base;
  for (int ww = 0; ww < w; ++ww) run += part[ww][l];
#pragma unroll
  for (int i = 0; i < kColChunk / 4; ++i) {
    const int64_t r = r0 + i;
    if (r < rows) tab[r * cols + col] = run;
    run += v[i];
  }
  const int64_t nc = (rows + kColChunk - 1) / kColChunk;
  if (w == 3 && (int64_t)blockIdx.y == nc - 1) totals[col] = run;
}

void column_scan(uint32_t *tab, int64_t rows, uint32_t cols, uint32_t *chs, uint32_t *totals,
                 hipStream_t s, const int64_t *rows_dev) {
  if (rows <= 0 || cols == 0) return;
  const int64_t nch = (rows + kColChunk - 1) / kColChunk;
  dim3 g((cols + 63) / 64, (unsigned)nch);
  k_colsum<<<g, 256, 0, s>>>(tab, rows, cols, chs, rows_dev);
  if (nch <= kFewChunks) {
    k_colbase_few<<<g, 256, 0, s>>>(tab, rows, cols, chs, totals, rows_dev);
  } else {
    k_chunkscan<<<(cols + 255) / 256, 256, 0, s>>>(chs, nch, cols, totals, rows, rows_dev);
    k_colbase<<<g, 256, 0, s>>>(tab, rows, cols, chs, rows_dev);
  }
}

// off[n] = rows of names before n (one block)
__global__ void __launch_bounds__(1024) k_pf_off(const uint32_t *__restrict__ pfc, uint32_t NN,
                                                 uint32_t *off) {
  __shared__ uint32_t sh[16];
  uint32_t carry = 0;
  for (uint32_t base = 0; base < NN; base += 1024) {
    const uint32_t n = base + threadIdx.x;
    const uint32_t pf = n < NN ? pfc[n] : 0u;
    uint32_t tot;
    const uint32_t pre = block_excl_scan_add<uint32_t>(pf, sh, &tot);
    if (n < NN) off[n] = carry + pre;
    carry += tot;
  }
}


// ---------------------------------------------------------------------------
// Stream-major order for launches with dense seq given in another order
// (opattr_attribute): a stable counting sort by stream of the launch-order
// view, one 4096-rank tile of it per block, that also gathers the launch
// arrays into that order. Launches with a stream id past the last stream
// sort after all others (the fused path counts them as bad records); seq
// ranks no launch claims (a false density promise) leave slots at the end,
// filled with records the fused path leaves out.
// ---------------------------------------------------------------------------
struct RemapArgs {
  const int32_t *sv;
  int64_t T, nt;
  uint32_t NS, NN;
  const uint32_t *seq, *name, *dur;
  const uint16_t *st;
  const uint64_t *start, *query;
  const int32_t *part;
  uint32_t *hist;  // [(NS + 1) * nt + 1], then its scan scratch
  int32_t *perm;  // slot -> launch (-1 past the placed ones)
  int32_t *inv;   // launch -> slot (-1 for a launch no seq rank holds)
  uint32_t *seq2, *name2, *dur2;
  uint16_t *st2;
  uint64_t *start2, *query2;
  int32_t *part2;
};

// the group of the launch at seq rank j: its stream, NS past the last
// stream, -1 when no launch holds the rank
__device__ __forceinline__ int remap_group(const RemapArgs &a, int64_t j, int32_t &i) {
  i = j < a.T ? a.sv[j] : -1;
  if (i < 0) return -1;
  const uint32_t s = a.st[i];
  return (int)(s < a.NS ? s : a.NS);
}

__global__ void __launch_bounds__(256) k_remap_hist(RemapArgs a) {
  __shared__ uint32_t c[kMaxSegStreams + 1];
  const int tid = threadIdx.x;
  if (tid <= (int)a.NS) c[tid] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  for (int e = tid; e < OPA_TILE; e += 256) {
    int32_t i;
    const int g = remap_group(a, base + e, i);
    if (g >= 0) atomicAdd(&c[g], 1u);
  }
  __syncthreads();
  if (tid <= (int)a.NS) a.hist[(int64_t)tid * a.nt + blockIdx.x] = c[tid];
  if (blockIdx.x == 0 && tid == 0) a.hist[(int64_t)(a.NS + 1) * a.nt] = 0;  // the total, after the scan
}

__global__ void __launch_bounds__(256) k_remap_scatter(RemapArgs a) {
  __shared__ uint16_t cnt[OPA_TILE_CHUNKS][4][kMaxSegStreams + 1];
  __shared__ int32_t lidx[OPA_TILE];  // the tile's launches in (group, rank) order
  __shared__ uint8_t lgrp[OPA_TILE];
  __shared__ uint32_t lbase[kMaxSegStreams + 1], sh[4];
  const int tid = threadIdx.x, w = wave_id();
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  const int ng = (int)a.NS + 1;
  for (int q = tid; q < OPA_TILE_CHUNKS * 4 * (kMaxSegStreams + 1); q += 256)
    (&cnt[0][0][0])[q] = 0;
  __syncthreads();
  int32_t ii[OPA_TILE_CHUNKS];
  uint32_t lr[OPA_TILE_CHUNKS];
  int gg[OPA_TILE_CHUNKS];
#pragma unroll
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int g = remap_group(a, base + c * 256 + tid, ii[c]);
    gg[c] = g;
    const uint64_t pm = peers8((uint32_t)(g >= 0 ? g : 255)) & __ballot(g >= 0);
    lr[c] = (uint32_t)__popcll(pm & lanemask_lt());
    if (g >= 0 && (pm & lanemask_lt()) == 0) cnt[c][w][g] = (uint16_t)__popcll(pm);
  }
  __syncthreads();
  uint32_t tot = 0;  // thread g: its group's counts over (chunk, wave), in rank order
  if (tid < ng)
    for (int c = 0; c < OPA_TILE_CHUNKS; ++c)
      for (int ww = 0; ww < 4; ++ww) {
        const uint32_t v = cnt[c][ww][tid];
        cnt[c][ww][tid] = (uint16_t)tot;
        tot += v;
      }
  uint32_t nl;
  const uint32_t lb = block_excl_scan_add<uint32_t>(tid < ng ? tot : 0u, sh, &nl);
  if (tid < ng) lbase[tid] = lb;
  __syncthreads();
  // each launch's place: in the tile's LDS order, and its final one (inv)
#pragma unroll
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int g = gg[c];
    if (g < 0) continue;
    const uint32_t r = cnt[c][w][g] + lr[c];
    lidx[lbase[g] + r] = ii[c];
    lgrp[lbase[g] + r] = (uint8_t)g;
    a.inv[ii[c]] = (int32_t)(a.hist[(int64_t)g * a.nt + blockIdx.x] + r);
  }
  __syncthreads();
  // written in that order: each group's launches go to consecutive slots
  for (int j = tid; j < (int)nl; j += 256) {
    const int32_t i = lidx[j];
    const int g = lgrp[j];
    const int64_t dst = (int64_t)a.hist[(int64_t)g * a.nt + blockIdx.x] + (j - (int)lbase[g]);
    a.perm[dst] = i;
    a.seq2[dst] = a.seq[i];
    a.name2[dst] = a.name[i];
    a.dur2[dst] = a.dur[i];
    a.st2[dst] = a.st[i];
    a.start2[dst] = a.start[i];
    if (a.query2) a.query2[dst] = a.query[i];
    if (a.part2) a.part2[dst] = a.part[i];
  }
}

// slots past the placed launches: records the fused path leaves out (seq
// past n, stream and name out of range)
__global__ void k_remap_tail(RemapArgs a) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t placed = a.hist[(int64_t)(a.NS + 1) * a.nt];
  if (x >= a.T || x < placed) return;
  a.perm[x] = -1;
  a.seq2[x] = (uint32_t)(a.T + (x - placed) < 0xFFFFFFFFll ? a.T + (x - placed) : 0xFFFFFFFFll);
  a.name2[x] = a.NN;
  a.dur2[x] = 0;
  a.st2[x] = 0xFFFFu;
  a.start2[x] = ~0ull;
  if (a.query2) a.query2[x] = ~0ull;
  if (a.part2) a.part2[x] = -1;
}

void remap_view(const opattr_kernels *k, void *ws, const Plan &pl, opattr_kernels *out) {
  *out = *k;
  out->seq = at<uint32_t>(ws, pl.rm_seq);
  out->name_id = at<uint32_t>(ws, pl.rm_name);
  out->dur_ns = at<uint32_t>(ws, pl.rm_dur);
  out->stream_id = at<uint16_t>(ws, pl.rm_st);
  out->start_ns = at<uint64_t>(ws, pl.rm_start);
  out->query_ns = k->query_ns ? at<uint64_t>(ws, pl.rm_query) : nullptr;
  out->part_id = k->part_id ? at<int32_t>(ws, pl.rm_part) : nullptr;
}

size_t remap_hist_entries(const Plan &pl) {
  const int64_t h = ((int64_t)pl.NS + 1) * pl.nt + 1;
  return (size_t)h + scan_scratch_entries(h);
}

void remap_launches(const opattr_kernels *k, const opattr_dims *d, void *ws, const Plan &pl,
                    opattr_kernels *out, hipStream_t s) {
  RemapArgs a{};
  a.sv = at<int32_t>(ws, pl.sv);
  a.T = pl.T;
  a.nt = pl.nt;
  a.NS = d->n_streams;
  a.NN = d->n_names;
  a.seq = k->seq;
  a.name = k->name_id;
  a.dur = k->dur_ns;
  a.st = k->stream_id;
  a.start = k->start_ns;
  a.query = k->query_ns;
  a.part = k->part_id;
  a.hist = at<uint32_t>(ws, pl.rm_hist);
  a.perm = at<int32_t>(ws, pl.rm_perm);
  a.inv = at<int32_t>(ws, pl.rm_inv);
  a.seq2 = at<uint32_t>(ws, pl.rm_seq);
  a.name2 = at<uint32_t>(ws, pl.rm_name);
  a.dur2 = at<uint32_t>(ws, pl.rm_dur);
  a.st2 = at<uint16_t>(ws, pl.rm_st);
  a.start2 = at<uint64_t>(ws, pl.rm_start);
  a.query2 = k->query_ns ? at<uint64_t>(ws, pl.rm_query) : nullptr;
  a.part2 = k->part_id ? at<int32_t>(ws, pl.rm_part) : nullptr;
  if (out) remap_view(k, ws, pl, out);
  if (pl.T <= 0) return;
  const int64_t h = ((int64_t)a.NS + 1) * a.nt + 1;
  fill_u32(reinterpret_cast<uint32_t *>(a.inv), 0xFFFFFFFFu, a.T, s);
  k_remap_hist<<<(unsigned)a.nt, 256, 0, s>>>(a);
  scan_excl_inplace(a.hist, h, a.hist + h, s);
  k_remap_scatter<<<(unsigned)a.nt, 256, 0, s>>>(a);
  k_remap_tail<<<(unsigned)((a.T + 255) / 256), 256, 0, s>>>(a);
}

// by launch, so that the caller's arrays are written in order
__global__ void k_remap_back(const int32_t *inv, const int32_t *m2, const int32_t *r2, int64_t T,
                             int32_t *match, int32_t *range_id) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= T) return;
  const int32_t x = inv[i];
  if (x < 0) return;  // no seq rank holds the launch (a false density promise)
  match[i] = m2[x];
  range_id[i] = r2[x];
}

void remap_back(void *ws, const Plan &pl, int32_t *match, int32_t *range_id, hipStream_t s) {
  if (pl.T > 0)
    k_remap_back<<<(unsigned)((pl.T + 255) / 256), 256, 0, s>>>(
        at<int32_t>(ws, pl.rm_inv), at<int32_t>(ws, pl.rm_match), at<int32_t>(ws, pl.rm_rid), pl.T,
        match, range_id);
}

// Layout promise of the kernels (checked under OPATTR_VALIDATE): sorted by
// (stream, seq) with seq unique, streams below n_streams, query points not
// decreasing along a stream.
__global__ void k_check_stream_major(const uint16_t *st, const uint32_t *seq, const uint64_t *q,
                                     int64_t T, uint32_t NS, opattr_diag *diag) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (i < T) {
    bad = st[i] >= NS;
    if (i > 0) {
      const uint16_t a = st[i - 1], b = st[i];
      bad = bad || a > b || (a == b && (seq[i - 1] >= seq[i] || q[i - 1] > q[i]));
    }
  }
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1) {
    atomicAdd((unsigned long long *)&diag->order_violations, (unsigned long long)__popcll(m));
    atomicOr(&diag->flags, OPATTR_F_ORDER);
  }
}

void check_kernel_layout(const opattr_kernels *k, const opattr_dims *d, opattr_diag *diag,
                         hipStream_t s) {
  if (!(d->flags & OPATTR_KERNELS_STREAM_MAJOR) || !(d->flags & OPATTR_VALIDATE) || k->n <= 0 ||
      !k->seq || !k->stream_id || !(k->query_ns || k->start_ns))
    return;
  k_check_stream_major<<<(unsigned)((k->n + 255) / 256), 256, 0, s>>>(
      k->stream_id, k->seq, k->query_ns ? k->query_ns : k->start_ns, k->n, d->n_streams, diag);
}

// ---------------------------------------------------------------------------
// layer dedup as its own pass (radix path and the standalone broadcast)
// ---------------------------------------------------------------------------
struct DedupArgs {
  int64_t T;
  const uint32_t *seq;
  const int32_t *rk;  // NULL when seq is dense
  const uint32_t *name;
  const int32_t *part;
  const int32_t *part_rep;
  uint32_t NN, NP;
  const uint32_t *pfirst, *plast, *pheads;
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
        bool ok = a.pheads[pt] == 1u && a.part_rep[r] == r && f != 0xFFFFFFFFu &&
                  a.pheads[r] == 1u;
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

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static bool has_dedup(const opattr_kernels *k, const opattr_dims *d) {
  return k->part_id && d->part_rep && d->n_parts > 0;
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
  a.seq = k->seq;
  a.bnd = at<uint32_t>(ws, pl.tbnd);
  a.kblk = at<int64_t>(ws, pl.kblk);
  a.NS = d->n_streams;
  a.vdiag = nullptr;
  return a;
}

static DedupArgs dedup_args(const opattr_kernels *k, const opattr_dims *d, int32_t *match,
                            opattr_diag *diag, void *ws, const Plan &pl) {
  DedupArgs a;
  a.T = pl.T;
  a.seq = k->seq;
  a.rk = pl.seq_dense ? nullptr : at<int32_t>(ws, pl.rk);
  a.name = k->name_id;
  a.part = k->part_id;
  a.part_rep = d->part_rep;
  a.NN = d->n_names;
  a.NP = d->n_parts;
  a.pfirst = at<uint32_t>(ws, pl.pfirst);
  a.plast = at<uint32_t>(ws, pl.plast);
  a.pheads = at<uint32_t>(ws, pl.pheads);
  a.mbs = at<int32_t>(ws, pl.mbs);
  a.nbs = at<uint32_t>(ws, pl.nbs);
  a.match = match;
  a.diag = diag;
  return a;
}

static void clear_partitions(FillJobs &f, void *ws, const Plan &pl) {
  f.add(at<uint32_t>(ws, pl.pfirst), 0xFFFFFFFFu, pl.NP);
  f.add(at<uint32_t>(ws, pl.plast), 0xFFFFFFFFu, pl.NP);
  f.add(at<uint32_t>(ws, pl.pheads), 0u, pl.NP);
}

void run_match(const IomArgs &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const opattr_kernels *k = x.k;
  const opattr_dims *d = x.d;
  void *ws = x.ws;
  const uint32_t NN = d->n_names;
  const bool dedup = has_dedup(k, d);
  const bool parts = dedup && x.want_dedup;
  const bool seg = pl.seg;  // implies the fast path
  const bool buckets = seg && x.buckets;
  const bool fast = NN <= kFastNames, fast_pf = NN <= kFastKeys;
  const size_t lds = (size_t)4 * NN * sizeof(uint16_t);
  uint32_t *tlh = at<uint32_t>(ws, pl.tlh), *pfh = at<uint32_t>(ws, pl.pfh);
  uint32_t *tlc = at<uint32_t>(ws, pl.tlc), *pfc = at<uint32_t>(ws, pl.pfc);
  uint32_t *off = at<uint32_t>(ws, pl.off);
  uint32_t *pfirst = at<uint32_t>(ws, pl.pfirst), *plast = at<uint32_t>(ws, pl.plast);
  uint32_t *pheads = at<uint32_t>(ws, pl.pheads);
  FillJobs clr;
  clr.add(tlc, 0, NN);
  clr.add(pfc, 0, NN);
  if (parts) clear_partitions(clr, ws, pl);
  // The tiles reach only the launches that the layout promises put in them
  // (the segment path), or that hold their seq slot in the view; under
  // OPATTR_VALIDATE, where a false promise must come out as an order error,
  // every launch's match starts unmatched so that none is read unwritten.
  // (The bucket path writes every match in storage order.)
  if (!buckets && x.validate && x.match) clr.add(x.match, 0xFFFFFFFFu, pl.T);
  const bool seg_pro = seg && pl.nt > 0;  // clears, class-map check and stream blocks in one launch
  if (seg_pro) {
    ProArgs pa{};
    pa.fill = clr;
    int64_t mx = 0;
    for (int q = 0; q < clr.count; ++q) mx = clr.n[q] > mx ? clr.n[q] : mx;
    pa.nf = (int)((mx + 255) / 256 < 1024 ? (mx + 255) / 256 : 1024);
    pa.nr = dedup ? (int)((d->n_parts + 255) / 256) : 0;
    pa.part_rep = d->part_rep;
    pa.NP = d->n_parts;
    pa.diag = x.diag;
    pa.st = k->stream_id;
    pa.T = pl.T;
    pa.NS = pl.NS;
    pa.kblk = at<int64_t>(ws, pl.kblk);
    const int nw = (int)((pl.NS + 1 + 3) / 4);
    k_seg_prologue<<<(unsigned)(pa.nf + pa.nr + nw), 256, 0, s>>>(pa);
  } else {
    fill_many(clr, s);
    if (dedup) k_rep_check<<<(d->n_parts + 255) / 256, 256, 0, s>>>(d->part_rep, d->n_parts, x.diag);
  }
  TlArgs ta = tl_args(k, d, ws, pl, dedup);
  if (seg && x.validate) ta.vdiag = x.diag;  // the density of seq, checked in the tiles
  PfArgs pa;
  pa.name = x.p->name_id;
  // the rows of this call (the plan may be sized for a longer list)
  const int64_t P = x.p->n < pl.P ? x.p->n : pl.P;
  const int64_t ntp = (P + OPA_TILE - 1) / OPA_TILE;
  pa.P = P;
  pa.NN = NN;
  // the profiled side depends only on the row names: it runs on its own
  // stream when one is given, joined back before the lookups
  const hipStream_t sp = x.pf_stream ? x.pf_stream : s;
  if (sp != s) {
    note(hipEventRecord(x.pf_fork, s));
    note(hipStreamWaitEvent(sp, x.pf_fork, 0));
  }
  probe_begin(OPATTR_PROBE_PF_HIST, sp);
  if (ntp > 0) {
    if (fast_pf) k_pf_hist_w<<<(unsigned)ntp, 256, lds, sp>>>(pa, pfh, x.diag);
    else k_pf_hist<<<(unsigned)ntp, 256, 0, sp>>>(pa, pfh, x.diag);
  }
  probe_end(OPATTR_PROBE_PF_HIST, sp);
  column_scan(pfh, ntp, NN, at<uint32_t>(ws, pl.pfch), pfc, sp, nullptr);
  if (NN) k_pf_off<<<1, 1024, 0, sp>>>(pfc, NN, off);
  probe_begin(OPATTR_PROBE_PF_SLOT, sp);
  if (ntp > 0) {
    if (fast_pf) k_pf_slot_w<<<(unsigned)ntp, 256, lds, sp>>>(pa, pfh, off, at<int32_t>(ws, pl.slot));
    else k_pf_slot<<<(unsigned)ntp, 256, 0, sp>>>(pa, pfh, off, at<int32_t>(ws, pl.slot));
  }
  probe_end(OPATTR_PROBE_PF_SLOT, sp);
  if (x.fused_order && sp != s) run_fused_order(k, ws, pl, sp);
  if (sp != s) note(hipEventRecord(x.pf_join, sp));

  // the timeline side
  if (seg && pl.nt > 0) {
    if (!seg_pro) launch_stream_blocks(k->stream_id, pl.T, pl.NS, at<int64_t>(ws, pl.kblk), s);
    const int64_t nb = (pl.nt + 1) * pl.NS;
    k_tile_bounds<<<(unsigned)((nb + 255) / 256), 256, 0, s>>>(k->seq, at<int64_t>(ws, pl.kblk),
                                                             pl.NS, pl.nt, at<uint32_t>(ws, pl.tbnd));
  }
  HistOut ho;
  ho.tlh = tlh;
  ho.kr = at<uint32_t>(ws, pl.nbs);
  ho.pfirst = pfirst;
  ho.plast = plast;
  ho.pheads = parts ? pheads : nullptr;
  ho.diag = x.diag;
  BucketOut bo;
  bo.tlh = tlh;
  bo.rec = at<uint32_t>(ws, pl.sv);  // the launch-order view is unused on the segment path
  bo.cnt = at<uint32_t>(ws, pl.bcnt);
  bo.pfirst = pfirst;
  bo.plast = plast;
  bo.pheads = parts ? pheads : nullptr;
  bo.diag = x.diag;
  probe_begin(OPATTR_PROBE_TL_HIST, s);
  if (pl.nt > 0) {
    if (buckets) {
      k_f_pass1<<<(unsigned)pl.nt, 256, (size_t)NN * 4, s>>>(ta, bo);
    } else if (seg) {
      k_tl_hist_w<true><<<(unsigned)pl.nt, 256, lds, s>>>(ta, ho);
    } else if (fast) {
      k_tl_hist_w<false><<<(unsigned)pl.nt, 256, lds, s>>>(ta, ho);
    } else {
      k_tl_hist<<<(unsigned)pl.nt, 256, 0, s>>>(ta, tlh, x.diag);
      if (parts) k_part_edges<<<(unsigned)pl.nt, 256, 0, s>>>(ta, pfirst, plast, pheads);
    }
  }
  probe_end(OPATTR_PROBE_TL_HIST, s);
  PartRec *prec = (parts && fast) ? at<PartRec>(ws, pl.prec) : nullptr;
  if (parts && pl.nt > 0)
    k_part_prep<<<(unsigned)((pl.NP + 255) / 256), 256, 0, s>>>(d->part_rep, pl.NP, pfirst, plast,
                                                                pheads, prec, x.diag);
  probe_begin(OPATTR_PROBE_COL_SCAN, s);
  column_scan(tlh, pl.nt, NN, at<uint32_t>(ws, pl.tlch), tlc, s, nullptr);
  probe_end(OPATTR_PROBE_COL_SCAN, s);
  if (sp != s) note(hipStreamWaitEvent(s, x.pf_join, 0));
  const int strict = x.policy == OPATTR_MISMATCH_STRICT ? 1 : 0;
  const bool names_in_pass2 = pl.nt > 0 && buckets;  // an extra block of the ranking
  if (NN && !names_in_pass2) k_names<<<1, 1024, 0, s>>>(tlc, pfc, NN, x.name_counts, x.diag, strict);
  probe_begin(OPATTR_PROBE_TL_MATCH, s);
  if (pl.nt > 0 && buckets) {
    RankArgs m;
    m.rec = bo.rec;
    m.cnt = bo.cnt;
    m.tlh = tlh;
    m.tlc = tlc;
    m.pfc = pfc;
    m.off = off;
    m.slot = at<int32_t>(ws, pl.slot);
    m.mbs = at<int32_t>(ws, pl.mbs);
    m.nbs = at<uint32_t>(ws, pl.nbs);
    m.NN = NN;
    m.skip_name = x.policy == OPATTR_MISMATCH_SKIP_NAME ? 1 : 0;
    m.ntiles = pl.nt;
    m.name_counts = x.name_counts;
    m.diag = x.diag;
    m.strict = strict;
    k_f_pass2<<<(unsigned)(pl.nt + (NN ? 1 : 0)), 256, lds, s>>>(m);
  } else if (pl.nt > 0) {
    if (fast) {
      LookArgs m;
      m.tlh = tlh;
      m.tlc = tlc;
      m.pfc = pfc;
      m.off = off;
      m.slot = at<int32_t>(ws, pl.slot);
      m.kr = ho.kr;
      m.prec = prec;
      m.match = x.match;
      m.skip_name = x.policy == OPATTR_MISMATCH_SKIP_NAME ? 1 : 0;
      m.diag = x.diag;
      if (seg) k_tl_look<true><<<(unsigned)pl.nt, 256, 0, s>>>(ta, m);
      else k_tl_look<false><<<(unsigned)pl.nt, 256, 0, s>>>(ta, m);
    } else {
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
      k_tl_match<<<(unsigned)pl.nt, 256, 0, s>>>(ta, ma);
    }
  }
  probe_end(OPATTR_PROBE_TL_MATCH, s);
  // the radix path broadcasts to duplicates in a pass of its own
  if (parts && !fast && pl.T > 0) {
    const DedupArgs da = dedup_args(k, d, x.match, x.diag, ws, pl);
    probe_begin(OPATTR_PROBE_DEDUP, s);
    k_dedup<<<(unsigned)((pl.T + 255) / 256), 256, 0, s>>>(da);
    probe_end(OPATTR_PROBE_DEDUP, s);
  }
}

// standalone broadcast over a given match array
void run_dedup(const opattr_kernels *k, const opattr_dims *d, int32_t *match, opattr_diag *diag,
               void *ws, const Plan &pl, hipStream_t s) {
  if (!has_dedup(k, d) || pl.T <= 0) return;
  const DedupArgs a = dedup_args(k, d, match, diag, ws, pl);
  const TlArgs ta = tl_args(k, d, ws, pl, true);
  const unsigned nb = (unsigned)((pl.T + 255) / 256);
  probe_begin(OPATTR_PROBE_DEDUP, s);
  FillJobs clr;
  clear_partitions(clr, ws, pl);
  fill_many(clr, s);
  k_part_edges<<<(unsigned)pl.nt, 256, 0, s>>>(ta, at<uint32_t>(ws, pl.pfirst),
                                               at<uint32_t>(ws, pl.plast),
                                               at<uint32_t>(ws, pl.pheads));
  k_part_prep<<<(unsigned)((pl.NP + 255) / 256), 256, 0, s>>>(
      d->part_rep, pl.NP, at<uint32_t>(ws, pl.pfirst), at<uint32_t>(ws, pl.plast),
      at<uint32_t>(ws, pl.pheads), nullptr, diag);
  k_src_fill<<<nb, 256, 0, s>>>(a);
  k_dedup<<<nb, 256, 0, s>>>(a);
  probe_end(OPATTR_PROBE_DEDUP, s);
}

// out[i * 20 + c] = counter c of row match[i]. A block writes 64 whole
// rows (1280 consecutive floats): thread t takes elements t, t + 256, ...,
// so every store is coalesced and the lanes of one row read its counters
// side by side (contiguous when the counters are row-major).
constexpr int kCoRows = 64;
__global__ void __launch_bounds__(256) k_counters_out(const float *__restrict__ cnt, int64_t rs,
                                                      int64_t cs, int64_t P, uint32_t absent,
                                                      const int32_t *__restrict__ match,
                                                      int64_t T, float *__restrict__ out) {
  const int64_t i0 = (int64_t)blockIdx.x * kCoRows;
  const int64_t nr = T - i0 < kCoRows ? T - i0 : kCoRows;
  const int ne = (int)nr * OPATTR_NUM_COUNTERS;
#pragma unroll
  for (int k = 0; k < kCoRows * OPATTR_NUM_COUNTERS / 256; ++k) {
    const int e = k * 256 + (int)threadIdx.x;
    if (e >= ne) break;
    const int r = e / OPATTR_NUM_COUNTERS, c = e - r * OPATTR_NUM_COUNTERS;
    const int32_t m = match[i0 + r];
    float v = __builtin_nanf("");
    if (m >= 0 && m < P && !((absent >> c) & 1u)) v = cnt[(int64_t)m * rs + (int64_t)c * cs];
    out[i0 * OPATTR_NUM_COUNTERS + e] = v;
  }
}

void run_counters_out(const opattr_profiled *p, const int32_t *match, int64_t T, float *out,
                      hipStream_t s) {
  if (T <= 0) return;
  const unsigned nb = (unsigned)((T + kCoRows - 1) / kCoRows);
  k_counters_out<<<nb, 256, 0, s>>>(p->counters, p->row_stride, p->col_stride, p->n,
                                    p->absent_mask, match, T, out);
}

}  // namespace opa
