// Dedup class discovery (Sec. 3.7) on the GPU.
//
// Two partitions are one class when their launches (valid name and
// partition) form the same (name, stream) sequence in launch order; a class
// is represented by its lowest-numbered partition, and a partition whose
// launches are not consecutive in launch order is a class of its own.
//
// Everything runs over launch-order ranks (the seq view), where a
// consecutive partition is one run of ranks, so that no per-launch offsets
// or counts need atomics:
//   1. per rank: the packed (name, stream) and the partition of its launch;
//      run edges give each partition its first and last rank and its number
//      of runs (one run = consecutive);
//   2. per rank: a position-keyed 64-bit hash of the element, summed per
//      partition (one atomic per piece of a partition inside a wave);
//   3. key -> lowest partition with that key (block-local table in LDS, then
//      an open-addressing table): the candidate representative, never above
//      the true one (equal sequences have equal keys);
//   4. per rank: compare the element with the candidate's element at the
//      same position; with no difference the candidate is the representative;
//   5. partitions that differ from their candidate (a key collision) search
//      exactly: the lowest-numbered partition with their key and sequence.
#include "common.h"
#include "impl.h"

namespace opa {

struct ClsArgs {
  int64_t T;
  const int32_t *sv;  // launch-order view: input index at each rank
  const uint32_t *name;
  const uint16_t *stream;
  const int32_t *part;
  uint32_t NN, NP;
  uint64_t *rs;  // [T] (name << 16 | stream) of the launch at each rank
  int32_t *rp;   // [T] its partition; -1 none, -2 a bad id, -3 no launch
  uint32_t *first, *last, *runs;  // [NP] first and last rank, runs of ranks
  uint64_t *key;                  // [NP] sequence hash, then with the length folded in
  uint32_t *cand, *fail;          // [NP] candidate representative, differs from it
  uint32_t *list, *nfail;         // partitions that differ from their candidate
  uint64_t *tkey;                 // [tmask + 1] table keys (0 = empty)
  uint32_t *tmin;                 // [tmask + 1] lowest partition with the key
  uint32_t tmask;
  uint64_t kmask;  // bits of the key kept (all but in tests of the exact search)
  int32_t *part_rep;
  opattr_diag *diag;
};

// splitmix64's output function (Steele, Lea and Flood, 2014)
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t elem_hash(uint64_t v, uint32_t pos) {
  return mix64(v + 0x9E3779B97F4A7C15ull * ((uint64_t)pos + 1));
}

// members of partition q when it is one run of ranks, else 0; ok = consecutive
__device__ __forceinline__ uint32_t members(const ClsArgs &a, uint32_t q, bool &ok) {
  const uint32_t n = a.runs[q];
  ok = n <= 1;
  return n == 1 ? a.last[q] - a.first[q] + 1 : 0u;
}

// partition of the launch at rank x (-1 none, -2 bad id, -3 no launch: only
// when a dense-seq promise is false); bad = an id out of range
__device__ __forceinline__ int32_t rank_part(const ClsArgs &a, int64_t x, uint64_t &v, bool &bad) {
  bad = false;
  v = 0;
  const int32_t i = a.sv[x];
  if (i < 0 || (int64_t)i >= a.T) return -3;
  const uint32_t nm = a.name[i];
  const int32_t p = a.part[i];
  v = ((uint64_t)nm << 16) | a.stream[i];
  bad = nm >= a.NN || p < -1 || (p >= 0 && (uint32_t)p >= a.NP);
  return bad ? -2 : p;
}

__device__ __forceinline__ void mark_fail(const ClsArgs &a, uint32_t q) {
  if (atomicOr(&a.fail[q], 1u) == 0u) a.list[atomicAdd(a.nfail, 1u)] = q;
}

// 1. elements and partitions by rank; run edges
__global__ void __launch_bounds__(256) k_cls_runs(ClsArgs a) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int l = lane_id();
  bool bad = false;
  uint64_t v = 0;
  const int32_t lp = x < a.T ? rank_part(a, x, v, bad) : -3;
  if (x < a.T) {
    a.rs[x] = v;
    a.rp[x] = lp;
  }
  const uint64_t mb = __ballot(bad);
  if (mb && l == __ffsll((unsigned long long)mb) - 1)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)__popcll(mb));
  // neighbours across the wave edges are classified again
  int32_t prev = __shfl_up(lp, 1, OPA_WAVE), next = __shfl_down(lp, 1, OPA_WAVE);
  uint64_t dv;
  bool db;
  if (l == 0) prev = (x > 0 && x - 1 < a.T) ? rank_part(a, x - 1, dv, db) : -3;
  if (l == OPA_WAVE - 1) next = x + 1 < a.T ? rank_part(a, x + 1, dv, db) : -3;
  if (lp >= 0) {
    if (prev != lp) {
      a.first[lp] = (uint32_t)x;
      atomicAdd(&a.runs[lp], 1u);
    }
    if (next != lp) a.last[lp] = (uint32_t)x;
  }
}

// 2a. PARTITION for partitions of several runs
__global__ void k_cls_consecutive(ClsArgs a) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  const bool nc = q < a.NP && a.runs[q] > 1;
  if (__ballot(nc) && lane_id() == 0) atomicOr(&a.diag->flags, OPATTR_F_PARTITION);
}

// 2b. sequence hash: position-keyed element hashes summed per partition; the
// lanes of a wave holding one partition are contiguous (ranks), so each such
// piece is summed in the wave and added once
__global__ void __launch_bounds__(256) k_cls_hash(ClsArgs a) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int l = lane_id();
  int32_t p = x < a.T ? a.rp[x] : -1;
  uint64_t h = 0;
  if (p >= 0) {
    if (a.runs[p] == 1) h = elem_hash(a.rs[x], (uint32_t)(x - a.first[p]));
    else p = -1;
  }
  const int32_t pp = __shfl_up(p, 1, OPA_WAVE), pn = __shfl_down(p, 1, OPA_WAVE);
  const bool head = l == 0 || pp != p;
  const bool tail = l == OPA_WAVE - 1 || pn != p;
  const uint64_t heads = __ballot(head);
  // first lane of this lane's piece: the highest head at or below it
  const uint64_t upto = l == OPA_WAVE - 1 ? heads : heads & ((2ull << l) - 1);
  const int start = 63 - __clzll((long long)upto);
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    const uint64_t y = __shfl_up(h, (unsigned)o, OPA_WAVE);
    if (l - o >= start) h += y;
  }
  if (tail && p >= 0) atomicAdd((unsigned long long *)&a.key[p], (unsigned long long)h);
}

__device__ __forceinline__ uint32_t table_home(uint64_t k, uint32_t mask) {
  return (uint32_t)(k ^ (k >> 32)) & mask;
}

constexpr int kLocalSlots = 512;  // block-local key table (256 partitions per block)

// 3a. key with the length folded in; the lowest partition per key, first in a
// block-local LDS table, then once per distinct key of the block in the
// global table (duplicates are the common case: every layer of a class)
__global__ void __launch_bounds__(256) k_cls_insert(ClsArgs a) {
  __shared__ unsigned long long lk[kLocalSlots];
  __shared__ uint32_t lq[kLocalSlots];
  for (int s = threadIdx.x; s < kLocalSlots; s += blockDim.x) {
    lk[s] = 0ull;
    lq[s] = 0xFFFFFFFFu;
  }
  __syncthreads();
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q < a.NP) {
    bool ok;
    const uint32_t n = members(a, q, ok);
    if (ok) {
      uint64_t k = mix64(a.key[q] ^ mix64((uint64_t)n + 0x632BE59BD9B4E019ull)) & a.kmask;
      if (k == 0) k = 1;
      a.key[q] = k;
      // at most 256 keys in 512 slots: an empty slot or k is always reached
      uint32_t s = table_home(k, kLocalSlots - 1);
      for (int it = 0; it < kLocalSlots; ++it) {
        const unsigned long long prev = atomicCAS(&lk[s], 0ull, (unsigned long long)k);
        if (prev == 0ull || prev == k) {
          atomicMin(&lq[s], q);
          break;
        }
        s = (s + 1) & (kLocalSlots - 1);
      }
    }
  }
  __syncthreads();
  for (int s = threadIdx.x; s < kLocalSlots; s += blockDim.x) {
    const uint64_t k = lk[s];
    if (k == 0) continue;
    const uint32_t lo = lq[s];
    // the table has at least twice as many slots as partitions: a slot that
    // is empty or holds k is reached within tmask + 1 probes
    uint32_t g = table_home(k, a.tmask);
    for (uint32_t it = 0; it <= a.tmask; ++it) {
      // keys and minima only ever go from empty to k and downwards, so a
      // stale read can only cost an atomic, never skip a needed one
      uint64_t cur = a.tkey[g];
      if (cur == 0ull)
        cur = atomicCAS((unsigned long long *)&a.tkey[g], 0ull, (unsigned long long)k);
      if (cur == 0ull || cur == k) {
        if (a.tmin[g] > lo) atomicMin(&a.tmin[g], lo);
        break;
      }
      g = (g + 1) & a.tmask;
    }
  }
}

// 3b. candidate representative; a length that differs is a collision
__global__ void k_cls_candidate(ClsArgs a) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= a.NP) return;
  uint32_t c = q;
  bool ok;
  const uint32_t n = members(a, q, ok);
  if (ok) {
    const uint64_t k = a.key[q];
    uint32_t g = table_home(k, a.tmask);
    for (uint32_t it = 0; it <= a.tmask; ++it) {
      if (a.tkey[g] == k) {
        c = a.tmin[g];
        break;
      }
      g = (g + 1) & a.tmask;
    }
    bool cok;
    if (c != q && members(a, c, cok) != n) mark_fail(a, q);
  }
  a.cand[q] = c;
  a.part_rep[q] = (int32_t)c;
}

// 4. element-wise comparison with the candidate
__global__ void __launch_bounds__(256) k_cls_verify(ClsArgs a) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= a.T) return;
  const int32_t p = a.rp[x];
  if (p < 0 || a.runs[p] != 1) return;
  const uint32_t c = a.cand[p];
  if (c == (uint32_t)p) return;
  bool ok;
  if (members(a, c, ok) != members(a, (uint32_t)p, ok)) return;  // failed already
  if (a.rs[a.first[c] + (x - a.first[p])] != a.rs[x]) mark_fail(a, (uint32_t)p);
}

// 5. exact search for the partitions that differ from their candidate: the
// lowest-numbered consecutive partition with the same key and sequence
// (itself when none). One block per such partition, striding.
__global__ void __launch_bounds__(256) k_cls_resolve(ClsArgs a) {
  const uint32_t nf = *a.nfail;
  for (uint32_t f = blockIdx.x; f < nf; f += gridDim.x) {
    const uint32_t q = a.list[f];
    const uint64_t kq = a.key[q];
    bool ok;
    const uint32_t n = members(a, q, ok);
    const uint32_t fq = a.first[q];
    uint32_t rep = q;
    for (uint32_t r = 0; r < q; ++r) {
      bool rok;
      // block-uniform: every thread reads the same entries
      if (a.key[r] != kq || members(a, r, rok) != n || !rok) continue;
      const uint32_t fr = a.first[r];
      bool diff = false;
      for (uint32_t j = threadIdx.x; j < n && !diff; j += blockDim.x)
        diff = a.rs[(int64_t)fq + j] != a.rs[(int64_t)fr + j];
      if (!__syncthreads_or(diff)) {
        rep = r;
        break;
      }
    }
    if (threadIdx.x == 0) a.part_rep[q] = (int32_t)rep;
  }
}

static uint32_t table_mask(uint32_t NP) {
  uint64_t n = 64;
  while (n < 2 * (uint64_t)NP) n <<= 1;
  return (uint32_t)(n - 1);
}

int64_t class_table_slots(uint32_t NP) { return NP ? (int64_t)table_mask(NP) + 1 : 0; }

void run_classes(const opattr_kernels *k, const opattr_dims *d, int32_t *part_rep,
                 opattr_diag *diag, void *ws, const Plan &pl, hipStream_t s) {
  const uint32_t NP = d->n_parts;
  if (NP == 0) return;
  ClsArgs a;
  a.T = pl.T;
  a.sv = at<int32_t>(ws, pl.sv);
  a.name = k->name_id;
  a.stream = k->stream_id;
  a.part = k->part_id;
  a.NN = d->n_names;
  a.NP = NP;
  a.rs = at<uint64_t>(ws, pl.sit);  // the aggregation's item keys: T entries
  a.rp = at<int32_t>(ws, pl.ig);    // the aggregation's item rows: T entries
  a.first = at<uint32_t>(ws, pl.c_first);
  a.last = at<uint32_t>(ws, pl.c_last);
  a.runs = at<uint32_t>(ws, pl.c_runs);
  a.key = at<uint64_t>(ws, pl.c_key);
  a.cand = at<uint32_t>(ws, pl.c_cand);
  a.fail = at<uint32_t>(ws, pl.c_fail);
  a.list = at<uint32_t>(ws, pl.c_list);
  a.nfail = at<uint32_t>(ws, pl.misc);
  a.tkey = at<uint64_t>(ws, pl.c_tkey);
  a.tmin = at<uint32_t>(ws, pl.c_tmin);
  a.tmask = table_mask(NP);
  a.kmask = g_class_key_bits >= 64 ? ~0ull : ((1ull << g_class_key_bits) - 1);
  a.part_rep = part_rep;
  a.diag = diag;
  const int64_t TS = (int64_t)a.tmask + 1;
  FillJobs f;
  f.add(a.runs, 0u, NP);
  f.add(a.key, 0u, 2 * (int64_t)NP);
  f.add(a.fail, 0u, NP);
  f.add(a.tkey, 0u, 2 * TS);
  f.add(a.tmin, 0xFFFFFFFFu, TS);
  f.add(a.nfail, 0u, 1);
  fill_many(f, s);
  const unsigned nbT = (unsigned)((pl.T + 255) / 256), nbP = (NP + 255) / 256;
  probe_begin(OPATTR_PROBE_DEDUP, s);
  if (pl.T > 0) k_cls_runs<<<nbT, 256, 0, s>>>(a);
  k_cls_consecutive<<<nbP, 256, 0, s>>>(a);
  if (pl.T > 0) k_cls_hash<<<nbT, 256, 0, s>>>(a);
  k_cls_insert<<<nbP, 256, 0, s>>>(a);
  k_cls_candidate<<<nbP, 256, 0, s>>>(a);
  if (pl.T > 0) k_cls_verify<<<nbT, 256, 0, s>>>(a);
  k_cls_resolve<<<NP < 256 ? NP : 256, 256, 0, s>>>(a);
  probe_end(OPATTR_PROBE_DEDUP, s);
}

}  // namespace opa
