// Dedup class discovery (Sec. 3.7) on the GPU.
//
// Two partitions are one class when their launches (valid name and
// partition) form the same (name, stream) sequence in launch order; a class
// is represented by its lowest-numbered partition, and a partition whose
// launches are not consecutive in launch order is a class of its own.
//
// Written data-parallel, exact whatever the hash does:
//   1. per partition, in input order: member count and lowest / highest
//      launch-order rank (wave-combined atomics); consecutive iff
//      highest - lowest + 1 = count;
//   2. member offsets of the consecutive partitions (exclusive scan);
//   3. every member stores its packed (name, stream) at offset + position
//      and adds a position-keyed 64-bit hash of it to its partition's key;
//   4. key -> lowest partition with that key (open-addressing table): the
//      candidate representative, never above the true one (equal sequences
//      have equal keys);
//   5. members of a partition compare their element with the candidate's
//      element at the same position: with no difference the candidate is the
//      representative;
//   6. partitions that differ from their candidate (a key collision) search
//      exactly: the lowest-numbered partition with their key and sequence.
#include "common.h"
#include "impl.h"

namespace opa {

struct ClsArgs {
  int64_t T;
  const uint32_t *seq;
  const int32_t *rk;  // launch-order rank per input index; NULL: seq is the rank
  const uint32_t *name;
  const uint16_t *stream;
  const int32_t *part;
  uint32_t NN, NP;
  uint32_t *cnt, *lo, *hi;  // [NP] members, lowest and highest rank
  uint32_t *cc, *off;       // [NP] members of consecutive partitions, their offsets
  uint64_t *key;            // [NP] hash of the sequence, then with the count folded in
  uint32_t *cand, *fail;    // [NP] candidate representative, differs from it
  uint32_t *list, *nfail;   // partitions that differ from their candidate
  uint64_t *tkey;           // [tmask + 1] table keys (0 = empty)
  uint32_t *tmin;           // [tmask + 1] lowest partition with the key
  uint32_t tmask;
  uint64_t kmask;           // bits of the key kept (all but in tests of the exact search)
  uint64_t *packed;         // [members] (name << 16 | stream) by partition and position
  uint32_t *pid;            // [members] partition of the element
  const int64_t *total;     // members of consecutive partitions
  int32_t *part_rep;
  opattr_diag *diag;
};

// splitmix64's output function (Steele, Lea and Flood, 2014)
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t elem_hash(uint64_t packed, uint32_t pos) {
  return mix64(packed + 0x9E3779B97F4A7C15ull * ((uint64_t)pos + 1));
}

__device__ __forceinline__ bool consecutive(const ClsArgs &a, uint32_t q) {
  const uint32_t c = a.cnt[q];
  return c == 0 || (uint64_t)a.hi[q] - a.lo[q] + 1 == c;
}

// A launch that belongs to a partition: its partition, else -1 (bad ids
// counted by the caller). rank gets its launch-order rank.
__device__ __forceinline__ int32_t member_of(const ClsArgs &a, int64_t i, bool &bad,
                                             uint32_t &rank) {
  const uint32_t nm = a.name[i];
  const int32_t p = a.part[i];
  bad = nm >= a.NN || p < -1 || (p >= 0 && (uint32_t)p >= a.NP);
  if (bad || p < 0) return -1;
  rank = a.rk ? (uint32_t)a.rk[i] : a.seq[i];
  return p;
}

__device__ __forceinline__ void mark_fail(const ClsArgs &a, uint32_t q) {
  if (atomicOr(&a.fail[q], 1u) == 0u) a.list[atomicAdd(a.nfail, 1u)] = q;
}

template <typename F>
__device__ __forceinline__ uint32_t wave_fold_u32(uint32_t x, F f) {
#pragma unroll
  for (int o = OPA_WAVE / 2; o > 0; o >>= 1) x = f(x, (uint32_t)__shfl_xor((int)x, o, OPA_WAVE));
  return x;
}

// 1. members, lowest and highest rank per partition; bad ids counted
__global__ void __launch_bounds__(256) k_cls_stats(ClsArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  uint32_t r = 0;
  const int32_t p = i < a.T ? member_of(a, i, bad, r) : -1;
  const uint64_t mb = __ballot(bad);
  if (mb && lane_id() == __ffsll((unsigned long long)mb) - 1)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)__popcll(mb));
  const int32_t p0 = __shfl(p, 0, OPA_WAVE);
  if (p0 >= 0 && __all(p == p0)) {  // the whole wave in one partition
    const uint32_t mn = wave_fold_u32(r, [](uint32_t x, uint32_t y) { return x < y ? x : y; });
    const uint32_t mx = wave_fold_u32(r, [](uint32_t x, uint32_t y) { return x > y ? x : y; });
    if (lane_id() == 0) {
      atomicAdd(&a.cnt[p0], (uint32_t)OPA_WAVE);
      atomicMin(&a.lo[p0], mn);
      atomicMax(&a.hi[p0], mx);
    }
  } else if (p >= 0) {
    atomicAdd(&a.cnt[p], 1u);
    atomicMin(&a.lo[p], r);
    atomicMax(&a.hi[p], r);
  }
}

// 2. scan input: members of consecutive partitions; PARTITION for the others
__global__ void k_cls_consecutive(ClsArgs a) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  bool nc = false;
  if (q < a.NP) {
    const bool ok = consecutive(a, q);
    a.cc[q] = ok ? a.cnt[q] : 0u;
    nc = !ok;
  }
  if (__ballot(nc) && lane_id() == 0) atomicOr(&a.diag->flags, OPATTR_F_PARTITION);
}

// 3. elements by partition and position, and the sequence hash
__global__ void __launch_bounds__(256) k_cls_place(ClsArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  uint32_t r = 0;
  int32_t p = i < a.T ? member_of(a, i, bad, r) : -1;
  uint64_t h = 0;
  if (p >= 0) {
    if (consecutive(a, (uint32_t)p)) {
      const uint32_t pos = r - a.lo[p];
      const int64_t e = (int64_t)a.off[p] + pos;
      const uint64_t v = ((uint64_t)a.name[i] << 16) | a.stream[i];
      a.packed[e] = v;
      a.pid[e] = (uint32_t)p;
      h = elem_hash(v, pos);
    } else {
      p = -1;
    }
  }
  const int32_t p0 = __shfl(p, 0, OPA_WAVE);
  if (p0 >= 0 && __all(p == p0)) {
    const uint64_t s = wave_reduce_add(h);
    if (lane_id() == 0) atomicAdd((unsigned long long *)&a.key[p0], (unsigned long long)s);
  } else if (p >= 0) {
    atomicAdd((unsigned long long *)&a.key[p], (unsigned long long)h);
  }
}

__device__ __forceinline__ uint32_t table_home(uint64_t k, uint32_t mask) {
  return (uint32_t)(k ^ (k >> 32)) & mask;
}

// 4a. key with the count folded in, into the table with the lowest partition
__global__ void k_cls_insert(ClsArgs a) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= a.NP || !consecutive(a, q)) return;
  uint64_t k = mix64(a.key[q] ^ mix64((uint64_t)a.cnt[q] + 0x632BE59BD9B4E019ull)) & a.kmask;
  if (k == 0) k = 1;
  a.key[q] = k;
  uint32_t slot = table_home(k, a.tmask);
  // the table has at least twice as many slots as partitions: a slot that
  // is empty or holds k is reached within tmask + 1 probes
  for (uint32_t it = 0; it <= a.tmask; ++it) {
    const unsigned long long prev =
        atomicCAS((unsigned long long *)&a.tkey[slot], 0ull, (unsigned long long)k);
    if (prev == 0ull || prev == k) {
      atomicMin(&a.tmin[slot], q);
      return;
    }
    slot = (slot + 1) & a.tmask;
  }
}

// 4b. candidate representative; a count that differs is a collision
__global__ void k_cls_candidate(ClsArgs a) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= a.NP) return;
  uint32_t c = q;
  if (consecutive(a, q)) {
    const uint64_t k = a.key[q];
    uint32_t slot = table_home(k, a.tmask);
    for (uint32_t it = 0; it <= a.tmask; ++it) {
      if (a.tkey[slot] == k) {
        c = a.tmin[slot];
        break;
      }
      slot = (slot + 1) & a.tmask;
    }
    if (c != q && a.cnt[c] != a.cnt[q]) mark_fail(a, q);
  }
  a.cand[q] = c;
  a.part_rep[q] = (int32_t)c;
}

// 5. element-wise comparison with the candidate
__global__ void __launch_bounds__(256) k_cls_verify(ClsArgs a) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= *a.total) return;
  const uint32_t q = a.pid[e];
  if (q >= a.NP) return;  // only when a dense-seq promise was false: holes stay stale
  const uint32_t c = a.cand[q];
  if (c == q || a.cnt[c] != a.cnt[q]) return;
  const uint32_t off_q = a.off[q];
  if (a.packed[e] != a.packed[(int64_t)a.off[c] + (e - off_q)]) mark_fail(a, q);
}

// 6. exact search for the partitions that differ from their candidate: the
// lowest-numbered consecutive partition with the same key and sequence
// (itself when none). One block per such partition, striding.
__global__ void __launch_bounds__(256) k_cls_resolve(ClsArgs a) {
  const uint32_t nf = *a.nfail;
  for (uint32_t f = blockIdx.x; f < nf; f += gridDim.x) {
    const uint32_t q = a.list[f];
    const uint64_t kq = a.key[q];
    const uint32_t c = a.cnt[q], oq = a.off[q];
    uint32_t rep = q;
    for (uint32_t r = 0; r < q; ++r) {
      if (a.key[r] != kq || a.cnt[r] != c || !consecutive(a, r)) continue;  // block-uniform
      const uint32_t orr = a.off[r];
      bool diff = false;
      for (uint32_t j = threadIdx.x; j < c && !diff; j += blockDim.x)
        diff = a.packed[(int64_t)oq + j] != a.packed[(int64_t)orr + j];
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
  a.seq = k->seq;
  a.rk = pl.seq_dense ? nullptr : at<int32_t>(ws, pl.rk);
  a.name = k->name_id;
  a.stream = k->stream_id;
  a.part = k->part_id;
  a.NN = d->n_names;
  a.NP = NP;
  a.cnt = at<uint32_t>(ws, pl.c_cnt);
  a.lo = at<uint32_t>(ws, pl.c_lo);
  a.hi = at<uint32_t>(ws, pl.c_hi);
  a.cc = at<uint32_t>(ws, pl.c_cc);
  a.off = at<uint32_t>(ws, pl.c_off);
  a.key = at<uint64_t>(ws, pl.c_key);
  a.cand = at<uint32_t>(ws, pl.c_cand);
  a.fail = at<uint32_t>(ws, pl.c_fail);
  a.list = at<uint32_t>(ws, pl.c_list);
  a.nfail = at<uint32_t>(ws, pl.misc);
  a.tkey = at<uint64_t>(ws, pl.c_tkey);
  a.tmin = at<uint32_t>(ws, pl.c_tmin);
  a.tmask = table_mask(NP);
  a.kmask = g_class_key_bits >= 64 ? ~0ull : ((1ull << g_class_key_bits) - 1);
  a.packed = at<uint64_t>(ws, pl.sit);  // the aggregation's item keys: T entries
  a.pid = at<uint32_t>(ws, pl.ig);      // the aggregation's item rows: T entries
  a.total = at<int64_t>(ws, pl.misc + 8);
  a.part_rep = part_rep;
  a.diag = diag;
  const int64_t TS = (int64_t)a.tmask + 1;
  FillJobs f;
  f.add(a.cnt, 0u, NP);
  f.add(a.lo, 0xFFFFFFFFu, NP);
  f.add(a.hi, 0u, NP);
  f.add(a.key, 0u, 2 * (int64_t)NP);
  f.add(a.fail, 0u, NP);
  f.add(a.tkey, 0u, 2 * TS);
  f.add(a.tmin, 0xFFFFFFFFu, TS);
  f.add(at<uint32_t>(ws, pl.misc), 0u, 4);  // nfail, total
  fill_many(f, s);
  const unsigned nbT = (unsigned)((pl.T + 255) / 256), nbP = (NP + 255) / 256;
  probe_begin(OPATTR_PROBE_DEDUP, s);
  if (pl.T > 0) k_cls_stats<<<nbT, 256, 0, s>>>(a);
  k_cls_consecutive<<<nbP, 256, 0, s>>>(a);
  launch_scan_excl(a.cc, a.off, NP, at<int64_t>(ws, pl.misc + 8), s);
  if (pl.T > 0) k_cls_place<<<nbT, 256, 0, s>>>(a);
  k_cls_insert<<<nbP, 256, 0, s>>>(a);
  k_cls_candidate<<<nbP, 256, 0, s>>>(a);
  if (pl.T > 0) k_cls_verify<<<nbT, 256, 0, s>>>(a);
  k_cls_resolve<<<NP < 256 ? NP : 256, 256, 0, s>>>(a);
  probe_end(OPATTR_PROBE_DEDUP, s);
}

}  // namespace opa
