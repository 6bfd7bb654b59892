// Tiered attribution (the attribution-methods table and the decision-tree
// figure) on the GPU.
//
// The correlation lookup is Alg. 1 with the correlation map's entries as the
// rows (run by the matching kernels, partitions off), which leaves each
// launch the index of its entry. One pass over the launches then takes the
// first tier that applies -- HIGH (an entry with a valid operator), NVTX
// (the enclosure walk's op range), FUSION (the first operator the fusion map
// lists for the kernel name), else UNATTRIBUTED -- marks the kernel fused
// when the walk collected several op ranges or the fusion map lists several
// operators, and sums kernels and nanoseconds per tier: a fixed grid
// strides over the launches with the sums in registers, each block writes
// its eight partial sums, and one block adds them up (atomics on eight hot
// addresses would serialise at a few ns each).
#include "common.h"
#include "impl.h"

namespace opa {

struct TierArgs {
  int64_t T;
  const uint32_t *name;
  const uint32_t *dur;
  const int32_t *entry;  // correlation entry of each launch (-1 none); NULL: no map
  const int32_t *corr_op;
  int64_t C;
  const int32_t *range_id;
  const uint8_t *walk_fused;  // optional
  int64_t R;
  const uint32_t *r_op;
  const uint32_t *f_off;  // fusion map, optional
  const int32_t *f_op;
  uint32_t NN, NOPS;
  uint8_t *tier;
  int32_t *op;
  uint8_t *fused;
  unsigned long long *part;  // [blocks][8]: kernels per tier, then ns per tier
  opattr_diag *diag;
};

constexpr int kTierBlocks = 1024;  // grid of the tier pass (4 blocks per CU)

// correlation entries with an operator outside [-1, n_ops) are bad records
__global__ void k_corr_bad(const int32_t *__restrict__ corr_op, int64_t C, uint32_t NOPS,
                           opattr_diag *diag) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (j < C) {
    const int32_t o = corr_op[j];
    bad = o < -1 || (o >= 0 && (uint32_t)o >= NOPS);
  }
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
    atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)__popcll(m));
}

constexpr int kTierPer = 4;  // launches per thread per step, their loads in flight together

// Tier, operator and fused of kTierPer launches (x[k] < 0: none): every load
// of one level for all of them before the next level (coalesced fields;
// the fusion list bounds, the entry's and the range's operators; the first
// fused operator), then the stores. Returns the tiers (-1: none).
__device__ __forceinline__ void tiers_of(const TierArgs &a, const int64_t (&x)[kTierPer],
                                         int (&t)[kTierPer], uint32_t (&d)[kTierPer],
                                         uint32_t &bad) {
  uint32_t nm[kTierPer];
  int32_t e[kTierPer], rid[kTierPer];
  uint8_t wf[kTierPer];
#pragma unroll
  for (int k = 0; k < kTierPer; ++k) {
    const bool v = x[k] >= 0;
    nm[k] = v ? a.name[x[k]] : 0xFFFFFFFFu;
    e[k] = (v && a.entry) ? a.entry[x[k]] : -1;
    rid[k] = v ? a.range_id[x[k]] : -1;
    d[k] = v ? a.dur[x[k]] : 0u;
    wf[k] = (v && a.walk_fused) ? a.walk_fused[x[k]] : 0;
  }
  uint32_t f0[kTierPer], nf[kTierPer];
  int32_t co[kTierPer], ro[kTierPer];
#pragma unroll
  for (int k = 0; k < kTierPer; ++k) {
    f0[k] = 0;
    nf[k] = 0;
    if (a.f_off && nm[k] < a.NN) {
      const uint32_t lo = a.f_off[nm[k]], hi = a.f_off[nm[k] + 1];
      if (hi > lo) {
        f0[k] = lo;
        nf[k] = hi - lo;
      }
    }
    co[k] = (e[k] >= 0 && e[k] < a.C) ? a.corr_op[e[k]] : -1;
    ro[k] = (rid[k] >= 0 && (int64_t)rid[k] < a.R) ? (int32_t)a.r_op[rid[k]] : -1;
  }
  int32_t fo[kTierPer];
#pragma unroll
  for (int k = 0; k < kTierPer; ++k) fo[k] = nf[k] > 0 ? a.f_op[f0[k]] : -1;
#pragma unroll
  for (int k = 0; k < kTierPer; ++k) {
    t[k] = -1;
    if (x[k] < 0) continue;
    if (rid[k] < -1 || (int64_t)rid[k] >= a.R) bad++;
    int tk = OPATTR_TIER_UNATTRIBUTED;
    int32_t o = -1;
    if (co[k] >= 0 && (uint32_t)co[k] < a.NOPS) {
      tk = OPATTR_TIER_HIGH;
      o = co[k];
    } else if (rid[k] >= 0 && (int64_t)rid[k] < a.R) {
      tk = OPATTR_TIER_NVTX;
      o = ro[k];
    } else if (nf[k] > 0 && fo[k] >= 0 && (uint32_t)fo[k] < a.NOPS) {
      tk = OPATTR_TIER_FUSION;
      o = fo[k];
    }
    a.tier[x[k]] = (uint8_t)tk;
    a.op[x[k]] = o;
    a.fused[x[k]] = (uint8_t)((wf[k] || nf[k] > 1) ? 1 : 0);
    t[k] = tk;
  }
}

__global__ void __launch_bounds__(256) k_tiers(TierArgs a) {
  __shared__ unsigned long long red[4][8];
  uint32_t cnt[4] = {0, 0, 0, 0}, bad = 0;
  unsigned long long ns[4] = {0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.T;
       i += stride * kTierPer) {
    int64_t x[kTierPer];
#pragma unroll
    for (int k = 0; k < kTierPer; ++k) x[k] = i + k * stride < a.T ? i + k * stride : -1;
    int t[kTierPer];
    uint32_t d[kTierPer];
    tiers_of(a, x, t, d, bad);
#pragma unroll
    for (int k = 0; k < kTierPer; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        cnt[q] += t[k] == q ? 1u : 0u;
        ns[q] += t[k] == q ? d[k] : 0u;
      }
  }
  const uint32_t bw = wave_reduce_add(bad);
  if (lane_id() == 0 && bw)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)bw);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const unsigned long long c = wave_reduce_add<unsigned long long>(cnt[q]);
    const unsigned long long n = wave_reduce_add(ns[q]);
    if (lane_id() == 0) {
      red[wave_id()][q] = c;
      red[wave_id()][4 + q] = n;
    }
  }
  __syncthreads();
  if (threadIdx.x < 8) {
    unsigned long long v = 0;
    for (int w = 0; w < 4; ++w) v += red[w][threadIdx.x];
    a.part[(int64_t)blockIdx.x * 8 + threadIdx.x] = v;
  }
}

// the per-block sums added up (one block), and the coverage record
__global__ void __launch_bounds__(256) k_cov_finish(const unsigned long long *part, int nblocks,
                                                    opattr_coverage *cov) {
  __shared__ unsigned long long red[4][8];
  unsigned long long v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int b = threadIdx.x; b < nblocks; b += blockDim.x)
#pragma unroll
    for (int f = 0; f < 8; ++f) v[f] += part[(int64_t)b * 8 + f];
#pragma unroll
  for (int f = 0; f < 8; ++f) {
    const unsigned long long r = wave_reduce_add(v[f]);
    if (lane_id() == 0) red[wave_id()][f] = r;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  opattr_coverage c;
  uint64_t total = 0;
  for (int f = 0; f < 8; ++f) v[f] = red[0][f] + red[1][f] + red[2][f] + red[3][f];
  for (int q = 0; q < 4; ++q) {
    c.count[q] = v[q];
    c.ns[q] = v[4 + q];
    total += v[4 + q];
  }
  for (int q = 0; q < 4; ++q)
    c.frac[q] = total ? (double)c.ns[q] / (double)total
                      : __longlong_as_double(0x7FF8000000000000ll);
  *cov = c;
}

// Per-dispatch key of each launch: its range when its operator (op[i], or
// the range's own op when op is NULL) is the range's operator, else R + its
// operator, else -1 (the last row, unattributed). Bad range ids and
// operators are counted.
// four consecutive int32 from p + i (one 16-byte load when aligned); nv of them valid
__device__ __forceinline__ void load4(const int32_t *p, int64_t i, int nv, int32_t (&o)[4]) {
  if (nv == 4 && (reinterpret_cast<uintptr_t>(p + i) & 15) == 0) {
    const int4 v = *reinterpret_cast<const int4 *>(p + i);
    o[0] = v.x;
    o[1] = v.y;
    o[2] = v.z;
    o[3] = v.w;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = k < nv ? p[i + k] : -1;
  }
}

__device__ __forceinline__ void store4(int32_t *p, int64_t i, int nv, const int32_t (&v)[4]) {
  if (nv == 4 && (reinterpret_cast<uintptr_t>(p + i) & 15) == 0) {
    *reinterpret_cast<int4 *>(p + i) = make_int4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (k < nv) p[i + k] = v[k];
  }
}

// four launches per thread
__global__ void k_dispatch_keys(const int32_t *__restrict__ range_id, const int32_t *__restrict__ op,
                                const uint32_t *__restrict__ r_op, int64_t R, uint32_t NOPS,
                                int64_t T, int32_t *key, int32_t *row, opattr_diag *diag) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  uint32_t bad = 0;
  if (i < T) {
    const int nv = T - i < 4 ? (int)(T - i) : 4;
    int32_t rid[4], o[4], ky[4], rw[4];
    load4(range_id, i, nv, rid);
    if (op) load4(op, i, nv, o);
    uint32_t ro[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bool rok = k < nv && rid[k] >= 0 && (int64_t)rid[k] < R;
      ro[k] = rok ? r_op[rid[k]] : 0xFFFFFFFFu;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (k >= nv) continue;
      const bool rok = rid[k] >= 0 && (int64_t)rid[k] < R;
      const int32_t ok_ = op ? o[k] : (rok ? (int32_t)ro[k] : -1);
      if (rid[k] < -1 || (int64_t)rid[k] >= R) bad++;
      if (op && (ok_ < -1 || (ok_ >= 0 && (uint32_t)ok_ >= NOPS))) bad++;
      const bool ook = ok_ >= 0 && (uint32_t)ok_ < NOPS;
      int64_t kk = -1;  // the last row, as an unattributed operator
      if (rok && ook && (uint32_t)ok_ == ro[k]) kk = rid[k];
      else if (ook) kk = R + ok_;
      ky[k] = (int32_t)kk;
      rw[k] = (int32_t)(kk >= 0 ? kk : R + NOPS);
    }
    store4(key, i, nv, ky);
    if (row) store4(row, i, nv, rw);
  }
  const uint32_t b = wave_reduce_add(bad);
  if (lane_id() == 0 && b) atomicAdd((unsigned long long *)&diag->bad_records, (unsigned long long)b);
}

void launch_dispatch_keys(const int32_t *range_id, const int32_t *op, const opattr_ranges *r,
                          uint32_t NOPS, int64_t T, int32_t *key, int32_t *row,
                          opattr_diag *diag, hipStream_t s) {
  if (T > 0)
    k_dispatch_keys<<<(unsigned)((T + 1023) / 1024), 256, 0, s>>>(range_id, op, r->op_id, r->n,
                                                                  NOPS, T, key, row, diag);
}

void run_tiers(const TierIn &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  const int64_t want = (pl.T + 255) / 256;
  const int nb = want < 1 ? 1 : (want < kTierBlocks ? (int)want : kTierBlocks);
  // partial sums: the aggregation's item rows (T 4-byte entries) hold them
  // when T >= 2 * 8 * nb, else the small scalars
  unsigned long long *part = pl.T >= 16 * (int64_t)nb ? at<unsigned long long>(x.ws, pl.ib)
                                                       : at<unsigned long long>(x.ws, pl.misc);
  if (x.corr && x.corr->n > 0)
    k_corr_bad<<<(unsigned)((x.corr->n + 255) / 256), 256, 0, s>>>(x.corr->op_id, x.corr->n,
                                                                   x.d->n_ops, x.diag);
  TierArgs a;
  a.T = pl.T;
  a.name = x.k->name_id;
  a.dur = x.k->dur_ns;
  a.entry = x.entry;
  a.corr_op = x.corr ? x.corr->op_id : nullptr;
  a.C = x.corr ? x.corr->n : 0;
  a.range_id = x.range_id;
  a.walk_fused = x.walk_fused;
  a.R = x.r->n;
  a.r_op = x.r->op_id;
  a.f_off = x.fmap ? x.fmap->off : nullptr;
  a.f_op = x.fmap ? x.fmap->op_id : nullptr;
  a.NN = x.d->n_names;
  a.NOPS = x.d->n_ops;
  a.tier = x.tier;
  a.op = x.op;
  a.fused = x.fused;
  a.part = part;
  a.diag = x.diag;
  k_tiers<<<nb, 256, 0, s>>>(a);
  k_cov_finish<<<1, 256, 0, s>>>(part, nb, x.cov);
}

}  // namespace opa
