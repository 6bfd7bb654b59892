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
// operators, and sums kernels and nanoseconds per tier: wave reductions,
// one LDS atomic per wave and tier, one global atomic per block and tier.
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
  unsigned long long *acc;  // [8]: kernels per tier, then ns per tier
  opattr_diag *diag;
};

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

__global__ void __launch_bounds__(256) k_tiers(TierArgs a) {
  __shared__ unsigned long long sacc[8];
  if (threadIdx.x < 8) sacc[threadIdx.x] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool live = i < a.T;
  int t = OPATTR_TIER_UNATTRIBUTED;
  uint64_t d = 0;
  bool bad = false;
  if (live) {
    const uint32_t nm = a.name[i];
    d = a.dur[i];
    const int32_t e = a.entry ? a.entry[i] : -1;
    const int32_t rid = a.range_id[i];
    bad = rid < -1 || (int64_t)rid >= a.R;
    uint32_t f0 = 0, nf = 0;  // the kernel name's fusion list
    if (a.f_off && nm < a.NN) {
      const uint32_t lo = a.f_off[nm], hi = a.f_off[nm + 1];
      if (hi > lo) {
        f0 = lo;
        nf = hi - lo;
      }
    }
    const int32_t co = (e >= 0 && e < a.C) ? a.corr_op[e] : -1;
    int32_t o = -1;
    if (co >= 0 && (uint32_t)co < a.NOPS) {
      t = OPATTR_TIER_HIGH;
      o = co;
    } else if (rid >= 0 && (int64_t)rid < a.R) {
      t = OPATTR_TIER_NVTX;
      o = (int32_t)a.r_op[rid];
    } else if (nf > 0) {
      const int32_t fo = a.f_op[f0];
      if (fo >= 0 && (uint32_t)fo < a.NOPS) {
        t = OPATTR_TIER_FUSION;
        o = fo;
      }
    }
    a.tier[i] = (uint8_t)t;
    a.op[i] = o;
    a.fused[i] = (uint8_t)(((a.walk_fused && a.walk_fused[i]) || nf > 1) ? 1 : 0);
  }
  const uint64_t mb = __ballot(bad);
  if (mb && lane_id() == __ffsll((unsigned long long)mb) - 1)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)__popcll(mb));
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool in = live && t == q;
    const uint64_t c = (uint64_t)__popcll(__ballot(in));
    const uint64_t ns = wave_reduce_add<uint64_t>(in ? d : 0);
    if (lane_id() == 0 && c) {
      atomicAdd(&sacc[q], (unsigned long long)c);
      atomicAdd(&sacc[4 + q], (unsigned long long)ns);
    }
  }
  __syncthreads();
  if (threadIdx.x < 8 && sacc[threadIdx.x]) atomicAdd(&a.acc[threadIdx.x], sacc[threadIdx.x]);
}

__global__ void k_cov_finish(const unsigned long long *acc, opattr_coverage *cov) {
  if (threadIdx.x != 0) return;
  opattr_coverage c;
  uint64_t total = 0;
  for (int q = 0; q < 4; ++q) {
    c.count[q] = acc[q];
    c.ns[q] = acc[4 + q];
    total += acc[4 + q];
  }
  for (int q = 0; q < 4; ++q)
    c.frac[q] = total ? (double)c.ns[q] / (double)total
                      : __longlong_as_double(0x7FF8000000000000ll);
  *cov = c;
}

void run_tiers(const TierIn &x, hipStream_t s) {
  const Plan &pl = *x.pl;
  unsigned long long *acc = at<unsigned long long>(x.ws, pl.misc);
  fill_u32(reinterpret_cast<uint32_t *>(acc), 0u, 16, s);
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
  a.acc = acc;
  a.diag = x.diag;
  if (pl.T > 0) k_tiers<<<(unsigned)((pl.T + 255) / 256), 256, 0, s>>>(a);
  k_cov_finish<<<1, 64, 0, s>>>(acc, x.cov);
}

}  // namespace opa
