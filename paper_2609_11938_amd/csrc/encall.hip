// All enclosing ranges of every launch (Alg. 2's all_enclosing) as CSR lists,
// innermost first: a count pass, an inclusive scan of the counts into the
// offsets, and a fill pass that writes the lists within the caller's
// capacity. Each launch finds its innermost range by a binary search over its
// stream's range starts (nesting order) and the lifting of Alg. 2, then walks
// outward through every range containing its query point: the parent, or,
// from a range starting at the point, the nearest earlier range in nesting
// order that ends at or after it (closed intervals).
#include "common.h"
#include "impl.h"

namespace opa {

struct AllArgs {
  int64_t T;
  const uint64_t *q;
  const uint16_t *stream;
  CoreRanges cr;
  const int64_t *rblk;
  const int64_t *ree;
  const int32_t *npg;
  uint32_t NS;
  int64_t *off;  // [T + 1]
  int32_t *ids;
  int64_t cap;
  opattr_diag *diag;
};

// innermost range (core position) containing the launch's point, or -1;
// slo = the first range of its stream
__device__ __forceinline__ int64_t innermost(const AllArgs &a, int64_t i, int64_t &slo,
                                             uint64_t &q, bool &bad) {
  const uint16_t st = a.stream[i];
  q = a.q[i];
  bad = st >= a.NS;
  if (bad || q >= (1ull << 63)) return -1;
  const int64_t lo = a.rblk[st], hi = a.rblk[st + 1];
  slo = lo;
  int64_t l = lo, h = hi;  // first start > q
  while (l < h) {
    const int64_t m = (l + h) >> 1;
    if (a.cr.s[m] <= q) l = m + 1;
    else h = m;
  }
  int64_t j = l - 1;
  for (int s = 0; j >= lo && a.ree[j] < (int64_t)q && s < kMaxWalk; ++s) j = a.npg[j];
  return (j >= lo && a.ree[j] >= (int64_t)q) ? j : -1;
}

__device__ __forceinline__ int64_t next_out(const AllArgs &a, int64_t j, int64_t slo, uint64_t q) {
  if ((uint64_t)a.cr.s[j] != q) return a.npg[j];
  int64_t c = j - 1;
  for (int h = 0; c >= slo && a.ree[c] < (int64_t)q && h < kMaxWalk; ++h) c = a.npg[c];
  return c >= slo ? c : -1;
}

__global__ void __launch_bounds__(256) k_all_count(AllArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (i < a.T) {
    int64_t slo = 0;
    uint64_t q = 0;
    int64_t n = 0;
    for (int64_t j = innermost(a, i, slo, q, bad); j >= 0 && n < kMaxWalk; j = next_out(a, j, slo, q))
      ++n;
    a.off[i + 1] = n;
  }
  if (i == 0) a.off[0] = 0;
  const uint64_t m = __ballot(bad);
  if (m && lane_id() == __ffsll((unsigned long long)m) - 1)
    atomicAdd((unsigned long long *)&a.diag->bad_records, (unsigned long long)__popcll(m));
}

__global__ void __launch_bounds__(256) k_all_fill(AllArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.T) return;
  const int64_t o = a.off[i], e = a.off[i + 1];
  if (e > a.cap) return;
  int64_t slo = 0;
  uint64_t q = 0;
  bool bad;
  int64_t n = 0;
  for (int64_t j = innermost(a, i, slo, q, bad); j >= 0 && o + n < e; j = next_out(a, j, slo, q)) {
    a.ids[o + n] = a.cr.perm ? a.cr.perm[j] : (int32_t)j;
    ++n;
  }
}

void run_enclose_all(const CoreRanges &cr, const opattr_kernels *k, const opattr_dims *d, void *ws,
                     const Plan &pl, int64_t *off, int32_t *ids, int64_t cap, opattr_diag *diag,
                     hipStream_t s) {
  AllArgs a;
  a.T = pl.T;
  a.q = k->query_ns ? k->query_ns : k->start_ns;
  a.stream = k->stream_id;
  a.cr = cr;
  a.rblk = at<int64_t>(ws, pl.rblk);
  a.ree = at<int64_t>(ws, pl.ree);
  a.npg = at<int32_t>(ws, pl.npg);
  a.NS = d->n_streams;
  a.off = off;
  a.ids = ids;
  a.cap = cap;
  a.diag = diag;
  const unsigned nb = (unsigned)((pl.T + 255) / 256);
  if (pl.T <= 0) {
    fill_u32(reinterpret_cast<uint32_t *>(off), 0u, 2, s);
    return;
  }
  k_all_count<<<nb, 256, 0, s>>>(a);
  scan_incl_i64_inplace(off + 1, pl.T, at<int64_t>(ws, pl.sv), s);
  if (cap > 0) k_all_fill<<<nb, 256, 0, s>>>(a);
}

}  // namespace opa
