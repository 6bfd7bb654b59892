// All enclosing ranges of every launch (Alg. 2's all_enclosing) as CSR lists,
// innermost first: the innermost range of every launch (the enclosure pass),
// a count pass, an inclusive scan of the counts into the offsets, and a fill
// pass that writes the lists within the caller's capacity. From the innermost
// range each launch walks outward through every range containing its query
// point: the parent, or, from a range starting at the point, the nearest
// earlier range in nesting order that ends at or after it (closed
// intervals).
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
  const int32_t *core;  // innermost range of each launch (core position, -1: none)
  int64_t *off;         // [T + 1]
  int32_t *ids;
  int64_t cap;
  opattr_diag *diag;
};

__device__ __forceinline__ int64_t next_out(const AllArgs &a, int64_t j, int64_t slo, uint64_t q) {
  if ((uint64_t)a.cr.s[j] != q) return a.npg[j];
  int64_t c = j - 1;
  for (int h = 0; c >= slo && a.ree[c] < (int64_t)q && h < kMaxWalk; ++h) c = a.npg[c];
  return c >= slo ? c : -1;
}

__global__ void __launch_bounds__(256) k_all_count(AllArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < a.T) {
    const int64_t j0 = a.core[i];
    int64_t n = 0;
    if (j0 >= 0) {
      const int64_t slo = a.rblk[a.stream[i]];
      const uint64_t q = a.q[i];
      for (int64_t j = j0; j >= 0 && n < kMaxWalk; j = next_out(a, j, slo, q)) ++n;
    }
    a.off[i + 1] = n;
  }
  if (i == 0) a.off[0] = 0;
}

__global__ void __launch_bounds__(256) k_all_fill(AllArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.T) return;
  const int64_t o = a.off[i], e = a.off[i + 1];
  if (e > a.cap || e == o) return;
  const int64_t slo = a.rblk[a.stream[i]];
  const uint64_t q = a.q[i];
  int64_t n = 0;
  for (int64_t j = a.core[i]; j >= 0 && o + n < e; j = next_out(a, j, slo, q)) {
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
  // the innermost ranges by the enclosure pass (LDS window of range starts,
  // searches continued along each stream); the item rows hold them
  int32_t *core = at<int32_t>(ws, pl.ig);
  launch_innermost(cr, k, d, ws, pl, core, diag, s);
  a.core = core;
  k_all_count<<<nb, 256, 0, s>>>(a);
  scan_incl_i64_inplace(off + 1, pl.T, at<int64_t>(ws, pl.sv), s);
  if (cap > 0) k_all_fill<<<nb, 256, 0, s>>>(a);
}

}  // namespace opa
