// Stable LSD radix sort of (u64 key, u32 value) pairs, 8-bit digits.
// Each pass: per-tile digit histograms -> one exclusive scan in digit-major
// order -> a scatter that ranks equal digits stably inside the tile with
// wave ballots (per-digit peer masks) and per-(chunk, wave) counts in LDS.
#include "common.h"
#include "impl.h"

namespace opa {

// n_dev (optional): the element count on the device, at most n; tiles past it
// count nothing and move nothing
__device__ __forceinline__ int64_t sort_count(int64_t n, const int64_t *n_dev) {
  if (!n_dev) return n;
  const int64_t m = *n_dev;
  return m < n ? (m > 0 ? m : 0) : n;
}

__global__ void __launch_bounds__(256) k_rs_hist(const uint32_t *__restrict__ keys, int64_t n_cap,
                                                 const int64_t *n_dev, int shift,
                                                 uint32_t *__restrict__ hist, int64_t ntiles) {
  __shared__ uint32_t c[256];
  c[threadIdx.x] = 0;
  __syncthreads();
  const int64_t n = sort_count(n_cap, n_dev);
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  for (int i = threadIdx.x; i < OPA_TILE; i += 256) {
    const int64_t x = base + i;
    if (x < n) atomicAdd(&c[(keys[x] >> shift) & 255u], 1u);
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = c[threadIdx.x];
}

// Exclusive scan of in[0..n) into out (in place when they are the same) by
// one block of 1024 threads, 16 consecutive elements per thread per round
// (loads of a round in flight together, 16-byte vectors when aligned);
// returns the total to every thread.
constexpr int kScanPer = 16;
__device__ inline uint32_t block_scan_rounds(const uint32_t *in, uint32_t *out, int64_t n) {
  __shared__ uint32_t sh[16];
  uint32_t carry = 0;
  const bool vec = ((reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out)) & 15) == 0;
  for (int64_t base = 0; base < n; base += (int64_t)1024 * kScanPer) {
    const int64_t x0 = base + (int64_t)threadIdx.x * kScanPer;
    const bool whole = vec && x0 + kScanPer <= n;
    uint32_t v[kScanPer];
    if (whole) {
      const uint4 *p = reinterpret_cast<const uint4 *>(in + x0);
#pragma unroll
      for (int q = 0; q < kScanPer / 4; ++q) {
        const uint4 t = p[q];
        v[4 * q] = t.x;
        v[4 * q + 1] = t.y;
        v[4 * q + 2] = t.z;
        v[4 * q + 3] = t.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; ++j) v[j] = x0 + j < n ? in[x0 + j] : 0u;
    }
    uint32_t s = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) s += v[j];
    uint32_t tot;
    uint32_t run = carry + block_excl_scan_add<uint32_t>(s, sh, &tot);
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const uint32_t t = v[j];
      v[j] = run;
      run += t;
    }
    if (whole) {
      uint4 *p = reinterpret_cast<uint4 *>(out + x0);
#pragma unroll
      for (int q = 0; q < kScanPer / 4; ++q) p[q] = make_uint4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; ++j)
        if (x0 + j < n) out[x0 + j] = v[j];
    }
    carry += tot;
  }
  return carry;
}

// Exclusive scan of a[0..n) in place by one block of 1024 threads.
__global__ void __launch_bounds__(1024) k_scan_excl_u32(uint32_t *__restrict__ a, int64_t n) {
  block_scan_rounds(a, a, n);
}

// Exclusive scan of in[0..n) into out by one block of 1024 threads.
__global__ void __launch_bounds__(1024) k_scan_excl_oop(const uint32_t *__restrict__ in,
                                                        uint32_t *__restrict__ out, int64_t n,
                                                        int64_t *total_out) {
  const uint32_t carry = block_scan_rounds(in, out, n);
  if (threadIdx.x == 0 && total_out) *total_out = carry;
}

// Exclusive scan of a long array in three passes: the sum of every
// 4096-element chunk (one block each), a one-block scan of the chunk sums,
// and each chunk scanned from its base.
constexpr int kScanChunk = 4096;

__global__ void __launch_bounds__(256) k_chunk_sums(const uint32_t *__restrict__ a, int64_t n,
                                                    uint32_t *__restrict__ sums) {
  __shared__ uint32_t sh[4];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk;
  uint32_t v = 0;
  for (int k = threadIdx.x; k < kScanChunk; k += 256) {
    const int64_t x = base + k;
    if (x < n) v += a[x];
  }
  uint32_t tot;
  block_excl_scan_add<uint32_t>(v, sh, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(256) k_chunk_scan(uint32_t *__restrict__ a, int64_t n,
                                                    const uint32_t *__restrict__ sums) {
  __shared__ uint32_t sh[4];
  constexpr int kPerThread = kScanChunk / 256;
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kPerThread;
  uint32_t v[kPerThread];
  uint32_t t = 0;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int64_t x = base + k;
    v[k] = x < n ? a[x] : 0u;
    t += v[k];
  }
  uint32_t run = sums[blockIdx.x] + block_excl_scan_add<uint32_t>(t, sh, nullptr);
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int64_t x = base + k;
    if (x < n) a[x] = run;
    run += v[k];
  }
}

// the same three passes for an inclusive scan of int64 values
__global__ void __launch_bounds__(256) k_chunk_sums64(const int64_t *__restrict__ a, int64_t n,
                                                      int64_t *__restrict__ sums) {
  __shared__ int64_t sh[4];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk;
  int64_t v = 0;
  for (int k = threadIdx.x; k < kScanChunk; k += 256) {
    const int64_t x = base + k;
    if (x < n) v += a[x];
  }
  int64_t tot;
  block_excl_scan_add<int64_t>(v, sh, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// exclusive scan of the chunk sums, one block, in place
__global__ void __launch_bounds__(256) k_scan_sums64(int64_t *a, int64_t n) {
  __shared__ int64_t sh[4];
  int64_t carry = 0;
  for (int64_t base = 0; base < n; base += 256) {
    const int64_t x = base + threadIdx.x;
    const int64_t v = x < n ? a[x] : 0;
    int64_t tot;
    const int64_t pre = block_excl_scan_add<int64_t>(v, sh, &tot);
    if (x < n) a[x] = carry + pre;
    carry += tot;
  }
}

__global__ void __launch_bounds__(256) k_chunk_scan64(int64_t *__restrict__ a, int64_t n,
                                                      const int64_t *__restrict__ sums) {
  __shared__ int64_t sh[4];
  constexpr int kPerThread = kScanChunk / 256;
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kPerThread;
  int64_t v[kPerThread];
  int64_t t = 0;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int64_t x = base + k;
    v[k] = x < n ? a[x] : 0;
    t += v[k];
  }
  int64_t run = sums[blockIdx.x] + block_excl_scan_add<int64_t>(t, sh, nullptr);
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int64_t x = base + k;
    run += v[k];
    if (x < n) a[x] = run;
  }
}

void scan_incl_i64_inplace(int64_t *a, int64_t n, int64_t *scratch, hipStream_t s) {
  if (n <= 0) return;
  const int64_t nb = (n + kScanChunk - 1) / kScanChunk;
  k_chunk_sums64<<<(unsigned)nb, 256, 0, s>>>(a, n, scratch);
  k_scan_sums64<<<1, 256, 0, s>>>(scratch, nb);
  k_chunk_scan64<<<(unsigned)nb, 256, 0, s>>>(a, n, scratch);
}

size_t scan_scratch_entries(int64_t n) { return (size_t)((n + kScanChunk - 1) / kScanChunk) + 1; }

// in place; scratch holds scan_scratch_entries(n) entries
void scan_excl_inplace(uint32_t *a, int64_t n, uint32_t *scratch, hipStream_t s) {
  if (n <= 0) return;
  if (n <= 16 * kScanChunk) {
    k_scan_excl_u32<<<1, 1024, 0, s>>>(a, n);
    return;
  }
  const int64_t nb = (n + kScanChunk - 1) / kScanChunk;
  k_chunk_sums<<<(unsigned)nb, 256, 0, s>>>(a, n, scratch);
  k_scan_excl_u32<<<1, 1024, 0, s>>>(scratch, nb);
  k_chunk_scan<<<(unsigned)nb, 256, 0, s>>>(a, n, scratch);
}

void launch_scan_excl(const uint32_t *in, uint32_t *out, int64_t n, int64_t *total_out,
                      hipStream_t s) {
  k_scan_excl_oop<<<1, 1024, 0, s>>>(in, out, n, total_out);
}

// One pass of the stable LSD sort over a tile of OPA_TILE pairs: the rank of
// each pair among the tile's pairs of its digit (wave match of the digit,
// then the counts scanned over chunks and waves), the pairs placed in digit
// order in LDS, then written out in that order so that each digit's run goes
// to consecutive addresses.
__global__ void __launch_bounds__(256) k_rs_scatter(const uint32_t *__restrict__ kin,
                                                    const uint32_t *__restrict__ vin,
                                                    uint32_t *__restrict__ kout,
                                                    uint32_t *__restrict__ vout, int64_t n_cap,
                                                    const int64_t *n_dev, int shift,
                                                    const uint32_t *__restrict__ offs,
                                                    int64_t ntiles) {
  __shared__ uint16_t cnt[OPA_TILE_CHUNKS][4][256];
  __shared__ uint32_t lk[OPA_TILE], lv[OPA_TILE];
  __shared__ uint32_t dbase[256], gbase[256], sh[4];
  const int tid = threadIdx.x, w = wave_id();
  const int64_t n = sort_count(n_cap, n_dev);
  const int64_t base = (int64_t)blockIdx.x * OPA_TILE;
  if (base >= n) return;  // uniform over the block
  for (int i = tid; i < OPA_TILE_CHUNKS * 4 * 256; i += 256) (&cnt[0][0][0])[i] = 0;
  __syncthreads();
  uint32_t key[OPA_TILE_CHUNKS], val[OPA_TILE_CHUNKS], lr[OPA_TILE_CHUNKS];
#pragma unroll
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int64_t x = base + c * 256 + tid;
    const bool ok = x < n;  // pairs past n are the wave's last lanes
    key[c] = ok ? kin[x] : 0u;
    val[c] = ok ? vin[x] : 0u;
    const uint32_t d = (key[c] >> shift) & 255u;
    const uint64_t pm = peers8(d) & __ballot(ok);
    lr[c] = (uint32_t)__popcll(pm & lanemask_lt());
    if (ok && (pm & lanemask_lt()) == 0) cnt[c][w][d] = (uint16_t)__popcll(pm);
  }
  __syncthreads();
  uint32_t tot = 0;  // thread d: the tile's pairs of digit d
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c)
    for (int ww = 0; ww < 4; ++ww) {
      const uint32_t v = cnt[c][ww][tid];
      cnt[c][ww][tid] = (uint16_t)tot;
      tot += v;
    }
  const uint32_t db = block_excl_scan_add<uint32_t>(tot, sh, nullptr);
  dbase[tid] = db;
  gbase[tid] = offs[(int64_t)tid * ntiles + blockIdx.x];
  __syncthreads();
#pragma unroll
  for (int c = 0; c < OPA_TILE_CHUNKS; ++c) {
    const int64_t x = base + c * 256 + tid;
    if (x < n) {
      const uint32_t d = (key[c] >> shift) & 255u;
      const uint32_t lp = dbase[d] + cnt[c][w][d] + lr[c];
      lk[lp] = key[c];
      lv[lp] = val[c];
    }
  }
  __syncthreads();
  const int nl = (int)(n - base < OPA_TILE ? n - base : OPA_TILE);
  for (int j = tid; j < nl; j += 256) {
    const uint32_t k = lk[j], d = (k >> shift) & 255u;
    const uint32_t dst = gbase[d] + ((uint32_t)j - dbase[d]);
    kout[dst] = k;
    vout[dst] = lv[j];
  }
}

// the digit histograms of every tile, then the scan's chunk sums
size_t radix_hist_entries(int64_t n) {
  const int64_t nt = (n + OPA_TILE - 1) / OPA_TILE;
  const int64_t h = (nt > 0 ? nt : 1) * 256;
  return (size_t)h + scan_scratch_entries(h);
}

bool radix_sort_pairs(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, int64_t n,
                      int begin_bit, int end_bit, uint32_t *hist, hipStream_t s,
                      const int64_t *n_dev) {
  if (n <= 0) return false;
  const int64_t nt = (n + OPA_TILE - 1) / OPA_TILE;
  bool in1 = false;
  for (int sh = begin_bit; sh < end_bit; sh += 8) {
    uint32_t *ki = in1 ? k1 : k0, *ko = in1 ? k0 : k1;
    uint32_t *vi = in1 ? v1 : v0, *vo = in1 ? v0 : v1;
    k_rs_hist<<<(unsigned)nt, 256, 0, s>>>(ki, n, n_dev, sh, hist, nt);
    scan_excl_inplace(hist, nt * 256, hist + nt * 256, s);
    k_rs_scatter<<<(unsigned)nt, 256, 0, s>>>(ki, vi, ko, vo, n, n_dev, sh, hist, nt);
    in1 = !in1;
  }
  return in1;
}

__global__ void k_iota(uint32_t *v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) v[i] = (uint32_t)i;
}
// pairs (src[i], i) for a sort of src
__global__ void k_key_pairs(const uint32_t *src, uint32_t *k, uint32_t *v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    k[i] = src[i];
    v[i] = (uint32_t)i;
  }
}

__global__ void k_fill_u32(uint32_t *p, uint32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}
__global__ void k_fill_u8(uint8_t *p, uint8_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

static unsigned blocks_for(int64_t n, int b) { return (unsigned)((n + b - 1) / b); }

__global__ void k_fill_many(FillJobs j) {
  const int q = blockIdx.y;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < j.n[q]; i += stride)
    j.p[q][i] = j.v[q];
}

void FillJobs::add(void *ptr, uint32_t value, int64_t words) {
  if (words <= 0) return;
  if (count >= kMaxJobs) {  // a caller bug: make the call fail
    note(hipErrorInvalidValue);
    return;
  }
  p[count] = static_cast<uint32_t *>(ptr);
  v[count] = value;
  n[count] = words;
  ++count;
}

void fill_many(const FillJobs &j, hipStream_t s) {
  if (j.count == 0) return;
  int64_t mx = 0;
  for (int q = 0; q < j.count; ++q) mx = j.n[q] > mx ? j.n[q] : mx;
  int64_t bx = (mx + 255) / 256;
  if (bx > 1024) bx = 1024;
  k_fill_many<<<dim3((unsigned)bx, (unsigned)j.count), 256, 0, s>>>(j);
}

void fill_u32(uint32_t *p, uint32_t v, int64_t n, hipStream_t s) {
  if (n > 0) k_fill_u32<<<blocks_for(n, 256), 256, 0, s>>>(p, v, n);
}
void fill_u8(uint8_t *p, uint8_t v, int64_t n, hipStream_t s) {
  if (n > 0) k_fill_u8<<<blocks_for(n, 256), 256, 0, s>>>(p, v, n);
}
void launch_iota(uint32_t *v, int64_t n, hipStream_t s) {
  if (n > 0) k_iota<<<blocks_for(n, 256), 256, 0, s>>>(v, n);
}
void launch_key_pairs(const uint32_t *src, uint32_t *k, uint32_t *v, int64_t n, hipStream_t s) {
  if (n > 0) k_key_pairs<<<blocks_for(n, 256), 256, 0, s>>>(src, k, v, n);
}

}  // namespace opa
