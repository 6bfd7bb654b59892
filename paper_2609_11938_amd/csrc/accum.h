// Per-launch accumulation of the operator table (Eq. 1, Sec. 3.8.1): counts
// and durations in u64, counter sums in fp64 (m or m * d), and for MAX
// counters an order-preserving key of the fp32 maximum. Shared by the
// in-place reduction of the enclosure pass and by the per-row reduction.
#pragma once
#include "common.h"

namespace opa {

// Partial result over some launches of one operator row (device scratch).
struct PartRow {
  unsigned long long kc, tns, mc, mns;
  unsigned long long v[OPATTR_NUM_COUNTERS];  // fp64 bits of a sum, or a MAX key
  uint32_t nan;                               // bit c: a NaN reached MAX counter c
  uint32_t g;                                 // operator row
};
static_assert(sizeof(PartRow) == 200, "PartRow layout");

struct AggIn {
  const uint32_t *dur;
  const int32_t *match;
  int64_t P;
  const float *counters;
  int64_t rs, cs;
  uint32_t dwmask, maxmask;
  int vec4;  // every counter row is 16-byte aligned and contiguous
};

struct Acc {
  unsigned long long kc, tns, mc, mns;
  unsigned long long v[OPATTR_NUM_COUNTERS];
  uint32_t nan;
};

__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
__device__ __forceinline__ double bits2d(unsigned long long b) { return __longlong_as_double((long long)b); }
__device__ __forceinline__ unsigned long long d2bits(double d) {
  return (unsigned long long)__double_as_longlong(d);
}

__device__ __forceinline__ void acc_zero(Acc &a) {
  a.kc = a.tns = a.mc = a.mns = 0;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) a.v[c] = 0;  // +0.0, and the smallest key
  a.nan = 0;
}

// One launch with duration d and profiled row m (m outside [0, P): unmatched).
__device__ __forceinline__ void acc_launch(Acc &a, const AggIn &in, int32_t m, uint32_t d) {
  a.kc += 1;
  a.tns += d;
  if (m < 0 || (int64_t)m >= in.P) return;
  a.mc += 1;
  a.mns += d;
  float v[OPATTR_NUM_COUNTERS];
  const float *row = in.counters + (int64_t)m * in.rs;
  if (in.vec4) {
    const float4 *r4 = reinterpret_cast<const float4 *>(row);
#pragma unroll
    for (int q = 0; q < OPATTR_NUM_COUNTERS / 4; ++q) {
      const float4 t = r4[q];
      v[4 * q] = t.x;
      v[4 * q + 1] = t.y;
      v[4 * q + 2] = t.z;
      v[4 * q + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) v[c] = row[(int64_t)c * in.cs];
  }
  const double dd = (double)d;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    if ((in.maxmask >> c) & 1u) {
      const unsigned long long k = f2key(v[c]);
      a.v[c] = k > a.v[c] ? k : a.v[c];
      if (v[c] != v[c]) a.nan |= 1u << c;
    } else {
      const double x = ((in.dwmask >> c) & 1u) ? (double)v[c] * dd : (double)v[c];  // m_i * d_i
      a.v[c] = d2bits(bits2d(a.v[c]) + x);
    }
  }
}

// a <- a (+) b, where b covers launches after a's
__device__ __forceinline__ void acc_merge(Acc &a, const Acc &b, uint32_t maxmask) {
  a.kc += b.kc;
  a.tns += b.tns;
  a.mc += b.mc;
  a.mns += b.mns;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    if ((maxmask >> c) & 1u) a.v[c] = b.v[c] > a.v[c] ? b.v[c] : a.v[c];
    else a.v[c] = d2bits(bits2d(a.v[c]) + bits2d(b.v[c]));
  }
  a.nan |= b.nan;
}

template <typename F>
__device__ __forceinline__ Acc acc_map(const Acc &a, F f) {
  Acc r;
  r.kc = f(a.kc);
  r.tns = f(a.tns);
  r.mc = f(a.mc);
  r.mns = f(a.mns);
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) r.v[c] = f(a.v[c]);
  r.nan = (uint32_t)f((unsigned long long)a.nan);
  return r;
}

__device__ __forceinline__ Acc acc_shfl_up(const Acc &a, int o) {
  return acc_map(a, [o](unsigned long long x) { return __shfl_up(x, (unsigned)o, OPA_WAVE); });
}
__device__ __forceinline__ Acc acc_shfl_xor(const Acc &a, int o) {
  return acc_map(a, [o](unsigned long long x) { return __shfl_xor(x, o, OPA_WAVE); });
}

// Butterfly reduction over the wave; every lane ends with the total. Each
// step adds two partials (addition is commutative), so the result does not
// depend on scheduling.
__device__ __forceinline__ void acc_wave_reduce(Acc &a, uint32_t maxmask) {
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    const Acc b = acc_shfl_xor(a, o);
    acc_merge(a, b, maxmask);
  }
}

__device__ __forceinline__ void acc_store(PartRow *p, const Acc &a, uint32_t g) {
  p->kc = a.kc;
  p->tns = a.tns;
  p->mc = a.mc;
  p->mns = a.mns;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) p->v[c] = a.v[c];
  p->nan = a.nan;
  p->g = g;
}

__device__ __forceinline__ void acc_load(Acc &a, const PartRow *p) {
  a.kc = p->kc;
  a.tns = p->tns;
  a.mc = p->mc;
  a.mns = p->mns;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) a.v[c] = p->v[c];
  a.nan = p->nan;
}

}  // namespace opa
