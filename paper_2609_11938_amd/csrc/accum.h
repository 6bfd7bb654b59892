// Per-launch accumulation of the operator table (Eq. 1, Sec. 3.8.1): counts
// and durations in u64, counter sums in fp64 (m or m * d), and for MAX
// counters an order-preserving key of the fp32 maximum. Shared by the
// in-place reduction of the enclosure pass and by the per-row reduction.
#pragma once
#include "common.h"
#include "impl.h"

namespace opa {

// Partial result over some launches of one operator row (device scratch).
struct PartRow {
  unsigned long long kc, tns, mc, mns;
  unsigned long long v[OPATTR_NUM_COUNTERS];  // fp64 bits of a sum, or a MAX key
  uint32_t nan;                               // bit c: a NaN reached MAX counter c
  uint32_t pad;
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
// mx / dw: MAX and DW-mean counters (compile-time constants in the kernels
// specialised for the default kinds, so the per-counter tests fold away).
__device__ __forceinline__ void acc_launch(Acc &a, const AggIn &in, int32_t m, uint32_t d,
                                           uint32_t mx, uint32_t dw) {
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
    if ((mx >> c) & 1u) {
      const unsigned long long k = f2key(v[c]);
      a.v[c] = k > a.v[c] ? k : a.v[c];
      if (v[c] != v[c]) a.nan |= 1u << c;
    } else {
      const double x = ((dw >> c) & 1u) ? (double)v[c] * dd : (double)v[c];  // m_i * d_i
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

// One step of a segmented inclusive scan over the lanes, field by field so
// that no second accumulator is held: a += value of lane (lane - o) if take.
__device__ __forceinline__ void acc_scan_step(Acc &a, int o, bool take, uint32_t maxmask) {
#define OPA_SCAN_U64(f)                                                  \
  {                                                                      \
    const unsigned long long y = __shfl_up(a.f, (unsigned)o, OPA_WAVE); \
    if (take) a.f += y;                                                  \
  }
  OPA_SCAN_U64(kc)
  OPA_SCAN_U64(tns)
  OPA_SCAN_U64(mc)
  OPA_SCAN_U64(mns)
#undef OPA_SCAN_U64
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
    const unsigned long long y = __shfl_up(a.v[c], (unsigned)o, OPA_WAVE);
    if (take) {
      if ((maxmask >> c) & 1u) a.v[c] = y > a.v[c] ? y : a.v[c];
      else a.v[c] = d2bits(bits2d(a.v[c]) + bits2d(y));
    }
  }
  const uint32_t yn = __shfl_up(a.nan, (unsigned)o, OPA_WAVE);
  if (take) a.nan |= yn;
}

// Butterfly reduction over the wave; every lane ends with the total. Each
// step adds two partials (addition is commutative), so the result does not
// depend on scheduling.
__device__ __forceinline__ void acc_wave_reduce(Acc &a, uint32_t maxmask) {
#pragma unroll
  for (int o = 1; o < OPA_WAVE; o <<= 1) {
    a.kc += __shfl_xor(a.kc, o, OPA_WAVE);
    a.tns += __shfl_xor(a.tns, o, OPA_WAVE);
    a.mc += __shfl_xor(a.mc, o, OPA_WAVE);
    a.mns += __shfl_xor(a.mns, o, OPA_WAVE);
#pragma unroll
    for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) {
      const unsigned long long y = __shfl_xor(a.v[c], o, OPA_WAVE);
      if ((maxmask >> c) & 1u) a.v[c] = y > a.v[c] ? y : a.v[c];
      else a.v[c] = d2bits(bits2d(a.v[c]) + bits2d(y));
    }
    a.nan |= __shfl_xor(a.nan, o, OPA_WAVE);
  }
}

__device__ __forceinline__ void acc_store(PartRow *p, const Acc &a) {
  p->kc = a.kc;
  p->tns = a.tns;
  p->mc = a.mc;
  p->mns = a.mns;
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) p->v[c] = a.v[c];
  p->nan = a.nan;
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
