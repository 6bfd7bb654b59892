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

// The counter row m (fp32), or nothing when m is outside [0, P): the load
// half of acc_launch, so that a caller can have the next row in flight.
__device__ __forceinline__ void acc_load_row(const AggIn &in, int32_t m,
                                             float (&v)[OPATTR_NUM_COUNTERS]) {
  if (m < 0 || (int64_t)m >= in.P) return;
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
}

// The accumulation half of acc_launch, with the row already loaded.
__device__ __forceinline__ void acc_add_row(Acc &a, const AggIn &in, int32_t m, uint32_t d,
                                            const float (&v)[OPATTR_NUM_COUNTERS], uint32_t mx,
                                            uint32_t dw) {
  a.kc += 1;
  a.tns += d;
  if (m < 0 || (int64_t)m >= in.P) return;
  a.mc += 1;
  a.mns += d;
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

// Lane shift of a 64-bit value by a DPP move of each half (register to
// register, no LDS round trip). Lanes without a source (bound_ctrl: 0) or in
// rows the row mask leaves out (not written) hold no shifted value: the scan
// steps use the result only in lanes that take it, which always have a
// source. The move needs no old value, hence no extra register move.
template <int CTRL, int ROWMASK, int BANKMASK>
__device__ __forceinline__ unsigned long long dpp64(unsigned long long v) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const uint32_t l2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)lo, CTRL, ROWMASK, BANKMASK, true);
  const uint32_t h2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)hi, CTRL, ROWMASK, BANKMASK, true);
  return ((unsigned long long)h2 << 32) | l2;
}

// One step of the segmented scan: a += the shifted value in the lanes that
// take it. Fields go in groups of four: the group's moves, then its adds
// under one branch, so that no second accumulator is held and the adds need
// no per-field select.
template <int CTRL, int ROWMASK, int BANKMASK>
__device__ __forceinline__ void acc_scan_dpp(Acc &a, bool take, uint32_t maxmask) {
  {
    const unsigned long long y0 = dpp64<CTRL, ROWMASK, BANKMASK>(a.kc);
    const unsigned long long y1 = dpp64<CTRL, ROWMASK, BANKMASK>(a.tns);
    const unsigned long long y2 = dpp64<CTRL, ROWMASK, BANKMASK>(a.mc);
    const unsigned long long y3 = dpp64<CTRL, ROWMASK, BANKMASK>(a.mns);
    const uint32_t yn = (uint32_t)__builtin_amdgcn_mov_dpp((int)a.nan, CTRL, ROWMASK, BANKMASK, true);
    if (take) {
      a.kc += y0;
      a.tns += y1;
      a.mc += y2;
      a.mns += y3;
      a.nan |= yn;
    }
  }
#pragma unroll
  for (int g = 0; g < OPATTR_NUM_COUNTERS; g += 4) {
    unsigned long long y[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) y[j] = dpp64<CTRL, ROWMASK, BANKMASK>(a.v[g + j]);
    if (take) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = g + j;
        if ((maxmask >> c) & 1u) a.v[c] = y[j] > a.v[c] ? y[j] : a.v[c];
        else a.v[c] = d2bits(bits2d(a.v[c]) + bits2d(y[j]));
      }
    }
  }
}

// Segmented inclusive scan over the wave (segment of lane l starts at lane
// sl): shifts by 1, 2, 4, 8 inside rows of 16 lanes, then the row totals
// broadcast from lane 15 to rows 1 and 3 and from lane 31 to rows 2 and 3.
__device__ __forceinline__ void acc_seg_scan(Acc &a, int sl, uint32_t maxmask) {
  const int ln = lane_id(), p = ln & 15, row = ln >> 4;
  acc_scan_dpp<0x111, 0xF, 0xF>(a, p >= 1 && ln - 1 >= sl, maxmask);
  acc_scan_dpp<0x112, 0xF, 0xF>(a, p >= 2 && ln - 2 >= sl, maxmask);
  acc_scan_dpp<0x114, 0xF, 0xF>(a, p >= 4 && ln - 4 >= sl, maxmask);
  acc_scan_dpp<0x118, 0xF, 0xF>(a, p >= 8 && ln - 8 >= sl, maxmask);
  acc_scan_dpp<0x142, 0xA, 0xF>(a, (row == 1 || row == 3) && sl <= row * 16 - 1, maxmask);
  acc_scan_dpp<0x143, 0xC, 0xF>(a, row >= 2 && sl <= 31, maxmask);
}

// Reduction over the wave; every lane ends with the total: an inclusive
// scan in a fixed lane order (DPP moves, as above), then lane 63's value is
// read into every lane. The order of the additions does not depend on
// scheduling.
__device__ __forceinline__ unsigned long long lane63(unsigned long long v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ void acc_wave_reduce(Acc &a, uint32_t maxmask) {
  acc_seg_scan(a, 0, maxmask);
  a.kc = lane63(a.kc);
  a.tns = lane63(a.tns);
  a.mc = lane63(a.mc);
  a.mns = lane63(a.mns);
#pragma unroll
  for (int c = 0; c < OPATTR_NUM_COUNTERS; ++c) a.v[c] = lane63(a.v[c]);
  a.nan = (uint32_t)__builtin_amdgcn_readlane((int)a.nan, 63);
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
