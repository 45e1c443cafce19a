// Device helpers shared by the libcure kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cure.h"

#define CURE_DEV __device__ __forceinline__

namespace cure {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// bf16 (raw bits) <-> float32. Widening is exact; narrowing rounds to nearest even.
CURE_DEV float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
CURE_DEV float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
CURE_DEV float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }
CURE_DEV uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);   // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}
CURE_DEV uint32_t pack_bf16x2(float lo, float hi) {
  return uint32_t(f32_to_bf16(lo)) | (uint32_t(f32_to_bf16(hi)) << 16);
}

// exp2 on the hardware transcendental unit (v_exp_f32).
CURE_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <typename T>
CURE_DEV T shfl_xor(T v, int mask) { return __shfl_xor(v, mask, kWave); }

// Top-2 under the order (value descending, index ascending). Empty slots hold
// (-inf, INT32_MAX), which every real entry -- even -inf -- beats.
struct Top2 {
  float v1, v2;
  int i1, i2;
};

CURE_DEV bool beats(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

CURE_DEV Top2 top2_empty() { return {-INFINITY, -INFINITY, INT32_MAX, INT32_MAX}; }

// Both updates are written as value selects: a branchy form leads the
// compiler to pick between the two records through a private-memory copy.
CURE_DEV void top2_push(Top2& t, float x, int i) {
  const bool c1 = beats(x, i, t.v1, t.i1);
  const bool c2 = !c1 && beats(x, i, t.v2, t.i2);
  t.v2 = c1 ? t.v1 : (c2 ? x : t.v2);
  t.i2 = c1 ? t.i1 : (c2 ? i : t.i2);
  t.v1 = c1 ? x : t.v1;
  t.i1 = c1 ? i : t.i1;
}

// The winner's first entry, then the better of the loser's first entry and
// the winner's second.
CURE_DEV Top2 top2_merge(const Top2& a, const Top2& b) {
  const bool bw = beats(b.v1, b.i1, a.v1, a.i1);
  const float w1 = bw ? b.v1 : a.v1, w2 = bw ? b.v2 : a.v2, l1 = bw ? a.v1 : b.v1;
  const int wi1 = bw ? b.i1 : a.i1, wi2 = bw ? b.i2 : a.i2, li1 = bw ? a.i1 : b.i1;
  const bool lw = beats(l1, li1, w2, wi2);
  return {w1, lw ? l1 : w2, wi1, lw ? li1 : wi2};
}

CURE_DEV Top2 top2_wave_reduce(Top2 t) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    Top2 o;
    o.v1 = shfl_xor(t.v1, m); o.i1 = shfl_xor(t.i1, m);
    o.v2 = shfl_xor(t.v2, m); o.i2 = shfl_xor(t.i2, m);
    t = top2_merge(t, o);
  }
  return t;
}

// Log-sum-exp state: the sum of exp(x - ref) over the entries seen, with a
// finite reference (a very negative sentinel until the first finite entry).
constexpr float kLseEmptyRef = -1.0e30f;

struct Lse {
  float ref, sum;
};

CURE_DEV Lse lse_merge(Lse a, Lse b) {
  float r = fmaxf(a.ref, b.ref);
  return {r, a.sum * fast_exp2((a.ref - r) * kLog2e) + b.sum * fast_exp2((b.ref - r) * kLog2e)};
}

CURE_DEV Lse lse_wave_reduce(Lse s) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    Lse o{shfl_xor(s.ref, m), shfl_xor(s.sum, m)};
    s = lse_merge(s, o);
  }
  return s;
}

CURE_DEV float lse_value(Lse s) {
  return s.sum > 0.f ? s.ref + logf(s.sum) : -INFINITY;
}

}  // namespace cure
