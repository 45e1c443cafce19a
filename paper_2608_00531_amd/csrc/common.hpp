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

CURE_DEV int lane_id() { return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// Butterfly partners for wave-wide reductions, on the VALU (DPP and lane
// permutes) instead of the LDS crossbar. Stage k pairs each lane with a lane
// whose group of k lanes is disjoint from its own:
//   1, 2   quad permutes (lane ^ 1, lane ^ 2)
//   4      half-row mirror (lane i <-> 7 - i within 8)
//   8      row mirror (lane i <-> 15 - i within 16)
//   16     swizzle, lane ^ 16 within 32
//   32     permlane32 swap, lane ^ 32
// Stages 4 and 8 are not xor patterns: they pair whole groups only once the
// stages below them have run, so they are used only in the full sequence
// 1, 2, 4, 8, 16, 32; stages 16 and 32 are true xors and may be used alone.
// After a full sequence with a commutative merge every lane holds the same
// wave-wide result.
template <int kStage>
CURE_DEV int partner(int v);
template <>
CURE_DEV int partner<1>(int v) { return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false); }
template <>
CURE_DEV int partner<2>(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false); }
template <>
CURE_DEV int partner<4>(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false); }
template <>
CURE_DEV int partner<8>(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false); }
template <>
CURE_DEV int partner<16>(int v) { return __builtin_amdgcn_ds_swizzle(v, 0x401F); }
template <>
CURE_DEV int partner<32>(int v) {
  // Lanes 0-31 of the first result repeat lanes 0-31 of v; lanes 0-31 of the
  // second hold lanes 32-63 of v (and the reverse for the upper half).
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return (int)(lane_id() < 32 ? r[1] : r[0]);
}
template <int kStage>
CURE_DEV float partner(float v) { return __int_as_float(partner<kStage>(__float_as_int(v))); }

// Sum and maximum of a value over lanes l and l ^ 32 (both halves get it).
CURE_DEV float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
CURE_DEV float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

CURE_DEV float wave_max(float x) {
  x = fmaxf(x, partner<1>(x));
  x = fmaxf(x, partner<2>(x));
  x = fmaxf(x, partner<4>(x));
  x = fmaxf(x, partner<8>(x));
  x = fmaxf(x, partner<16>(x));
  return max_halves(x);
}
CURE_DEV int wave_max(int x) {
  x = max(x, partner<1>(x));
  x = max(x, partner<2>(x));
  x = max(x, partner<4>(x));
  x = max(x, partner<8>(x));
  x = max(x, partner<16>(x));
  return max(x, partner<32>(x));
}
CURE_DEV float wave_sum(float x) {
  x += partner<1>(x);
  x += partner<2>(x);
  x += partner<4>(x);
  x += partner<8>(x);
  x += partner<16>(x);
  return sum_halves(x);
}

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

template <int kStage>
CURE_DEV Top2 top2_stage(const Top2& t) {
  const Top2 o{partner<kStage>(t.v1), partner<kStage>(t.v2), partner<kStage>(t.i1),
               partner<kStage>(t.i2)};
  return top2_merge(t, o);
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

template <int kStage>
CURE_DEV Lse lse_stage(const Lse& s) {
  return lse_merge(s, Lse{partner<kStage>(s.ref), partner<kStage>(s.sum)});
}

CURE_DEV Lse lse_wave_reduce(Lse s) {
  s = lse_stage<1>(s);
  s = lse_stage<2>(s);
  s = lse_stage<4>(s);
  s = lse_stage<8>(s);
  s = lse_stage<16>(s);
  return lse_stage<32>(s);
}

CURE_DEV float lse_value(Lse s) {
  return s.sum > 0.f ? s.ref + logf(s.sum) : -INFINITY;
}

}  // namespace cure
