// canon.hpp -- device fp32 primitives in the engine's canonical evaluation
// order.  Every fp32 reduction over n terms is the "wave64 order": term i is
// added to lane i mod 64's partial sum (ascending i, partials start at +0),
// then partials combine by an xor butterfly over offsets 32, 16, 8, 4, 2, 1.
// Because fp32 addition is commutative, every lane of the butterfly ends with
// the same value, and that value does not depend on how the terms were
// scheduled beyond the per-lane ascending order.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace mnmt {

// The canonical butterfly without the LDS crossbar.  Step `off` gives lane i
// op(x_i, x_{i^off}).  The 32 and 16 steps use gfx950's permlane swaps: after
// v_permlane32_swap of a value with itself the two results hold, in every
// lane, x_i and x_{i^32} (in some order), and likewise x_i and x_{i^16} after
// v_permlane16_swap.  After those steps a lane's value depends only on i mod
// 16, so the 8, 4, 2, 1 steps can take the partner from a rotation of the
// lane's 16-lane row (DPP row_ror), whose source lane is congruent to i^off
// modulo 2 off.  op is commutative (fp32 add and max, integer add and max),
// so every lane computes exactly the value of the xor butterfly.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xf, 0xf, false);
}
constexpr int kRowRor8 = 0x128, kRowRor4 = 0x124, kRowRor2 = 0x122, kRowRor1 = 0x121;

// Partner values of steps 32 and 16: returns {a, b} with {a, b} = {x_i, x_{i^off}}.
__device__ __forceinline__ void swap32(uint32_t v, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ void swap16(uint32_t v, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  a = r[0];
  b = r[1];
}

template <class Op>
__device__ __forceinline__ float butterfly_f32(float x, Op op) {
  uint32_t a, b;
  swap32(__float_as_uint(x), a, b);
  x = op(__uint_as_float(a), __uint_as_float(b));
  swap16(__float_as_uint(x), a, b);
  x = op(__uint_as_float(a), __uint_as_float(b));
  x = op(x, __uint_as_float(dpp_u32<kRowRor8>(__float_as_uint(x))));
  x = op(x, __uint_as_float(dpp_u32<kRowRor4>(__float_as_uint(x))));
  x = op(x, __uint_as_float(dpp_u32<kRowRor2>(__float_as_uint(x))));
  x = op(x, __uint_as_float(dpp_u32<kRowRor1>(__float_as_uint(x))));
  return x;
}

// Sum of the 64 lanes' partials in the canonical butterfly.
__device__ __forceinline__ float wave_sum(float p) {
  return butterfly_f32(p, [](float u, float v) { return u + v; });
}

__device__ __forceinline__ float wave_max(float v) {
  return butterfly_f32(v, [](float u, float w) { return fmaxf(u, w); });
}

__device__ __forceinline__ int wave_isum(int v) {
  uint32_t a, b;
  swap32((uint32_t)v, a, b);
  v = (int)(a + b);
  swap16((uint32_t)v, a, b);
  v = (int)(a + b);
  v += (int)dpp_u32<kRowRor8>((uint32_t)v);
  v += (int)dpp_u32<kRowRor4>((uint32_t)v);
  v += (int)dpp_u32<kRowRor2>((uint32_t)v);
  v += (int)dpp_u32<kRowRor1>((uint32_t)v);
  return v;
}

// Symmetric int8 code: clamp(rint(y), -127, 127) (round half to even).
__device__ __forceinline__ int8_t code_of(float y) {
  float r = rintf(y);
  r = fminf(fmaxf(r, -127.0f), 127.0f);
  return (int8_t)(int)r;
}

// e^x for x <= 0: k = rint(x log2 e); r = x - k ln2 with ln2 split into a
// 12-bit-trimmed high part and its remainder (two fmas, Cody-Waite);
// e^r by the Taylor series through r^7 in Horner form; scaled by 2^k.
__device__ __forceinline__ float canon_exp(float x) {
  if (x < -87.0f) return 0.0f;
  const float k = rintf(x * 1.44269504088896341f);
  float r = fmaf(-k, 0x1.62e400p-1f, x);
  r = fmaf(-k, (float)(0.69314718055994530942 - 0.693145751953125), r);
  float p = (float)(1.0 / 5040.0);
  p = fmaf(p, r, (float)(1.0 / 720.0));
  p = fmaf(p, r, (float)(1.0 / 120.0));
  p = fmaf(p, r, (float)(1.0 / 24.0));
  p = fmaf(p, r, (float)(1.0 / 6.0));
  p = fmaf(p, r, 0.5f);
  p = fmaf(p, r, 1.0f);
  p = fmaf(p, r, 1.0f);
  return ldexpf(p, (int)k);
}

// ln x for normal x > 0: x = m 2^e with m in [sqrt(1/2), sqrt(2));
// ln m = 2 atanh(f), f = (m - 1) / (m + 1), odd series through f^9.
__device__ __forceinline__ float canon_log(float x) {
  const uint32_t bits = __float_as_uint(x);
  int e = (int)((bits >> 23) & 0xff) - 126;                      // x = m 2^e, m in [0.5, 1)
  float m = __uint_as_float((bits & 0x007fffffu) | 0x3f000000u);
  if (m < 0.70710678118654752f) {
    m = m * 2.0f;
    e = e - 1;
  }
  const float f = (m - 1.0f) / (m + 1.0f);
  const float s = f * f;
  float p = (float)(1.0 / 9.0);
  p = fmaf(p, s, (float)(1.0 / 7.0));
  p = fmaf(p, s, (float)(1.0 / 5.0));
  p = fmaf(p, s, (float)(1.0 / 3.0));
  p = fmaf(p, s, 1.0f);
  const float ln_m = (2.0f * f) * p;
  const float ef = (float)e;
  return fmaf(ef, 0x1.62e400p-1f, fmaf(ef, (float)(0.69314718055994530942 - 0.693145751953125), ln_m));
}

// Order-preserving 32-bit key of a float (larger float -> larger key).
__device__ __forceinline__ uint32_t ordered_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// (value, index) packed so that the unsigned maximum is the largest value and,
// among equal values, the smallest index.
__device__ __forceinline__ unsigned long long pack_argmax(float v, int idx) {
  return ((unsigned long long)ordered_key(v) << 32) | (unsigned long long)(0xffffffffu - (uint32_t)idx);
}

__device__ __forceinline__ int unpack_index(unsigned long long key) {
  return (int)(0xffffffffu - (uint32_t)(key & 0xffffffffull));
}

// Tagged form of a pack_argmax key (index < 2^18): the ordered value, a
// 14-bit tag, 0x3FFFF - index; 0 (no candidate) becomes the bare tag.
__device__ __forceinline__ unsigned long long tagged_key(unsigned long long key, unsigned tag) {
  if (key == 0ull) return (unsigned long long)tag << 18;
  const uint32_t idx = 0xffffffffu - (uint32_t)(key & 0xffffffffull);
  return (key & 0xffffffff00000000ull) | ((unsigned long long)tag << 18) | (unsigned long long)(0x3FFFFu - idx);
}
__device__ __forceinline__ unsigned key_tag(unsigned long long k) { return (unsigned)(k >> 18) & 0x3FFFu; }
__device__ __forceinline__ int tagged_index(unsigned long long k) { return (int)(0x3FFFFu - (uint32_t)(k & 0x3FFFFull)); }
// the pack_argmax key of a tagged key
__device__ __forceinline__ unsigned long long untag_key(unsigned long long k) {
  return (k & 0xffffffff00000000ull) | (unsigned long long)(0xffffffffu - (uint32_t)tagged_index(k));
}

__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long v) {
  auto mx = [](unsigned long long u, unsigned long long w) { return u > w ? u : w; };
  auto join = [](uint32_t lo, uint32_t hi) { return ((unsigned long long)hi << 32) | lo; };
  uint32_t a0, b0, a1, b1;
  swap32((uint32_t)v, a0, b0);
  swap32((uint32_t)(v >> 32), a1, b1);
  v = mx(join(a0, a1), join(b0, b1));
  swap16((uint32_t)v, a0, b0);
  swap16((uint32_t)(v >> 32), a1, b1);
  v = mx(join(a0, a1), join(b0, b1));
  v = mx(v, join(dpp_u32<kRowRor8>((uint32_t)v), dpp_u32<kRowRor8>((uint32_t)(v >> 32))));
  v = mx(v, join(dpp_u32<kRowRor4>((uint32_t)v), dpp_u32<kRowRor4>((uint32_t)(v >> 32))));
  v = mx(v, join(dpp_u32<kRowRor2>((uint32_t)v), dpp_u32<kRowRor2>((uint32_t)(v >> 32))));
  v = mx(v, join(dpp_u32<kRowRor1>((uint32_t)v), dpp_u32<kRowRor1>((uint32_t)(v >> 32))));
  return v;
}
}  // namespace mnmt
