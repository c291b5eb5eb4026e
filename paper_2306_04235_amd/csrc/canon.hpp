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

// Sum of the 64 lanes' partials in the canonical butterfly.
__device__ __forceinline__ float wave_sum(float p) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) p = p + __shfl_xor(p, off, 64);
  return p;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

__device__ __forceinline__ int wave_isum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
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

__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const unsigned long long o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

}  // namespace mnmt
