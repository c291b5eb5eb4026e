// blocks.hpp -- device building blocks shared by the kernels: 16-byte int8
// dot products, one-wave attention, and LayerNorm + quantization of a row.
// All fp32 arithmetic follows the canonical order of canon.hpp.
#pragma once

#include <cfloat>

#include "canon.hpp"

namespace mnmt {

constexpr int kMaxAttnLen = 256;  // longest attended sequence (4 keys per lane)
constexpr int kMaxHeadDim = 128;  // 8 x 16 bytes of query in registers
constexpr int kMaxRowLen = 1024;  // LayerNorm width (16 values per lane)

__device__ __forceinline__ int dot16(const int4 a, const int4 b, int acc) {
  acc = __builtin_amdgcn_sdot4(a.x, b.x, acc, false);
  acc = __builtin_amdgcn_sdot4(a.y, b.y, acc, false);
  acc = __builtin_amdgcn_sdot4(a.z, b.z, acc, false);
  acc = __builtin_amdgcn_sdot4(a.w, b.w, acc, false);
  return acc;
}

// Attention of one query row over n keys for one head, by one wave
// (Appendix A self-weight / self-sum equations with the quantizer figure's
// precisions): int8 scores, fp32 softmax in the canonical order, context
// accumulated over ascending key index with one fma per key, requantized.
// key(t) / val(t) return the head's dh codes of key / value t (global or LDS
// addresses).  Softmax weights are exchanged by lane shuffles, so the wave
// needs no barrier and may share its block with other waves.
template <class KeyFn, class ValFn>
__device__ __forceinline__ void attend_wave(const int8_t* __restrict__ q, int n, int dh, KeyFn key, ValFn val,
                                            float c_qk, float c_pv, int8_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int nc = dh / 16;
  int4 qv[kMaxHeadDim / 16];
#pragma unroll
  for (int c = 0; c < kMaxHeadDim / 16; ++c) qv[c] = c < nc ? *(const int4*)(q + 16 * c) : make_int4(0, 0, 0, 0);
  float sv[kMaxAttnLen / 64];
  float mx = -FLT_MAX;
#pragma unroll
  for (int i = 0; i < kMaxAttnLen / 64; ++i) {
    const int t = lane + 64 * i;
    sv[i] = 0.0f;
    if (t < n) {
      const int8_t* kp = key(t);
      int acc = 0;
#pragma unroll
      for (int c = 0; c < kMaxHeadDim / 16; ++c)
        if (c < nc) acc = dot16(*(const int4*)(kp + 16 * c), qv[c], acc);
      sv[i] = (float)acc * c_qk;
      mx = fmaxf(mx, sv[i]);
    }
  }
  mx = wave_max(mx);
  float part = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxAttnLen / 64; ++i) {
    const int t = lane + 64 * i;
    if (t < n) {
      sv[i] = canon_exp(sv[i] - mx);
      part = part + sv[i];
    }
  }
  const float inv = 1.0f / wave_sum(part);
#pragma unroll
  for (int i = 0; i < kMaxAttnLen / 64; ++i) sv[i] = sv[i] * inv;  // p_t for t = lane + 64 i
  for (int j0 = 0; j0 < dh; j0 += 64) {
    const int j = j0 + lane;
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < kMaxAttnLen / 64; ++i) {
      const int tn = n - 64 * i < 64 ? n - 64 * i : 64;
      for (int tl = 0; tl < tn; ++tl) {
        const float p = __shfl(sv[i], tl, 64);
        const int8_t* vp = val(64 * i + tl);
        if (j < dh) acc = fmaf(p, (float)vp[j], acc);
      }
    }
    if (j < dh) out[j] = code_of(acc * c_pv);
  }
}

// LayerNorm of one row by one wave (element i in lane i % 64, ascending i),
// optionally without the normalization (do_ln = 0: y = x).  Writes the int8
// codes quant(y, inv_s) to q (any address space) and, if y_out, the fp32 y.
__device__ __forceinline__ void ln_row_wave(const float* __restrict__ x, int d, int do_ln, const float* __restrict__ g,
                                            const float* __restrict__ b, float eps, float inv_s, int8_t* q,
                                            float* y_out) {
  const int lane = threadIdx.x & 63;
  float v[kMaxRowLen / 64];
  const int n = (d + 63) / 64;
#pragma unroll
  for (int j = 0; j < kMaxRowLen / 64; ++j) {
    const int i = lane + 64 * j;
    v[j] = (j < n && i < d) ? x[i] : 0.0f;
  }
  if (do_ln) {
    float p = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxRowLen / 64; ++j)
      if (j < n && lane + 64 * j < d) p = p + v[j];
    const float inv_d = 1.0f / (float)d;
    const float mu = wave_sum(p) * inv_d;
    float p2 = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxRowLen / 64; ++j) {
      if (j < n && lane + 64 * j < d) {
        v[j] = v[j] - mu;
        p2 = fmaf(v[j], v[j], p2);
      }
    }
    const float var = wave_sum(p2) * inv_d;
    const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
    for (int j = 0; j < kMaxRowLen / 64; ++j) {
      const int i = lane + 64 * j;
      if (j < n && i < d) v[j] = fmaf(v[j] * rstd, g[i], b[i]);
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxRowLen / 64; ++j) {
    const int i = lane + 64 * j;
    if (j < n && i < d) {
      if (q) q[i] = code_of(v[j] * inv_s);
      if (y_out) y_out[i] = v[j];
    }
  }
}

}  // namespace mnmt
