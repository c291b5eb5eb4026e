// blocks.hpp -- device building blocks shared by the kernels: 16-byte int8
// dot products, one-wave attention, and LayerNorm + quantization of a row.
// All fp32 arithmetic follows the canonical order of canon.hpp.
#pragma once

#include <cfloat>

#include "canon.hpp"
#include "internal.h"

namespace mnmt {

constexpr int kMaxAttnLen = 256;  // longest attended sequence (4 keys per lane)
constexpr int kMaxHeadDim = 128;  // 8 x 16 bytes of query in registers
constexpr int kMaxRowLen = 1024;  // LayerNorm width (16 values per lane)

// 16 bytes as a native vector (copied as a value, never through memory)
typedef int v4i __attribute__((ext_vector_type(4)));

// One v_mfma_i32_16x16x64_i8: lane l holds 16 bytes of K at 16 (l / 16) of
// row l % 16 of A and of B; D[i] of lane l is row 4 (l / 16) + i, column l % 16.
__device__ __forceinline__ v4i mfma16(const v4i a, const v4i b, const v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// 4-bit weight codes (the paper's W-E-A 4-8-8 setting) widened to int8: in
// each group of 16 codes of a row, packed byte i (i < 8) holds code i in its
// low nibble and code i + 8 in its high nibble, each plus 8.  Per byte,
// ((u & 15) + 0x78) ^ 0x80 = u - 8 as a signed byte, with no carry between
// bytes (u + 0x78 <= 0x87).
__device__ __forceinline__ v4i unpack_i4x16(uint2 p) {
  const unsigned m = 0x0F0F0F0Fu, b = 0x78787878u, s = 0x80808080u;
  v4i r;
  r.x = (int)(((p.x & m) + b) ^ s);         // codes 0..3
  r.y = (int)(((p.y & m) + b) ^ s);         // codes 4..7
  r.z = (int)((((p.x >> 4) & m) + b) ^ s);  // codes 8..11
  r.w = (int)((((p.y >> 4) & m) + b) ^ s);  // codes 12..15
  return r;
}

// A 16-byte weight fragment (16 consecutive codes of a weight row) held in
// registers.  4-bit weights are loaded as their 8 packed bytes and widened
// where the matrix instruction takes them, so that a kernel still issues all
// of its loads before it waits for any.
template <bool W4>
struct WFrag {
  v4i v;
  __device__ __forceinline__ v4i get() const { return v; }
};
template <>
struct WFrag<true> {
  uint2 p;
  __device__ __forceinline__ v4i get() const { return unpack_i4x16(p); }
};

// The fragment of row `row` of a [N, K] weight at column k0 (a multiple of
// 16); W4: W holds the packed 4-bit rows (K / 2 bytes each).
template <bool W4>
__device__ __forceinline__ WFrag<W4> load_wfrag(const int8_t* W, size_t row, int K, int k0) {
  WFrag<W4> f;
  if constexpr (W4)
    f.p = *(const uint2*)(reinterpret_cast<const uint8_t*>(W) + row * (size_t)(K / 2) + k0 / 2);
  else
    f.v = *(const v4i*)(W + row * (size_t)K + k0);
  return f;
}

__device__ __forceinline__ int dot16(const int4 a, const int4 b, int acc) {
  acc = __builtin_amdgcn_sdot4(a.x, b.x, acc, false);
  acc = __builtin_amdgcn_sdot4(a.y, b.y, acc, false);
  acc = __builtin_amdgcn_sdot4(a.z, b.z, acc, false);
  acc = __builtin_amdgcn_sdot4(a.w, b.w, acc, false);
  return acc;
}
__device__ __forceinline__ int dot16(const v4i a, const int4 b, int acc) {
  return dot16(make_int4(a.x, a.y, a.z, a.w), b, acc);
}

// The 16 weight codes of row `row` at column k (a multiple of 16) of an int8
// [N, K] weight or, W4, of its packed 4-bit rows; zeros where `ok` is false.
template <bool W4>
__device__ __forceinline__ WFrag<W4> load_wfrag_if(bool ok, const int8_t* W, size_t row, int K, int k) {
  return ok ? load_wfrag<W4>(W, row, K, k) : WFrag<W4>{};
}

// Workgroup barrier that orders LDS accesses only: the fences name the local
// address space, so the barrier waits for the wave's LDS operations but not
// for its global loads (__syncthreads would wait for every load in flight,
// including prefetches meant for a later phase).  Every block-level exchange
// in these kernels goes through LDS.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// LDS-visibility barrier for the lanes of one wave (the other waves of the
// block are not involved).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// LayerNorm of one row held by a wave (element i = lane + 64 j in v[j]) in
// the canonical order: lane partials over ascending i, then the butterfly.
template <int NJ>
__device__ __forceinline__ void ln_row(float (&v)[NJ], const float (&g)[NJ], const float (&b)[NJ], int d, float eps) {
  const int lane = threadIdx.x & 63;
  const float inv_d = 1.0f / (float)d;
  float p = 0.0f;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (lane + 64 * j < d) p = p + v[j];
  const float mu = wave_sum(p) * inv_d;
  float p2 = 0.0f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (lane + 64 * j < d) {
      v[j] = v[j] - mu;
      p2 = fmaf(v[j], v[j], p2);
    }
  }
  const float rstd = 1.0f / sqrtf(wave_sum(p2) * inv_d + eps);
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (lane + 64 * j < d) v[j] = fmaf(v[j] * rstd, g[j], b[j]);
}

// LDS one wave's attention needs: softmax weights and the value rows.
template <int NMAX, int DHMAX>
struct AttnLdsT {
  alignas(16) float p[NMAX];
  int8_t v[NMAX][DHMAX];
};

// The softmax and context of one query row for one head, by one wave
// (Appendix A self-weight / self-sum equations with the quantizer figure's
// precisions): sv[i] holds the scaled int8 score (float)(q . k_t) * c_qk of
// key t = lane + 64 i (valid for t < n); fp32 softmax in the canonical order
// (lane partials over ascending i, then the butterfly); context accumulated
// over ascending key index with one fma per key from the values in LDS
// (value t's codes at v + t * v_stride), requantized into out[0, dh).  p is
// the wave's LDS row of at least n weights, 16-byte aligned.
template <int NI>
__device__ __forceinline__ void softmax_context(float (&sv)[NI], int n, int dh, float c_pv, float* p,
                                                const int8_t* v, int v_stride, int8_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  float mx = -FLT_MAX;
#pragma unroll
  for (int i = 0; i < NI; ++i)
    if (lane + 64 * i < n) mx = fmaxf(mx, sv[i]);
  mx = wave_max(mx);
  float part = 0.0f;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    if (lane + 64 * i < n) {
      sv[i] = canon_exp(sv[i] - mx);
      part = part + sv[i];
    }
  }
  const float inv = 1.0f / wave_sum(part);
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int t = lane + 64 * i;
    if (t < n) p[t] = sv[i] * inv;
  }
  wave_sync();  // the weights visible to every lane of this wave
  // (8 keys per group: their weights and values are read from LDS before the
  // group's chain of fmas, so the chain does not wait on each read)
  for (int j = lane; j < dh; j += 64) {
    float acc = 0.0f;
    int t = 0;
#pragma unroll 2
    for (; t + 8 <= n; t += 8) {
      const float4 pa = *(const float4*)(p + t);
      const float4 pb = *(const float4*)(p + t + 4);
      float vv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) vv[k] = (float)v[(t + k) * v_stride + j];
      acc = fmaf(pa.x, vv[0], acc);
      acc = fmaf(pa.y, vv[1], acc);
      acc = fmaf(pa.z, vv[2], acc);
      acc = fmaf(pa.w, vv[3], acc);
      acc = fmaf(pb.x, vv[4], acc);
      acc = fmaf(pb.y, vv[5], acc);
      acc = fmaf(pb.z, vv[6], acc);
      acc = fmaf(pb.w, vv[7], acc);
    }
    for (; t < n; ++t) acc = fmaf(p[t], (float)v[t * v_stride + j], acc);
    out[j] = code_of(acc * c_pv);
  }
  wave_sync();  // every lane done with p and v before the wave reuses them
}

// Input rows -> int8 rows in LDS (Section 4.2 fusion of the element-wise work
// in front of a GEMM): row r of the block is global row row0 + r, taken from
// the residual stream or computed as the token embedding, optionally layer-
// normalized, then quantized into a_lds + r * lds_stride.  `writer` blocks
// also store the embedding (wb_input) or the normalized row (post-LN) to
// in.x_out.  Wave w prepares rows w, w + 4, ...; each wave works on G rows
// at once (kPrepGroup by default) so that their loads and reductions
// overlap: a wave with all its rows in one group pays one memory round trip.
constexpr int kPrepGroup = 4;

// Row-width classes the fused kernels are compiled for (d <= class).
__host__ __device__ constexpr int row_class(int d) {
  return d <= 64 ? 64 : d <= 128 ? 128 : d <= 256 ? 256 : d <= 384 ? 384 : d <= 512 ? 512 : 1024;
}
// Lanes per weight row of a GEMV over rows of that width (a power of two,
// leaving each lane at most two 16-byte chunks).
__host__ __device__ constexpr int lanes_per_row(int dmax) {
  return dmax >= 1024 ? 64 : dmax >= 512 ? 32 : dmax >= 256 ? 16 : dmax >= 128 ? 8 : 4;
}

// Every global load is unconditional, with clamped indexes (rows past `rows`
// read row row0, elements past d read element d - 1; neither is used), and
// the LayerNorm's gain and bias are loaded once before the rows: a load under
// a lane condition makes the compiler wait for it where the paths join, which
// would turn the loads of a row group into one memory round trip each.
template <int NJ, int G = kPrepGroup, bool PEND = false>  // d <= 64 * NJ; G rows per wave at once; PEND: in.nparts may be > 0
__device__ __forceinline__ void prepare_rows(const FusedIn& in, int rows, int row0, int d, int t, int8_t* a_lds,
                                             int lds_stride, bool writer) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  writer = writer && in.x_out != nullptr;
  const int n = (d + 63) / 64;
  float gj[NJ], bj[NJ];
  if (in.do_ln) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = min(lane + 64 * j, d - 1);
      gj[j] = in.g[i];
      bj[j] = in.b[i];
    }
  }
  for (int r0 = wave; r0 < rows; r0 += 4 * G) {
    float v[G][NJ];
    // the branches are uniform and hold whole loops, so that every load of
    // the group is issued before the first use in each of them
    if (in.embed) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int r = r0 + 4 * g;
        const size_t gr = (size_t)(row0 + (r < rows ? r : 0));
        int tok = in.tok[gr];
        tok = tok < 0 ? 0 : (tok >= in.V ? in.V - 1 : tok);
        const int pos = in.S_pos > 0 ? (int)(gr % (size_t)in.S_pos) : t;
        const float c = in.c_emb[tok];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int i = min(lane + 64 * j, d - 1);
          v[g][j] = fmaf((float)in.E[(size_t)tok * d + i], c, in.pe[(size_t)pos * d + i]);
        }
      }
    } else if (!PEND || in.nparts == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int r = r0 + 4 * g;
        const size_t gr = (size_t)(row0 + (r < rows ? r : 0));
#pragma unroll
        for (int j = 0; j < NJ; ++j) v[g][j] = in.x[gr * d + min(lane + 64 * j, d - 1)];
      }
    } else if constexpr (PEND) {
      // the pending update: the rows, their partial sums and the constants
      // loaded together (slices past nparts repeat the last, not added)
      int pa[G][kMaxSplits][NJ];
      float ps[NJ], pb[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int i = min(lane + 64 * j, d - 1);
        ps[j] = in.pscale[i];
        pb[j] = in.pbias[i];
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int r = r0 + 4 * g;
        const size_t gr = (size_t)(row0 + (r < rows ? r : 0));
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int i = min(lane + 64 * j, d - 1);
          v[g][j] = in.x[gr * d + i];
#pragma unroll
          for (int p = 0; p < kMaxSplits; ++p)
            pa[g][p][j] = in.part[(size_t)min(p, in.nparts - 1) * in.part_stride + gr * d + i];
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          int acc = pa[g][0][j];
#pragma unroll
          for (int p = 1; p < kMaxSplits; ++p) acc += p < in.nparts ? pa[g][p][j] : 0;
          v[g][j] = fmaf(in.pgamma, v[g][j], fmaf((float)acc, ps[j], pb[j]));
        }
    }
    if (writer && in.wb_input) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int r = r0 + 4 * g;
        if (r >= rows) continue;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int i = lane + 64 * j;
          if (j < n && i < d) in.x_out[(size_t)(row0 + r) * d + i] = v[g][j];
        }
      }
    }
    if (in.do_ln) {
      // mean: canonical sum of each row (lane partials over ascending i, then
      // the butterfly without the LDS crossbar)
      float p[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        p[g] = 0.0f;
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          if (j < n && lane + 64 * j < d) p[g] = p[g] + v[g][j];
      }
#pragma unroll
      for (int g = 0; g < G; ++g) p[g] = wave_sum(p[g]);
      const float inv_d = 1.0f / (float)d;
      float p2[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float mu = p[g] * inv_d;
        p2[g] = 0.0f;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          if (j < n && lane + 64 * j < d) {
            v[g][j] = v[g][j] - mu;
            p2[g] = fmaf(v[g][j], v[g][j], p2[g]);
          }
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) p2[g] = wave_sum(p2[g]);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float var = p2[g] * inv_d;
        const float rstd = 1.0f / sqrtf(var + in.eps);
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          if (j < n && lane + 64 * j < d) v[g][j] = fmaf(v[g][j] * rstd, gj[j], bj[j]);
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int r = r0 + 4 * g;
      if (r >= rows) continue;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int i = lane + 64 * j;
        if (j < n && i < d) {
          a_lds[r * lds_stride + i] = code_of(v[g][j] * in.inv_s);
          if (writer && !in.wb_input) in.x_out[(size_t)(row0 + r) * d + i] = v[g][j];
        }
      }
    }
  }
}

}  // namespace mnmt
