// decode_step.hip -- the decoder step for at most 2 rows (the batch-1 latency
// path) in 3 kernels per decoder layer plus the output projection and the
// commit, instead of one kernel per operation:
//   k_step_attn<SELF> (one block per head):
//       [pending residual update + LayerNorm + quantization of the rows]
//       -> the head's rows of Q (and K, V) -> [append K, V to the int8 cache]
//       -> attention -> the head's context times its columns of W_o, added
//       to an int32 accumulator (exact, so the heads may add in any order)
//   k_step_ffn (one block per 64 hidden units):
//       [pending update + LayerNorm + quantization] -> 64 rows of W1 + ReLU
//       requantization -> the hidden slice times its columns of W2 -> int32
//       accumulator
//   k_step_logits: [pending update + final LayerNorm] -> tied output
//       projection with the fused arg-max (spread over 32 slots per row)
// Each kernel's prologue applies the previous sublayer's epilogue
// x <- fma(gamma, x, fma(acc, scale, bias)) (and, for post-LN models, the
// LayerNorm that follows it) to the full rows it needs; block 0 stores the
// updated rows for the next update (into the other of two buffers, because
// the other blocks still read the old ones) and clears an accumulator whose
// consumer has finished.  This is the paper's fusion of everything between
// two GEMMs (Section 4.2) extended across the GEMM boundaries through the
// exact integer accumulators.
#include "blocks.hpp"
#include "internal.h"

namespace mnmt {
namespace {

constexpr int kStepRows = 2;     // rows (greedy batch) of this path
constexpr int kStepMaxLen = 128; // longest self / cross attention
constexpr int kStepHeadDim = 64; // widest head
constexpr int kFfnChunk = 64;    // hidden units per k_step_ffn block

// The rows of a sublayer input: y (fp32, the updated residual stream) and
// a = quant(LN(y)) or quant(y), in LDS.  Wave w prepares row w (R <= 2).
template <int NJ>
__device__ __forceinline__ void step_rows(const StepIn& in, int R, int d, int8_t* a_lds) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (blockIdx.x == 0 && in.zero_acc)
    for (int i = threadIdx.x; i < in.zero_n; i += blockDim.x) in.zero_acc[i] = 0;
  if (wave >= R) return;
  const int r = wave;
  float v[NJ];
  if (in.embed) {
    int tok = in.tok[r];
    tok = tok < 0 ? 0 : (tok >= in.V ? in.V - 1 : tok);
    const float c = in.c_emb[tok];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      v[j] = i < d ? fmaf((float)in.E[(size_t)tok * d + i], c, in.pe[(size_t)in.t * d + i]) : 0.0f;
    }
  } else if (in.acc) {
    // pending residual update of the previous sublayer (its fp32 epilogue)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      v[j] = i < d ? fmaf(in.gamma, in.x_in[(size_t)r * d + i],
                          fmaf((float)in.acc[(size_t)r * d + i], in.scale[i], in.bias[i]))
                   : 0.0f;
    }
  } else {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      v[j] = i < d ? in.x_in[(size_t)r * d + i] : 0.0f;
    }
  }
  const float inv_d = 1.0f / (float)d;
  // LayerNorm in the canonical order (element i in lane i % 64, ascending i)
  auto layer_norm = [&](const float* g, const float* b) {
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
    const float rstd = 1.0f / sqrtf(wave_sum(p2) * inv_d + in.eps);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (i < d) v[j] = fmaf(v[j] * rstd, g[i], b[i]);
    }
  };
  if (in.post_g) layer_norm(in.post_g, in.post_b);  // post-LN: normalize the residual stream
  if (blockIdx.x == 0 && in.x_out) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (i < d) in.x_out[(size_t)r * d + i] = v[j];
    }
  }
  if (in.pre_g) layer_norm(in.pre_g, in.pre_b);  // pre-LN: normalize the sublayer input
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = lane + 64 * j;
    if (i < d) a_lds[r * d + i] = code_of(v[j] * in.inv_s);
  }
}

// One block per head.  DMAX: model width class; rows of W are d bytes.
template <int DMAX, bool SELF>
__global__ __launch_bounds__(256) void k_step_attn(StepIn in, StepAttn at) {
  constexpr int LPR = lanes_per_row(DMAX);
  constexpr int RPI = 64 / LPR;
  constexpr int KC = (DMAX / 16 + LPR - 1) / LPR;           // 16-byte chunks per lane
  constexpr int NROWS = (SELF ? 3 : 1) * kStepHeadDim;       // projection rows per head (max)
  constexpr int U = (NROWS + 4 * RPI - 1) / (4 * RPI);       // row groups per wave
  constexpr int ND = (DMAX + 255) / 256;                     // W_o rows per thread
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kStepRows * DMAX];
  __shared__ __attribute__((aligned(16))) int8_t qkv[3][kStepRows][kStepHeadDim];
  __shared__ __attribute__((aligned(16))) int8_t ctx[kStepRows][kStepHeadDim];
  __shared__ AttnLdsT<kStepMaxLen, kStepHeadDim> att[kStepRows];
  const int hd = blockIdx.x;
  const int R = at.R, d = at.d, dh = at.dh;
  const int nrows = (SELF ? 3 : 1) * dh;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, kl = lane % LPR;
  auto row_of = [&](int j) { return (j / dh) * d + hd * dh + (j % dh); };
  // 1. weight loads: the head's projection rows and its W_o columns
  int4 wv[U][KC];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int j = (u * 4 + wave) * RPI + sub;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (kl + c * LPR) * 16;
      wv[u][c] = (j < nrows && k < d) ? *(const int4*)(at.W + (size_t)row_of(j) * d + k) : make_int4(0, 0, 0, 0);
    }
  }
  int4 wo[ND][kStepHeadDim / 16];
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    const int n = threadIdx.x + 256 * i;
#pragma unroll
    for (int c = 0; c < kStepHeadDim / 16; ++c)
      wo[i][c] = (n < d && 16 * c < dh) ? *(const int4*)(at.Wo + (size_t)n * d + hd * dh + 16 * c)
                                        : make_int4(0, 0, 0, 0);
  }
  // 2. the rows
  step_rows<(DMAX + 63) / 64>(in, R, d, a_lds);
  __syncthreads();
  // 3. Q (K, V) of the head, requantized
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int j = (u * 4 + wave) * RPI + sub;
    int acc[kStepRows] = {0, 0};
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (kl + c * LPR) * 16;
      if (k < d)
#pragma unroll
        for (int m = 0; m < kStepRows; ++m)
          if (m < R) acc[m] = dot16(wv[u][c], *(const int4*)(a_lds + m * d + k), acc[m]);
    }
#pragma unroll
    for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
      for (int m = 0; m < kStepRows; ++m) acc[m] += __shfl_xor(acc[m], off, 64);
    if (kl == 0 && j < nrows) {
      const int n = row_of(j);
#pragma unroll
      for (int m = 0; m < kStepRows; ++m)
        if (m < R) qkv[j / dh][m][j % dh] = code_of(fmaf((float)acc[m], at.scale[n], at.bias[n]));
    }
  }
  __syncthreads();
  // 4. attention, wave r for row r
  if (wave < R) {
    const int r = wave;
    if (SELF) {
      const int T = at.T, t = at.t;
      const int8_t* knew = qkv[1][r];
      const int8_t* vnew = qkv[2][r];
      for (int j = lane; j < dh; j += 64) {
        at.kcache[((size_t)r * T + t) * d + hd * dh + j] = knew[j];
        at.vcache[((size_t)r * T + t) * d + hd * dh + j] = vnew[j];
      }
      auto key = [&](int tp) -> const int8_t* {
        return tp == t ? knew : at.kcache + ((size_t)r * T + tp) * d + hd * dh;
      };
      auto val = [&](int tp) -> const int8_t* {
        return tp == t ? vnew : at.vcache + ((size_t)r * T + tp) * d + hd * dh;
      };
      attend_wave(qkv[0][r], t + 1, dh, key, val, at.c_qk, at.c_pv, ctx[r], att[r]);
    } else {
      int n = at.len[r];
      n = n < 1 ? 1 : (n > at.S ? at.S : n);
      const int8_t* base = at.kv + (size_t)r * at.S * 2 * d;
      auto key = [&](int s) -> const int8_t* { return base + (size_t)s * 2 * d + hd * dh; };
      auto val = [&](int s) -> const int8_t* { return base + (size_t)s * 2 * d + d + hd * dh; };
      attend_wave(qkv[0][r], n, dh, key, val, at.c_qk, at.c_pv, ctx[r], att[r]);
    }
  }
  __syncthreads();
  // 5. this head's share of the output projection, exact int32 partial sums
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    const int n = threadIdx.x + 256 * i;
    if (n >= d) continue;
#pragma unroll
    for (int m = 0; m < kStepRows; ++m) {
      if (m >= R) continue;
      int s = 0;
#pragma unroll
      for (int c = 0; c < kStepHeadDim / 16; ++c)
        if (16 * c < dh) s = dot16(wo[i][c], *(const int4*)(ctx[m] + 16 * c), s);
      atomicAdd(at.acc_out + (size_t)m * d + n, s);
    }
  }
}

// One block per kFfnChunk hidden units: W1 rows of the chunk (ReLU
// requantization), then the chunk's W2 columns into the int32 accumulator.
template <int DMAX>
__global__ __launch_bounds__(256) void k_step_ffn(StepIn in, StepFfn f) {
  constexpr int LPR = lanes_per_row(DMAX);
  constexpr int RPI = 64 / LPR;
  constexpr int KC = (DMAX / 16 + LPR - 1) / LPR;
  constexpr int U = (kFfnChunk + 4 * RPI - 1) / (4 * RPI);
  constexpr int ND = (DMAX + 255) / 256;
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kStepRows * DMAX];
  __shared__ __attribute__((aligned(16))) int8_t h[kStepRows][kFfnChunk];
  const int R = f.R, d = f.d, F = f.F;
  const int f0 = blockIdx.x * kFfnChunk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, kl = lane % LPR;
  int4 wv[U][KC];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int j = (u * 4 + wave) * RPI + sub;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (kl + c * LPR) * 16;
      wv[u][c] = (j < kFfnChunk && f0 + j < F && k < d) ? *(const int4*)(f.W1 + (size_t)(f0 + j) * d + k)
                                                         : make_int4(0, 0, 0, 0);
    }
  }
  int4 w2[ND][kFfnChunk / 16];
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    const int n = threadIdx.x + 256 * i;
#pragma unroll
    for (int c = 0; c < kFfnChunk / 16; ++c)
      w2[i][c] = (n < d && f0 + 16 * c < F) ? *(const int4*)(f.W2 + (size_t)n * F + f0 + 16 * c)
                                            : make_int4(0, 0, 0, 0);
  }
  step_rows<(DMAX + 63) / 64>(in, R, d, a_lds);
  __syncthreads();
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int j = (u * 4 + wave) * RPI + sub;
    int acc[kStepRows] = {0, 0};
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (kl + c * LPR) * 16;
      if (k < d)
#pragma unroll
        for (int m = 0; m < kStepRows; ++m)
          if (m < R) acc[m] = dot16(wv[u][c], *(const int4*)(a_lds + m * d + k), acc[m]);
    }
#pragma unroll
    for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
      for (int m = 0; m < kStepRows; ++m) acc[m] += __shfl_xor(acc[m], off, 64);
    if (kl == 0 && j < kFfnChunk) {
      const int n = f0 + j;
#pragma unroll
      for (int m = 0; m < kStepRows; ++m)
        if (m < R) h[m][j] = n < F ? code_of(fmaxf(fmaf((float)acc[m], f.scale1[n], f.bias1[n]), 0.0f)) : 0;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    const int n = threadIdx.x + 256 * i;
    if (n >= d) continue;
#pragma unroll
    for (int m = 0; m < kStepRows; ++m) {
      if (m >= R) continue;
      int s = 0;
#pragma unroll
      for (int c = 0; c < kFfnChunk / 16; ++c) s = dot16(w2[i][c], *(const int4*)(h[m] + 16 * c), s);
      atomicAdd(f.acc_out + (size_t)m * d + n, s);
    }
  }
}

// Output projection over the shared embedding with the fused arg-max.
template <int DMAX>
__global__ __launch_bounds__(256) void k_step_logits(StepIn in, StepLogits g) {
  constexpr int LPR = lanes_per_row(DMAX);
  constexpr int RPI = 64 / LPR;
  constexpr int KC = (DMAX / 16 + LPR - 1) / LPR;
  constexpr int U = 8;
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kStepRows * DMAX];
  __shared__ unsigned long long wmax[4][kStepRows];
  const int R = g.R, d = g.d, N = g.V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, kl = lane % LPR;
  const int row0 = (blockIdx.x * 4 + wave) * RPI * U;
  int4 wv[U][KC];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int n = row0 + u * RPI + sub;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (kl + c * LPR) * 16;
      wv[u][c] = (n < N && k < d) ? *(const int4*)(g.E + (size_t)n * d + k) : make_int4(0, 0, 0, 0);
    }
  }
  step_rows<(DMAX + 63) / 64>(in, R, d, a_lds);
  __syncthreads();
  unsigned long long best[kStepRows] = {0ull, 0ull};
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int n = row0 + u * RPI + sub;
    int acc[kStepRows] = {0, 0};
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int k = (kl + c * LPR) * 16;
      if (k < d)
#pragma unroll
        for (int m = 0; m < kStepRows; ++m)
          if (m < R) acc[m] = dot16(wv[u][c], *(const int4*)(a_lds + m * d + k), acc[m]);
    }
#pragma unroll
    for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
      for (int m = 0; m < kStepRows; ++m) acc[m] += __shfl_xor(acc[m], off, 64);
    if (kl == 0 && n < N) {
#pragma unroll
      for (int m = 0; m < kStepRows; ++m) {
        if (m < R) {
          const float z = (float)acc[m] * g.c_out[n];
          if (g.logits) g.logits[(size_t)m * N + n] = z;
          const unsigned long long key = pack_argmax(z, n);
          best[m] = key > best[m] ? key : best[m];
        }
      }
    }
  }
#pragma unroll
  for (int m = 0; m < kStepRows; ++m) {
    const unsigned long long w = wave_max_u64(best[m]);
    if (lane == 0) wmax[wave][m] = w;
  }
  __syncthreads();
  if (threadIdx.x < R) {
    const int m = threadIdx.x;
    unsigned long long b = wmax[0][m];
#pragma unroll
    for (int w = 1; w < 4; ++w) b = wmax[w][m] > b ? wmax[w][m] : b;
    if (b != 0ull) atomicMax(g.slots + m * g.nslots + blockIdx.x % g.nslots, b);
  }
}

}  // namespace

bool step_path_fits(int R, int d, int dh, int F, int T, int S) {
  return R >= 1 && R <= kStepRows && d <= 512 && d % 64 == 0 && dh <= kStepHeadDim && dh % 16 == 0 &&
         F % kFfnChunk == 0 && T <= kStepMaxLen && S <= kStepMaxLen;
}

#define MNMT_BY_D(d, CALL)            \
  switch (row_class(d)) {             \
    case 64: CALL(64); break;         \
    case 128: CALL(128); break;       \
    case 256: CALL(256); break;       \
    case 384: CALL(384); break;       \
    default: CALL(512); break;        \
  }

hipError_t launch_step_attn(const StepIn& in, const StepAttn& at, int self, int heads, hipStream_t s) {
#define MNMT_ATTN(DM)                                                                              \
  if (self)                                                                                        \
    hipLaunchKernelGGL((k_step_attn<DM, true>), dim3(heads), dim3(256), 0, s, in, at);              \
  else                                                                                             \
    hipLaunchKernelGGL((k_step_attn<DM, false>), dim3(heads), dim3(256), 0, s, in, at);
  MNMT_BY_D(at.d, MNMT_ATTN)
#undef MNMT_ATTN
  return hipGetLastError();
}

hipError_t launch_step_ffn(const StepIn& in, const StepFfn& f, hipStream_t s) {
  const int blocks = (f.F + kFfnChunk - 1) / kFfnChunk;
#define MNMT_FFN(DM) hipLaunchKernelGGL((k_step_ffn<DM>), dim3(blocks), dim3(256), 0, s, in, f);
  MNMT_BY_D(f.d, MNMT_FFN)
#undef MNMT_FFN
  return hipGetLastError();
}

hipError_t launch_step_logits(const StepIn& in, const StepLogits& g, hipStream_t s) {
  const int rpb = 4 * (64 / lanes_per_row(row_class(g.d))) * 8;  // rows per block
  const int blocks = (g.V + rpb - 1) / rpb;
#define MNMT_LOGITS(DM) hipLaunchKernelGGL((k_step_logits<DM>), dim3(blocks), dim3(256), 0, s, in, g);
  MNMT_BY_D(g.d, MNMT_LOGITS)
#undef MNMT_LOGITS
  return hipGetLastError();
}

}  // namespace mnmt
