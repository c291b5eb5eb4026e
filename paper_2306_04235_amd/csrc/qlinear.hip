// qlinear.hip -- int8 x int8 -> int32 linear layers with fused epilogues
// (8-bit GEMM of Section 4.1; requantization, bias, ReLU, residual and
// dequantization fused between GEMMs as in Section 4.2).
//
// Two kernels:
//  * qgemv: M <= 8 rows (batch-1 decoding).  Bandwidth bound: every weight
//    byte is read once.  A weight row of K bytes is split over LPR lanes that
//    each load 16 contiguous bytes (one dwordx4) per step, so one wave
//    instruction reads 64 * 16 = 1024 contiguous bytes; U independent row
//    groups per wave keep several loads in flight.  Products use the 4-way
//    int8 dot instruction; the LPR partial sums meet in an xor butterfly.
//  * qgemm_small: 8 < M <= 64 and K <= 1024 (the batch-1 encoder), and the
//    batched decoder's 65-512-row projections of moderate N, 16x16x64
//    matrix-core fragments loaded straight from memory.
// Larger M runs the tiled matrix-core GEMM of gemm.hip.
// Integer accumulation is exact, so neither kernel's order matters; the fp32
// epilogue is the same single expression in both.
#include "blocks.hpp"
#include "internal.h"

namespace mnmt {
namespace {


// The epilogue operands of one lane's column (and, for the residual, of its
// rows), loaded before the matrix product so that they arrive with the
// operands instead of one round trip after it.
struct EpiPre {
  float sc = 0.0f, bi = 0.0f;
  float y[4] = {0.0f, 0.0f, 0.0f, 0.0f};
};

// Whether epilogue kind k is one that epilogue_pre handles.
__device__ __forceinline__ bool epi_pre_kind(int k) {
  return k == MNMT_EPI_I8 || k == MNMT_EPI_I8_RELU || k == MNMT_EPI_F32_RESID;
}

// The same expressions as epilogue_store, from the preloaded operands.
__device__ __forceinline__ void epilogue_pre(const EpiArgs& e, int m, int n, int acc, const EpiPre& p, int i) {
  const float a = (float)acc;
  const size_t o = (size_t)m * e.ldo + n;
  if (e.kind == MNMT_EPI_I8)
    ((int8_t*)e.out)[o] = code_of(fmaf(a, p.sc, p.bi));
  else if (e.kind == MNMT_EPI_I8_RELU)
    ((int8_t*)e.out)[o] = code_of(fmaxf(fmaf(a, p.sc, p.bi), 0.0f));
  else
    ((float*)e.out)[o] = fmaf(e.gamma, p.y[i], fmaf(a, p.sc, p.bi));
}

// The fused epilogue of one output element (row m, column n).
__device__ __forceinline__ void epilogue_store(const EpiArgs& e, int m, int n, int acc, const float* scale,
                                               const float* bias) {
  const float a = (float)acc;
  const size_t o = (size_t)m * e.ldo + n;
  switch (e.kind) {
    case MNMT_EPI_I32:
      ((int*)e.out)[o] = acc;
      break;
    case MNMT_EPI_I8:
      ((int8_t*)e.out)[o] = code_of(fmaf(a, scale[n], bias[n]));
      break;
    case MNMT_EPI_I8_RELU:
      ((int8_t*)e.out)[o] = code_of(fmaxf(fmaf(a, scale[n], bias[n]), 0.0f));
      break;
    case MNMT_EPI_F32:
      ((float*)e.out)[o] = fmaf(a, scale[n], bias[n]);
      break;
    case MNMT_EPI_F32_RESID: {
      float* y = (float*)e.out + o;
      *y = fmaf(e.gamma, *y, fmaf(a, scale[n], bias[n]));
      break;
    }
    default:  // LOGITS
      ((float*)e.out)[o] = a * scale[n];
      break;
  }
}

// ---------------------------------------------------------------------------
// qgemv: MR = max rows of X, LPR = lanes per weight row, U = row groups per wave
// W4: W holds packed 4-bit rows (K / 2 bytes each), widened in registers.
template <int MR, int LPR, int U, bool W4>
__global__ __launch_bounds__(256) void k_qgemv(const int8_t* __restrict__ X, int ldx, const int8_t* __restrict__ W,
                                               int M, int K, int N, const float* __restrict__ scale,
                                               const float* __restrict__ bias, EpiArgs e) {
  constexpr int RPI = 64 / LPR;  // weight rows per wave instruction
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int sub = lane / LPR;
  const int kl = lane % LPR;
  const int row0 = wave * RPI * U;
  int acc[U][MR];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[u][m] = 0;

  for (int k = kl * 16; k < K; k += LPR * 16) {
    WFrag<W4> wv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int n = row0 + u * RPI + sub;
      wv[u] = load_wfrag_if<W4>(n < N, W, n, K, k);
    }
#pragma unroll
    for (int m = 0; m < MR; ++m) {
      if (m < M) {
        const int4 xv = *(const int4*)(X + (size_t)m * ldx + k);
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u][m] = dot16(wv[u].get(), xv, acc[u][m]);
      }
    }
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MR; ++m) acc[u][m] += __shfl_xor(acc[u][m], off, 64);

  if (e.kind == EPI_LOGITS_ARGMAX) {
#pragma unroll
    for (int m = 0; m < MR; ++m) {
      if (m >= M) break;
      unsigned long long best = 0ull;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int n = row0 + u * RPI + sub;
        if (kl == 0 && n < N) {
          const float z = (float)acc[u][m] * scale[n];
          if (e.out) ((float*)e.out)[(size_t)m * e.ldo + n] = z;
          const unsigned long long key = pack_argmax(z, n);
          best = key > best ? key : best;
        }
      }
      best = wave_max_u64(best);
      if (lane == 0 && best != 0ull) atomicMax(e.argmax + m, best);
    }
    return;
  }
  if (kl != 0) return;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int n = row0 + u * RPI + sub;
    if (n >= N) continue;
#pragma unroll
    for (int m = 0; m < MR; ++m)
      if (m < M) epilogue_store(e, m, n, acc[u][m], scale, bias);
  }
}

template <int MR, int LPR, bool W4>
hipError_t gemv_u(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                  int N, const EpiArgs& e, hipStream_t s) {
  constexpr int RPI = 64 / LPR;
  // Enough waves to cover the chip: fewer row groups per wave for small N.
  const long waves4 = ((long)N + RPI * 4 - 1) / (RPI * 4);
  if (waves4 >= 1024) {
    const int blocks = (int)((waves4 + 3) / 4);
    hipLaunchKernelGGL((k_qgemv<MR, LPR, 4, W4>), dim3(blocks), dim3(256), 0, s, X, ldx, W, M, K, N, scale, bias, e);
  } else if (waves4 * 2 >= 1024) {
    const long waves = ((long)N + RPI * 2 - 1) / (RPI * 2);
    hipLaunchKernelGGL((k_qgemv<MR, LPR, 2, W4>), dim3((int)((waves + 3) / 4)), dim3(256), 0, s, X, ldx, W, M, K, N,
                       scale, bias, e);
  } else {
    const long waves = ((long)N + RPI - 1) / RPI;
    hipLaunchKernelGGL((k_qgemv<MR, LPR, 1, W4>), dim3((int)((waves + 3) / 4)), dim3(256), 0, s, X, ldx, W, M, K, N,
                       scale, bias, e);
  }
  return hipGetLastError();
}

template <int MR, bool W4>
hipError_t gemv_lpr(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                    int N, const EpiArgs& e, hipStream_t s) {
  const int chunks = K / 16;
  if (chunks >= 64) return gemv_u<MR, 64, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (chunks >= 32) return gemv_u<MR, 32, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (chunks >= 16) return gemv_u<MR, 16, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (chunks >= 8) return gemv_u<MR, 8, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  return gemv_u<MR, 4, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
}

// ---------------------------------------------------------------------------
// qgemm_small: K <= 1024, up to 512 rows (see qgemm_rows_fit).  A 32x32 output tile
// per block, one 16x16 tile per wave on v_mfma_i32_16x16x64_i8.  Each lane's
// operand is 16 contiguous K bytes of one row, so weight fragments are loaded
// straight from global memory, all of K at once (a single round trip).  The
// input rows come from global int8 X or, with LN, from prepare_rows
// (embedding / LayerNorm / quantization of fp32 rows) into LDS.
constexpr int kSmallMaxK = 1024;

// WAVES 4: a 32x32 tile per block; WAVES 1 (no LN): a 16x16 tile per
// one-wave block, four times the blocks over the same waves.  WIDE (with LN):
// 16 rows x 64 columns per block, wave w the columns 16 w.., so that each
// wave normalizes 4 of the rows (the LayerNorm is repeated by every column
// block, and its instructions, not the loads, set the prologue's length).
// W4: W holds packed 4-bit rows (K / 2 bytes each), widened in registers.
template <bool LN, int KMAX, int WAVES = 4, bool W4 = false, bool WIDE = false>  // K <= KMAX
__global__ __launch_bounds__(64 * WAVES) void k_qgemm_small(FusedIn in, const int8_t* __restrict__ X, int ldx,
                                                            const int8_t* __restrict__ W, int M, int K, int N,
                                                            const float* __restrict__ scale,
                                                            const float* __restrict__ bias, EpiArgs e) {
  static_assert(WAVES == 4 || (WAVES == 1 && !LN), "32x32 tiles, or 16x16 without the row prologue");
  static_assert(!WIDE || (LN && WAVES == 4), "16x64 tiles normalize their rows");
  constexpr int NK = (KMAX + 63) / 64;
  constexpr int TM = WIDE ? 16 : WAVES == 4 ? 32 : 16, TN = WIDE ? 64 : TM;
  __shared__ __attribute__((aligned(16))) int8_t As[LN ? TM * (KMAX + 16) : 16];
  const int lane = threadIdx.x & 63, wave = WAVES == 4 ? threadIdx.x >> 6 : 0;
  const int wm = WIDE ? 0 : wave >> 1, wn = WIDE ? wave : wave & 1;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  const int nk = K / 64;
  const int col = n0 + 16 * wn + (lane & 15);
  const int koff = 16 * (lane >> 4);
  WFrag<W4> bf[NK];
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) bf[kk] = load_wfrag_if<W4>(kk < nk && col < N, W, col, K, kk * 64 + koff);
  const int arow = m0 + 16 * wm + (lane & 15);
  // the epilogue's operands (clamped indexes, unused past M or N)
  EpiPre pre;
  const bool pre_ok = epi_pre_kind(e.kind);
  if (pre_ok) {
    const int cc = col < N ? col : N - 1;
    pre.sc = scale[cc];
    pre.bi = bias[cc];
    if (e.kind == MNMT_EPI_F32_RESID) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + 16 * wm + 4 * (lane >> 4) + i;
        pre.y[i] = ((const float*)e.out)[(size_t)(row < M ? row : M - 1) * e.ldo + cc];
      }
    }
  }
  v4i acc = {0, 0, 0, 0};
  if (LN) {
    const int KP = K + 16;
    const int rows = M - m0 < TM ? M - m0 : TM;
    // the wave's TM / 4 rows in one group (one round trip) up to 512-wide rows
    prepare_rows<(KMAX + 63) / 64, KMAX <= 512 ? TM / 4 : kPrepGroup>(in, rows, m0, K, 0, As, KP, blockIdx.x == 0);
    __syncthreads();
    const int lr = 16 * wm + (lane & 15);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      if (kk < nk) {
        const v4i a = lr < rows ? *(const v4i*)(As + lr * KP + kk * 64 + koff) : v4i{0, 0, 0, 0};
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, bf[kk].get(), acc, 0, 0, 0);
      }
    }
  } else {
    v4i af[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk)
      af[kk] = (kk < nk && arow < M) ? *(const v4i*)(X + (size_t)arow * ldx + kk * 64 + koff) : v4i{0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < NK; ++kk)
      if (kk < nk) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[kk], bf[kk].get(), acc, 0, 0, 0);
  }
  // 16x16 fragment: element i of lane l sits at row 4*(l/16) + i, column l%16
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + 16 * wm + 4 * (lane >> 4) + i;
    if (row < M && col < N) {
      if (pre_ok)
        epilogue_pre(e, row, col, acc[i], pre, i);
      else
        epilogue_store(e, row, col, acc[i], scale, bias);
    }
  }
}

}  // namespace

bool qgemm_small_fits(int M, int K) { return M >= 1 && M <= 64 && K <= kSmallMaxK && K % 64 == 0; }

// Up to 256 rows and N <= 1024, or 512 rows and N <= 512, the one-round-trip
// kernel (every block loads its weight fragments for all of K at once) also
// beats the LDS-slab GEMM, whose 64x64 tiles leave such shapes with a few
// dozen blocks (the batched decoder's projections and feed-forward layers).
// At 512 rows with N >= 1536, or N = 2048, the repeated weight loads make it
// the slower of the two.
constexpr int kSmallMaxRows = 512;
bool qgemm_rows_fit(int M, int K, int N) {
  return M >= 1 && (M <= 256 ? N <= 1024 : M <= kSmallMaxRows && N <= 512) && K <= kSmallMaxK && K % 64 == 0;
}

hipError_t launch_qgemm_small(const FusedIn* in, const int8_t* X, int ldx, const int8_t* W, const float* scale,
                              const float* bias, int M, int K, int N, const EpiArgs& e, hipStream_t s, bool w4) {
  if (M < 1 || M > kSmallMaxRows || K > kSmallMaxK || K % 64 || (in && (K > kMaxRowLen || in->nparts)))
    return hipErrorInvalidValue;
  // 65-256 rows (the mobile beam decoder): one-wave blocks of 16x16 (at 512
  // rows their four-fold block count made the base beam step slower); rows
  // normalized in the prologue above 64 rows: 16x64 tiles
  const bool one = !in && M > 64 && M <= 256, wide = in && M > 64;
  const dim3 grid = one    ? dim3((N + 15) / 16, (M + 15) / 16)
                    : wide ? dim3((N + 63) / 64, (M + 15) / 16)
                           : dim3((N + 31) / 32, (M + 31) / 32);
  const FusedIn none{};
#define MNMT_SMALL_W(KM, W4)                                                                                   \
  if (wide)                                                                                                    \
    hipLaunchKernelGGL((k_qgemm_small<true, KM, 4, W4, true>), grid, dim3(256), 0, s, *in, X, ldx, W, M, K, N,  \
                       scale, bias, e);                                                                        \
  else if (in)                                                                                                 \
    hipLaunchKernelGGL((k_qgemm_small<true, KM, 4, W4>), grid, dim3(256), 0, s, *in, X, ldx, W, M, K, N, scale, \
                       bias, e);                                                                               \
  else if (one)                                                                                                \
    hipLaunchKernelGGL((k_qgemm_small<false, KM, 1, W4>), grid, dim3(64), 0, s, none, X, ldx, W, M, K, N, scale, \
                       bias, e);                                                                               \
  else                                                                                                         \
    hipLaunchKernelGGL((k_qgemm_small<false, KM, 4, W4>), grid, dim3(256), 0, s, none, X, ldx, W, M, K, N, scale, \
                       bias, e);
#define MNMT_SMALL(KM)      \
  if (w4) {                 \
    MNMT_SMALL_W(KM, true)  \
  } else {                  \
    MNMT_SMALL_W(KM, false) \
  }
  switch (row_class(K)) {
    case 64: MNMT_SMALL(64) break;
    case 128: MNMT_SMALL(128) break;
    case 256: MNMT_SMALL(256) break;
    case 384: MNMT_SMALL(384) break;
    case 512: MNMT_SMALL(512) break;
    default: MNMT_SMALL(1024) break;
  }
#undef MNMT_SMALL
#undef MNMT_SMALL_W
  return hipGetLastError();
}

template <bool W4>
hipError_t gemv_rows(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                     int N, const EpiArgs& e, hipStream_t s) {
  if (M == 1) return gemv_lpr<1, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (M == 2) return gemv_lpr<2, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (M <= 4) return gemv_lpr<4, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  return gemv_lpr<8, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
}

int qgemm_splits(int M, int K, int N) {
  if (M <= 8 || M > kSmallMaxRows || N > 1024 || K <= kSmallMaxK || K % kSplitKb || K / kSplitKb > kMaxSplits)
    return 0;
  return K / kSplitKb;
}

hipError_t launch_qgemm_split(const int8_t* X, int ldx, const int8_t* W, int M, int K, int N, int32_t* part,
                              hipStream_t s, bool w4) {
  const int splits = qgemm_splits(M, K, N);
  if (!splits) return hipErrorInvalidValue;
  return launch_gemm_split(X, ldx, W, M, K, N, splits, part, s, w4);
}

hipError_t launch_qlinear(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M,
                          int K, int N, const EpiArgs& e, hipStream_t s, bool w4) {
  if (M <= 0) return hipSuccess;
  if (w4 && (e.kind == EPI_LOGITS_ARGMAX || K % 64)) return hipErrorInvalidValue;
  if (M <= 8)
    return w4 ? gemv_rows<true>(X, ldx, W, scale, bias, M, K, N, e, s)
              : gemv_rows<false>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (e.kind == EPI_LOGITS_ARGMAX) return hipErrorInvalidValue;  // arg-max fusion is a batch-1 path
  if (qgemm_small_fits(M, K) || qgemm_rows_fit(M, K, N))
    return launch_qgemm_small(nullptr, X, ldx, W, scale, bias, M, K, N, e, s, w4);
  return launch_gemm(X, ldx, W, scale, bias, M, K, N, e, s, w4);
}

}  // namespace mnmt
