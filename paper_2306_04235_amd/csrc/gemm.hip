// gemm.hip -- int8 GEMM with fused epilogues for more than 64 rows (the
// batched encoder, beam decoding and the quantized-linear sweep), on the i8
// matrix cores: Y[m, n] = epilogue(sum_k X[m, k] W[n, k]) (Section 4.1's 8-bit
// GEMM; the epilogues of Section 4.2 applied as the tile is written).
//
// Tiles.  A 256-thread block owns a BN x BM tile of (output column n, row m);
// its 4 waves split it WN x WM.  K is walked in 64-byte slabs staged through
// LDS with double buffering: the next slab's global loads are in flight while
// the current one feeds v_mfma_i32_32x32x32_i8, one LDS barrier per slab.
// Loads clamp their row index instead of branching, so rows past M or N read
// valid memory and produce outputs that are never stored.
//
// Operand order.  W is the MFMA A operand and X the B operand, so a 32x32
// accumulator holds D[n][m]: element r of lane l is column n = 8 (r / 4) +
// 4 (l / 32) + r % 4 of row m = l % 32, four consecutive columns per r / 4.
// For int8 outputs two v_permlane32_swap exchanges between lanes l and l + 32
// leave each lane with 16 consecutive columns of one row, written by one
// 16-byte store; fp32 and int32 outputs are written 4 columns per store.
//
// Accumulators live in VGPRs (the file is built with the MFMA VGPR form), so
// the epilogue reads them without accumulator-register moves.
//
// Placement.  Blocks are dispatched to the 8 XCDs round-robin; the linear
// block id is remapped so that each XCD works through one contiguous range of
// tiles (m fastest), which keeps the W and X tiles it shares in its own L2.
#include "blocks.hpp"
#include "internal.h"

namespace mnmt {
namespace {

typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kBK = 64;            // K bytes per slab
constexpr int kLdsRow = kBK + 16;  // padded LDS row (spreads rows over banks)
constexpr int kXcds = 8;

// clamp(rint(y), -127, 127) in the low byte: after the clamp, adding 1.5 * 2^23
// rounds to an integer (round half to even, as rintf) and leaves it in the
// low mantissa bits in two's complement.  NaN clamps to -127 as in code_of.
__device__ __forceinline__ uint32_t code_bits(float y) {
  return __float_as_uint(fminf(fmaxf(y, -127.0f), 127.0f) + 12582912.0f);
}
// Low bytes of a, b, c, d in bytes 0..3 (three byte permutes).
__device__ __forceinline__ uint32_t pack4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  const uint32_t ab = __builtin_amdgcn_perm(b, a, 0x0c0c0400u);  // [a0, b0, 0, 0]
  const uint32_t cd = __builtin_amdgcn_perm(d, c, 0x0c0c0400u);  // [c0, d0, 0, 0]
  return __builtin_amdgcn_perm(cd, ab, 0x05040100u);            // [a0, b0, c0, d0]
}

template <int EPI>
__device__ __forceinline__ float epi_value(int acc, float sc, float bi) {
  const float a = (float)acc;
  if (EPI == MNMT_EPI_LOGITS) return a * sc;
  const float y = fmaf(a, sc, bi);
  return EPI == MNMT_EPI_I8_RELU ? fmaxf(y, 0.0f) : y;
}

// Writes one 32x32 accumulator fragment (columns nb .. nb + 31, this lane's
// row m = row of lane l % 32).  FAST: the whole fragment is inside the output
// and rows are 16-byte aligned, so no lane checks anything.
template <int EPI, bool FAST>
__device__ __forceinline__ void store_fragment(const EpiArgs& e, const v16i& c, const float (&sc)[4][4],
                                               const float (&bi)[4][4], int m, int nb, int h, int M, int N) {
  constexpr bool INT8_OUT = EPI == MNMT_EPI_I8 || EPI == MNMT_EPI_I8_RELU;
  if (INT8_OUT) {
    uint32_t w4[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t q[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) q[t] = code_bits(epi_value<EPI>(c[4 * g + t], sc[g][t], bi[g][t]));
      w4[g] = pack4(q[0], q[1], q[2], q[3]);
    }
    // lanes l and l + 32 trade groups (the upper half of the first operand
    // with the lower half of the second): lane l ends with columns
    // nb + 0..15, lane l + 32 with nb + 16..31, 4 columns per word
    const auto s02 = __builtin_amdgcn_permlane32_swap(w4[0], w4[2], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w4[1], w4[3], false, false);
    const uint32_t o[4] = {s02[0], s02[1], s13[0], s13[1]};
    int n = nb + 16 * h;
    if (!FAST) asm volatile("" : "+v"(n), "+v"(m));  // keeps the checks below inside this path
    int8_t* y = (int8_t*)e.out + (size_t)m * e.ldo + n;
    if (FAST) {
      *(v4i*)y = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    } else if (m < M) {
#pragma unroll
      for (int t = 0; t < 16; ++t)
        if (n + t < N) y[t] = (int8_t)(o[t >> 2] >> (8 * (t & 3)));
    }
    return;
  }
  if (!FAST) asm volatile("" : "+v"(nb), "+v"(m));
  if (!FAST && m >= M) return;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int n = nb + 8 * g + 4 * h;
    if (EPI == MNMT_EPI_I32) {
      int* y = (int*)e.out + (size_t)m * e.ldo + n;
      if (FAST) {
        *(v4i*)y = v4i{c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (n + t < N) y[t] = c[4 * g + t];
      }
    } else {
      float* y = (float*)e.out + (size_t)m * e.ldo + n;
      v4f v;
#pragma unroll
      for (int t = 0; t < 4; ++t) v[t] = epi_value<EPI>(c[4 * g + t], sc[g][t], bi[g][t]);
      if (FAST) {
        if (EPI == MNMT_EPI_F32_RESID) {
          const v4f old = *(const v4f*)y;
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = fmaf(e.gamma, old[t], v[t]);
        }
        *(v4f*)y = v;
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (n + t < N) y[t] = EPI == MNMT_EPI_F32_RESID ? fmaf(e.gamma, y[t], v[t]) : v[t];
      }
    }
  }
}

// W4: W holds packed 4-bit rows [N, K / 2]; each 16-code chunk is loaded as
// its 8 packed bytes and widened to int8 on its way into LDS.  K split
// (gridDim.y > 1, MNMT_EPI_I32): block row y takes columns [y kb, (y + 1) kb)
// of K (the row length) and stores its int32 partial sums into slice y of
// e.out, M * e.ldo words apart.
template <int BN, int BM, int WN, int WM, int EPI, bool W4>
__global__ __launch_bounds__(256) void k_gemm(const int8_t* __restrict__ X, int ldx, const int8_t* __restrict__ W,
                                              int M, int K, int N, const float* __restrict__ scale,
                                              const float* __restrict__ bias, EpiArgs e, int tiles_m, int tiles,
                                              int kb) {
  static_assert(WN * WM == 4, "4 waves");
  constexpr int TN = BN / WN, TM = BM / WM;  // wave tile
  constexpr int FN = TN / 32, FM = TM / 32;  // 32x32 fragments per wave
  static_assert(FN >= 1 && FM >= 1, "whole fragments");
  constexpr int CW = BN * (kBK / 16) / 256, CX = BM * (kBK / 16) / 256;  // 16-byte chunks per thread
  static_assert(CW >= 1 && CX >= 1, "every thread loads");
  constexpr bool INT8_OUT = EPI == MNMT_EPI_I8 || EPI == MNMT_EPI_I8_RELU;
  __shared__ __attribute__((aligned(16))) int8_t Ws[2][BN * kLdsRow];
  __shared__ __attribute__((aligned(16))) int8_t Xs[2][BM * kLdsRow];
  __shared__ float sc_lds[BN], bi_lds[BN];  // the tile's epilogue constants

  // tile of this block: XCD x takes tiles [x * per, (x + 1) * per), m fastest
  const int b = blockIdx.x;
  const int per = (tiles + kXcds - 1) / kXcds;
  const int tile = (b % kXcds) * per + b / kXcds;
  if (tile >= tiles) return;  // the grid is rounded up to whole XCD ranges
  const int m0 = (tile % tiles_m) * BM, n0 = (tile / tiles_m) * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave / WM, wm = wave % WM;
  const int l32 = lane & 31, h = lane >> 5;

  if (EPI != MNMT_EPI_I32) {
    for (int c = tid; c < BN; c += 256) {
      const int n = min(n0 + c, N - 1);
      sc_lds[c] = scale[n];
      bi_lds[c] = EPI == MNMT_EPI_LOGITS ? 0.0f : bias[n];
    }
  }

  // 32-bit offsets of this thread's 16-byte chunks (the slab adds k0; in
  // packed 4-bit rows a chunk is 8 bytes)
  constexpr int WDIV = W4 ? 2 : 1;
  uint32_t ow[CW], ox[CX];
#pragma unroll
  for (int i = 0; i < CW; ++i) {
    const int c = tid + 256 * i;
    ow[i] = (uint32_t)min(n0 + (c >> 2), N - 1) * (uint32_t)(K / WDIV) + 16 / WDIV * (c & 3);
  }
#pragma unroll
  for (int i = 0; i < CX; ++i) {
    const int c = tid + 256 * i;
    ox[i] = (uint32_t)min(m0 + (c >> 2), M - 1) * (uint32_t)ldx + 16 * (c & 3);
  }
  WFrag<W4> rw[CW];
  v4i rx[CX];
  const int kbeg = blockIdx.y * kb;  // this block's first K column
  if (gridDim.y > 1) e.out = (int*)e.out + (size_t)blockIdx.y * M * e.ldo;
  auto gload = [&](int k0) {
    const int8_t* wk = W + (kbeg + k0) / WDIV;
    const int8_t* xk = X + kbeg + k0;
#pragma unroll
    for (int i = 0; i < CW; ++i) {
      if constexpr (W4)
        rw[i].p = *(const uint2*)(wk + ow[i]);
      else
        rw[i].v = *(const v4i*)(wk + ow[i]);
    }
#pragma unroll
    for (int i = 0; i < CX; ++i) rx[i] = *(const v4i*)(xk + ox[i]);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CW; ++i) {
      const int c = tid + 256 * i;
      *(v4i*)(&Ws[buf][(c >> 2) * kLdsRow + 16 * (c & 3)]) = rw[i].get();
    }
#pragma unroll
    for (int i = 0; i < CX; ++i) {
      const int c = tid + 256 * i;
      *(v4i*)(&Xs[buf][(c >> 2) * kLdsRow + 16 * (c & 3)]) = rx[i];
    }
  };

  v16i acc[FN][FM];
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int i = 0; i < FM; ++i) acc[j][i] = v16i{};

  const int slabs = kb / kBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int s = 0; s < slabs; ++s) {
    const int buf = s & 1;
    if (s + 1 < slabs) gload((s + 1) * kBK);
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 32) {
      v4i a[FN], bx[FM];
#pragma unroll
      for (int j = 0; j < FN; ++j)
        a[j] = *(const v4i*)(&Ws[buf][(wn * TN + 32 * j + l32) * kLdsRow + kk + 16 * h]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
        bx[i] = *(const v4i*)(&Xs[buf][(wm * TM + 32 * i + l32) * kLdsRow + kk + 16 * h]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[j], bx[i], acc[j][i], 0, 0, 0);
    }
    if (s + 1 < slabs) lstore(buf ^ 1);
    __syncthreads();
  }

  // epilogue: whole fragments take the check-free path
  const bool aligned = INT8_OUT ? (e.ldo % 16 == 0 && (reinterpret_cast<uintptr_t>(e.out) & 15) == 0)
                                : (e.ldo % 4 == 0 && (reinterpret_cast<uintptr_t>(e.out) & 15) == 0);
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int cb = wn * TN + 32 * j;  // fragment's first column within the tile
    float sc[4][4], bi[4][4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const v4f s4 = *(const v4f*)(sc_lds + cb + 8 * g + 4 * h);
      const v4f b4 = *(const v4f*)(bi_lds + cb + 8 * g + 4 * h);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        sc[g][t] = EPI == MNMT_EPI_I32 ? 0.0f : s4[t];
        bi[g][t] = EPI == MNMT_EPI_I32 ? 0.0f : b4[t];
      }
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int mb = m0 + wm * TM + 32 * i;
      const bool fast = aligned && n0 + cb + 32 <= N && mb + 32 <= M;  // uniform over the wave
      if (fast)
        store_fragment<EPI, true>(e, acc[j][i], sc, bi, mb + l32, n0 + cb, h, M, N);
      else
        store_fragment<EPI, false>(e, acc[j][i], sc, bi, mb + l32, n0 + cb, h, M, N);
    }
  }
}

// Persistent variant for whole BN x BM tiles (M and N multiples of the tile,
// K = KC KCN) and many of them.  Each block (4 waves, 2 per CU) walks its
// XCD's tiles with a stride; a tile's K is taken in KC-byte chunks, each held
// whole in LDS, and the next chunk (of this tile or the next) is loaded into
// registers while the current one feeds the matrix cores and while the
// finished tile's epilogue runs, so the loads of a tile overlap the previous
// tile's work instead of being exposed at its start.  The barriers order LDS
// only, so the prefetch stays in flight across them.  The loop body is
// straight-line (the chunk loop unrolled, the prefetch unconditional: after
// the last tile it reloads that tile), so the wait for the prefetch before it
// goes to LDS does not include the tile's output stores issued after it
// (loads and stores share one in-order counter).
// W4: packed 4-bit rows, widened on their way into LDS (as k_gemm).
template <int EPI, int BN, int BM, int KC, int KCN, bool W4>
__global__ __launch_bounds__(256) void k_gemm_p(const int8_t* X, int ldx, const int8_t* W, int M, int K, int N,
                                                const float* scale, const float* bias, EpiArgs e, int tiles_m,
                                                int tiles, int nblk) {
  constexpr int ROW = KC + 16;                 // padded LDS row
  constexpr int CPR = KC / 16;                 // 16-byte chunks per row
  constexpr int LW = BN * CPR / 256, LX = BM * CPR / 256;  // loads per thread and chunk
  constexpr int FN = BN / 64, FM = BM / 64;    // 32 x 32 fragments per wave (2 x 2 waves)
  static_assert(LW >= 1 && LX >= 1 && BN * CPR % 256 == 0 && BM * CPR % 256 == 0, "whole loads");
  static_assert(256 % CPR == 0, "a load step covers whole rows");
  constexpr int RPS = 256 / CPR;               // rows per load step
  __shared__ __attribute__((aligned(16))) int8_t Ws[BN * ROW];
  __shared__ __attribute__((aligned(16))) int8_t Xs[BM * ROW];
  __shared__ __attribute__((aligned(16))) float sc_lds[2][BN], bi_lds[2][BN];  // per tile, alternating

  // tiles of this block: its XCD's contiguous range (m fastest), strided by
  // the XCD's block count
  const int xcd = blockIdx.x % kXcds, nbx = nblk / kXcds;
  const int per = (tiles + kXcds - 1) / kXcds;
  const int end = min((xcd + 1) * per, tiles);
  int tile = xcd * per + blockIdx.x / kXcds;
  if (tile >= end) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave >> 1, wm = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;
  const int lrow = tid / CPR, lcol = 16 * (tid % CPR);  // this thread's loads: rows lrow + RPS i, 16 bytes at lcol

  WFrag<W4> rw[LW];
  v4i rx[LX];
  float rs[(2 * BN + 255) / 256];
  auto gload = [&](int t, int c) {  // c: compile-time after unrolling
    const int m0 = (t % tiles_m) * BM, n0 = (t / tiles_m) * BN;
    const int k0 = c * KC + lcol;
#pragma unroll
    for (int i = 0; i < LW; ++i) rw[i] = load_wfrag<W4>(W, (size_t)(n0 + lrow + RPS * i), K, k0);
#pragma unroll
    for (int i = 0; i < LX; ++i) rx[i] = *(const v4i*)(X + (size_t)(m0 + lrow + RPS * i) * ldx + k0);
    if (c == 0 && EPI != MNMT_EPI_I32) {
#pragma unroll
      for (int i = 0; i < (2 * BN + 255) / 256; ++i) {
        const int q = tid + 256 * i;  // scale[0..BN), then bias[0..BN)
        if (q < 2 * BN) rs[i] = q < BN ? scale[n0 + q] : (EPI == MNMT_EPI_LOGITS ? 0.0f : bias[n0 + q - BN]);
      }
    }
  };
  auto lstore = [&](int c, int sb) {
#pragma unroll
    for (int i = 0; i < LW; ++i) *(v4i*)(&Ws[(lrow + RPS * i) * ROW + lcol]) = rw[i].get();
#pragma unroll
    for (int i = 0; i < LX; ++i) *(v4i*)(&Xs[(lrow + RPS * i) * ROW + lcol]) = rx[i];
    if (c == 0 && EPI != MNMT_EPI_I32) {
#pragma unroll
      for (int i = 0; i < (2 * BN + 255) / 256; ++i) {
        const int q = tid + 256 * i;
        if (q < 2 * BN) (q < BN ? sc_lds[sb] : bi_lds[sb])[q % BN] = rs[i];
      }
    }
  };

  int sb = 0;
  gload(tile, 0);
  lstore(0, 0);
  lds_barrier();
  for (;;) {
    const int ntile = tile + nbx;
    const bool has_next = ntile < end;
    v16i acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int i = 0; i < FM; ++i) acc[j][i] = v16i{};
#pragma unroll
    for (int c = 0; c < KCN; ++c) {
      if (c + 1 < KCN) gload(tile, c + 1);
      else gload(has_next ? ntile : tile, 0);
      // keeps the prefetch here: the compiler would otherwise sink the loads
      // to their use after the epilogue (the LDS-only barriers let it; the
      // operands are not declared restrict, so the loads cannot pass this)
      asm volatile("" ::: "memory");
#pragma unroll
      for (int kk = 0; kk < KC; kk += 32) {
        v4i a[FN], bx[FM];
#pragma unroll
        for (int j = 0; j < FN; ++j) a[j] = *(const v4i*)(&Ws[(BN / 2 * wn + 32 * j + l32) * ROW + kk + 16 * h]);
#pragma unroll
        for (int i = 0; i < FM; ++i) bx[i] = *(const v4i*)(&Xs[(BM / 2 * wm + 32 * i + l32) * ROW + kk + 16 * h]);
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int i = 0; i < FM; ++i)
            acc[j][i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[j], bx[i], acc[j][i], 0, 0, 0);
      }
      lds_barrier();  // every wave is done with the chunk in LDS
      if (c + 1 < KCN) {
        lstore(c + 1, sb);
        lds_barrier();
      }
    }
    {
      const int m0 = (tile % tiles_m) * BM, n0 = (tile / tiles_m) * BN;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int cb = BN / 2 * wn + 32 * j;  // fragment's first column within the tile
        float sc[4][4], bi[4][4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const v4f s4 = *(const v4f*)(&sc_lds[sb][cb + 8 * g + 4 * h]);
          const v4f b4 = *(const v4f*)(&bi_lds[sb][cb + 8 * g + 4 * h]);
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            sc[g][t] = EPI == MNMT_EPI_I32 ? 0.0f : s4[t];
            bi[g][t] = EPI == MNMT_EPI_I32 ? 0.0f : b4[t];
          }
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
          store_fragment<EPI, true>(e, acc[j][i], sc, bi, m0 + BM / 2 * wm + 32 * i + l32, n0 + cb, h, M, N);
      }
    }
    if (!has_next) break;
    sb ^= 1;  // the next tile's constants go to the other buffer
    lstore(0, sb);
    lds_barrier();
    tile = ntile;
  }
}

template <int BN, int BM, int WN, int WM, bool W4>
hipError_t launch_cfg(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                      int N, const EpiArgs& e, hipStream_t s, int splits = 1) {
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  const int grid = (tiles + kXcds - 1) / kXcds * kXcds;
#define MNMT_GEMM(EPI)                                                                                          \
  hipLaunchKernelGGL((k_gemm<BN, BM, WN, WM, EPI, W4>), dim3(grid, splits), dim3(256), 0, s, X, ldx, W, M, K, N, \
                     scale, bias, e, tiles_m, tiles, K / splits)
  switch (e.kind) {
    case MNMT_EPI_I32: MNMT_GEMM(MNMT_EPI_I32); break;
    case MNMT_EPI_I8: MNMT_GEMM(MNMT_EPI_I8); break;
    case MNMT_EPI_I8_RELU: MNMT_GEMM(MNMT_EPI_I8_RELU); break;
    case MNMT_EPI_F32: MNMT_GEMM(MNMT_EPI_F32); break;
    case MNMT_EPI_F32_RESID: MNMT_GEMM(MNMT_EPI_F32_RESID); break;
    case MNMT_EPI_LOGITS: MNMT_GEMM(MNMT_EPI_LOGITS); break;
    default: return hipErrorInvalidValue;
  }
#undef MNMT_GEMM
  return hipGetLastError();
}

template <int BN, int BM, int KC, int KCN, bool W4>
hipError_t launch_persistent(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M,
                             int K, int N, const EpiArgs& e, hipStream_t s) {
  const int tiles_m = M / BM, tiles = tiles_m * (N / BN);
  // two blocks per CU: 32 CUs per XCD
  const int nblk = min(kXcds * 64, (tiles + kXcds - 1) / kXcds * kXcds);
#define MNMT_GEMM(EPI)                                                                                    \
  hipLaunchKernelGGL((k_gemm_p<EPI, BN, BM, KC, KCN, W4>), dim3(nblk), dim3(256), 0, s, X, ldx, W, M, K, N, scale, \
                     bias, e, tiles_m, tiles, nblk)
  switch (e.kind) {
    case MNMT_EPI_I32: MNMT_GEMM(MNMT_EPI_I32); break;
    case MNMT_EPI_I8: MNMT_GEMM(MNMT_EPI_I8); break;
    case MNMT_EPI_I8_RELU: MNMT_GEMM(MNMT_EPI_I8_RELU); break;
    case MNMT_EPI_F32: MNMT_GEMM(MNMT_EPI_F32); break;
    case MNMT_EPI_F32_RESID: MNMT_GEMM(MNMT_EPI_F32_RESID); break;
    case MNMT_EPI_LOGITS: MNMT_GEMM(MNMT_EPI_LOGITS); break;
    default: return hipErrorInvalidValue;
  }
#undef MNMT_GEMM
  return hipGetLastError();
}

// Persistent configuration: 256 x 128 tiles (waves of 128 x 64, the fewest
// LDS reads per MFMA that fit two waves per SIMD), 128-byte K chunks.
constexpr int kPBN = 256, kPBM = 128, kPKC = 128;

// ---------------------------------------------------------------------------
// Weight-stationary kernel for K = 256 and long runs of rows (the 4096-row
// sweep shapes, large batched logits).  A 512-thread block owns 256 output
// columns: wave w keeps the int8 weights of its 64 columns (w mod 4) for the
// whole K in registers (16 KB per wave, 64 VGPRs), and its per-column
// constants too, and walks a range of 64-row steps of X.  Waves w and w + 4
// take rows 0-31 and 32-63 of each step, so all eight waves pass the same
// barriers and finish together (with two independent blocks per CU the
// hardware's preference for older waves let one block finish well before the
// other).  Each step's X rows (16 KB) go through LDS, double buffered; they
// are loaded into registers at the start of the previous step and stored to
// LDS at its end.  The LDS then feeds only the X operand: 0.5 KB of LDS
// reads per 32x32x32 MFMA instead of 0.75 KB with both operands staged.
//
// The epilogue of step t - 1 runs interleaved with the MFMAs of step t (two
// accumulator sets), so its VALU work overlaps the matrix cores.  For a
// uniform loop body the first step also runs an epilogue, of zeros, over its
// own rows, which the real epilogue rewrites one step later (same wave, same
// addresses, program order): every step then issues the same memory
// operations, and each wait for the X prefetch counts exactly the output
// stores issued after it (loads and stores share one in-order counter), so
// no wait covers stores of the current step.
constexpr int kWsK = 256, kWsRows = 64, kWsMinSteps = 16;

template <int EPI>
struct WsConst {
  float sc[2][16], bi[2][16];  // [fragment][4 g + t]: column 32 f + 8 g + 4 h + t of the wave
};

// Group G (4 outputs) of fragment F: int8 outputs are packed into w4[G] and
// written after group 3 (one 16-byte store of 16 consecutive columns per
// lane, after two lane swaps); wider outputs are written per group.
// Byte T of d = the low byte of (y + 1.5 * 2^23) for y already clamped to
// [-127, 127]: the add rounds y to an integer (round half to even) and leaves
// its two's complement code in the low byte (as code_bits), and the SDWA
// destination select writes that byte alone (byte 0 clears the others), so
// four codes are packed without byte permutes.
template <int T>
__device__ __forceinline__ void add_code_byte(uint32_t& d, float y) {
  const float magic = 12582912.0f;
  if (T == 0) asm("v_add_f32_sdwa %0, %1, %2 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:DWORD" : "=v"(d) : "v"(y), "v"(magic));
  if (T == 1) asm("v_add_f32_sdwa %0, %1, %2 dst_sel:BYTE_1 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:DWORD" : "+v"(d) : "v"(y), "v"(magic));
  if (T == 2) asm("v_add_f32_sdwa %0, %1, %2 dst_sel:BYTE_2 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:DWORD" : "+v"(d) : "v"(y), "v"(magic));
  if (T == 3) asm("v_add_f32_sdwa %0, %1, %2 dst_sel:BYTE_3 dst_unused:UNUSED_PRESERVE src0_sel:DWORD src1_sel:DWORD" : "+v"(d) : "v"(y), "v"(magic));
}

template <int EPI, int F, int G>
__device__ __forceinline__ void ws_epi_group(const EpiArgs& e, const v16i (&P)[2], const WsConst<EPI>& c,
                                             uint32_t (&w4)[4], int m, int nw, int h) {
  constexpr bool INT8_OUT = EPI == MNMT_EPI_I8 || EPI == MNMT_EPI_I8_RELU;
  if (INT8_OUT) {
    float y[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
      y[t] = fminf(fmaxf(epi_value<EPI>(P[F][4 * G + t], c.sc[F][4 * G + t], c.bi[F][4 * G + t]), -127.0f), 127.0f);
    add_code_byte<0>(w4[G], y[0]);
    add_code_byte<1>(w4[G], y[1]);
    add_code_byte<2>(w4[G], y[2]);
    add_code_byte<3>(w4[G], y[3]);
    if (G == 3) {
      const auto s02 = __builtin_amdgcn_permlane32_swap(w4[0], w4[2], false, false);
      const auto s13 = __builtin_amdgcn_permlane32_swap(w4[1], w4[3], false, false);
      int8_t* y = (int8_t*)e.out + (size_t)m * e.ldo + nw + 32 * F + 16 * h;
      *(v4i*)y = v4i{(int)s02[0], (int)s02[1], (int)s13[0], (int)s13[1]};
    }
  } else if (EPI == MNMT_EPI_I32) {
    int* y = (int*)e.out + (size_t)m * e.ldo + nw + 32 * F + 8 * G + 4 * h;
    *(v4i*)y = v4i{P[F][4 * G], P[F][4 * G + 1], P[F][4 * G + 2], P[F][4 * G + 3]};
  } else {
    static_assert(EPI != MNMT_EPI_F32_RESID, "the zero epilogue of the first step would overwrite the residual");
    float* y = (float*)e.out + (size_t)m * e.ldo + nw + 32 * F + 8 * G + 4 * h;
    v4f v;
#pragma unroll
    for (int t = 0; t < 4; ++t) v[t] = epi_value<EPI>(P[F][4 * G + t], c.sc[F][4 * G + t], c.bi[F][4 * G + t]);
    *(v4f*)y = v;
  }
}

// The 8 groups (2 fragments x 4) of the epilogue spread over the K steps:
// step KK takes groups [8 KK / NKK, 8 (KK + 1) / NKK).
template <int EPI, int KK, int NKK>
__device__ __forceinline__ void ws_epi_part(const EpiArgs& e, const v16i (&P)[2], const WsConst<EPI>& c,
                                            uint32_t (&w4)[4], int m, int nw, int h) {
#pragma unroll
  for (int q = 8 * KK / NKK; q < 8 * (KK + 1) / NKK; ++q) {
    if (q == 0) ws_epi_group<EPI, 0, 0>(e, P, c, w4, m, nw, h);
    if (q == 1) ws_epi_group<EPI, 0, 1>(e, P, c, w4, m, nw, h);
    if (q == 2) ws_epi_group<EPI, 0, 2>(e, P, c, w4, m, nw, h);
    if (q == 3) ws_epi_group<EPI, 0, 3>(e, P, c, w4, m, nw, h);
    if (q == 4) ws_epi_group<EPI, 1, 0>(e, P, c, w4, m, nw, h);
    if (q == 5) ws_epi_group<EPI, 1, 1>(e, P, c, w4, m, nw, h);
    if (q == 6) ws_epi_group<EPI, 1, 2>(e, P, c, w4, m, nw, h);
    if (q == 7) ws_epi_group<EPI, 1, 3>(e, P, c, w4, m, nw, h);
  }
}

// K step KK onward: two MFMAs into C (the wave's two 32-column fragments
// against one 32-row X fragment from LDS), then part KK of P's epilogue.
template <int EPI, int NKK, int KK = 0>
__device__ __forceinline__ void ws_steps(const int8_t* xs, const v4i (&wr)[2][NKK], v16i (&C)[2], const EpiArgs& e,
                                         const v16i (&P)[2], const WsConst<EPI>& c, uint32_t (&w4)[4], int m, int nw,
                                         int h) {
  if constexpr (KK < NKK) {
    const v4i bx = *(const v4i*)(xs + 32 * KK);
    C[0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wr[0][KK], bx, C[0], 0, 0, 0);
    C[1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wr[1][KK], bx, C[1], 0, 0, 0);
    ws_epi_part<EPI, KK, NKK>(e, P, c, w4, m, nw, h);
    ws_steps<EPI, NKK, KK + 1>(xs, wr, C, e, P, c, w4, m, nw, h);
  }
}

template <int EPI, int NKK, int KK = 0>
__device__ __forceinline__ void ws_epilogue(const EpiArgs& e, const v16i (&P)[2], const WsConst<EPI>& c,
                                            uint32_t (&w4)[4], int m, int nw, int h) {
  if constexpr (KK < NKK) {
    ws_epi_part<EPI, KK, NKK>(e, P, c, w4, m, nw, h);
    ws_epilogue<EPI, NKK, KK + 1>(e, P, c, w4, m, nw, h);
  }
}

template <int EPI>
__global__ __launch_bounds__(512, 1) void k_gemm_ws(const int8_t* X, int ldx, const int8_t* W, int M,
                                                    const float* scale, const float* bias, EpiArgs e, int ncol,
                                                    int steps_per_block) {
  constexpr int KB = kWsK, TM = kWsRows, NKK = KB / 32, XROW = KB + 16;  // padded LDS row
  constexpr int CPR = KB / 16, RPS = 512 / CPR, LX = TM / RPS;  // X loads: 16 bytes, rows per pass, passes
  static_assert(TM % RPS == 0 && LX >= 1, "whole X loads");
  __shared__ __attribute__((aligned(16))) int8_t Xs[2][TM * XROW];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5;
  const int cb = blockIdx.x % ncol, ms = blockIdx.x / ncol;
  const int nw = cb * 256 + 64 * (wave & 3);       // the wave's first column
  const int row = (lane & 31) + 32 * (wave >> 2);  // the lane's row within a step
  const int t0 = ms * steps_per_block, t1 = min(t0 + steps_per_block, M / TM);
  if (t0 >= t1) return;
  const int lrow = tid / CPR, lcol = 16 * (tid % CPR);  // this thread's X loads: rows lrow + RPS i

  v4i px[LX];
  auto xload = [&](int t) {
#pragma unroll
    for (int i = 0; i < LX; ++i) px[i] = *(const v4i*)(X + (size_t)(t * TM + lrow + RPS * i) * ldx + lcol);
  };
  auto xstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LX; ++i) *(v4i*)(&Xs[buf][(lrow + RPS * i) * XROW + lcol]) = px[i];
  };
  xload(t0);
  v4i wr[2][NKK];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      wr[f][kk] = *(const v4i*)(W + (size_t)(nw + 32 * f + (lane & 31)) * KB + 32 * kk + 16 * h);
  WsConst<EPI> c;
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = nw + 32 * f + 8 * g + 4 * h;
      const v4f s4 = EPI == MNMT_EPI_I32 ? v4f{} : *(const v4f*)(scale + n);
      const v4f b4 = (EPI == MNMT_EPI_I32 || EPI == MNMT_EPI_LOGITS) ? v4f{} : *(const v4f*)(bias + n);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        c.sc[f][4 * g + t] = s4[t];
        c.bi[f][4 * g + t] = b4[t];
      }
    }
  xstore(0);
  // the weights and constants arrive here, before the loop: a wait for them
  // inside it would be counted from the loop entry on every step
#pragma unroll
  for (int f = 0; f < 2; ++f) {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) asm volatile("" : "+v"(wr[f][kk]));
#pragma unroll
    for (int q = 0; q < 16; ++q) asm volatile("" : "+v"(c.sc[f][q]), "+v"(c.bi[f][q]));
  }
  lds_barrier();

  uint32_t w4[4];
  v16i A[2] = {v16i{}, v16i{}}, B[2] = {v16i{}, v16i{}};
  const int xoff = row * XROW + 16 * h;
  int t = t0, buf = 0;
  for (;;) {
    // step t into A, the epilogue of step t - 1 from B (zeros over step t0's
    // rows the first time)
    xload(min(t + 1, t1 - 1));
    asm volatile("" ::: "memory");  // keeps the prefetch ahead of the step
    A[0] = A[1] = v16i{};
    ws_steps<EPI, NKK>(&Xs[buf][xoff], wr, A, e, B, c, w4, max(t - 1, t0) * TM + row, nw, h);
    xstore(buf ^ 1);
    lds_barrier();
    if (t + 1 >= t1) {
      ws_epilogue<EPI, NKK>(e, A, c, w4, t * TM + row, nw, h);
      break;
    }
    ++t;
    buf ^= 1;
    // step t into B, the epilogue of step t - 1 from A
    xload(min(t + 1, t1 - 1));
    asm volatile("" ::: "memory");
    B[0] = B[1] = v16i{};
    ws_steps<EPI, NKK>(&Xs[buf][xoff], wr, B, e, A, c, w4, (t - 1) * TM + row, nw, h);
    xstore(buf ^ 1);
    lds_barrier();
    if (t + 1 >= t1) {
      ws_epilogue<EPI, NKK>(e, B, c, w4, t * TM + row, nw, h);
      break;
    }
    ++t;
    buf ^= 1;
  }
}

// Blocks for the weight-stationary kernel: one per CU, the column blocks
// times a split of the row steps.
struct WsPlan {
  int ncol, steps_per_block, nblk;
};
__host__ inline WsPlan ws_plan(int M, int N) {
  const int ncol = N / 256, steps = M / kWsRows;
  const int split = max(1, min(steps, 256 / max(1, ncol)));
  const int spb = (steps + split - 1) / split;
  return WsPlan{ncol, spb, ncol * ((steps + spb - 1) / spb)};
}

hipError_t launch_ws(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M,
                     const EpiArgs& e, const WsPlan& p, hipStream_t s) {
#define MNMT_GEMM(EPI)                                                                                          \
  hipLaunchKernelGGL((k_gemm_ws<EPI>), dim3(p.nblk), dim3(512), 0, s, X, ldx, W, M, scale, bias, e, p.ncol, \
                     p.steps_per_block)
  switch (e.kind) {
    case MNMT_EPI_I32: MNMT_GEMM(MNMT_EPI_I32); break;
    case MNMT_EPI_I8: MNMT_GEMM(MNMT_EPI_I8); break;
    case MNMT_EPI_I8_RELU: MNMT_GEMM(MNMT_EPI_I8_RELU); break;
    case MNMT_EPI_F32: MNMT_GEMM(MNMT_EPI_F32); break;
    case MNMT_EPI_LOGITS: MNMT_GEMM(MNMT_EPI_LOGITS); break;
    default: return hipErrorInvalidValue;
  }
#undef MNMT_GEMM
  return hipGetLastError();
}

template <bool W4>
hipError_t launch_tiled(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                        int N, const EpiArgs& e, hipStream_t s, bool aligned) {
  auto tiles = [&](int bn, int bm) { return (long)((N + bn - 1) / bn) * ((M + bm - 1) / bm); };
  if (aligned && M % kPBM == 0 && N % kPBN == 0 && tiles(kPBN, kPBM) >= kXcds * 64 && ldx % 16 == 0 &&
      (reinterpret_cast<uintptr_t>(X) & 15) == 0 && (reinterpret_cast<uintptr_t>(W) & 15) == 0 && K % kPKC == 0) {
    switch (K / kPKC) {
      case 1: return launch_persistent<kPBN, kPBM, kPKC, 1, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
      case 2: return launch_persistent<kPBN, kPBM, kPKC, 2, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
      case 4: return launch_persistent<kPBN, kPBM, kPKC, 4, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
      case 8: return launch_persistent<kPBN, kPBM, kPKC, 8, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
      case 16: return launch_persistent<kPBN, kPBM, kPKC, 16, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
      default: break;
    }
  }
  constexpr long kFill = 512;
  if (tiles(256, 128) >= kFill) return launch_cfg<256, 128, 2, 2, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (tiles(128, 128) >= kFill) return launch_cfg<128, 128, 2, 2, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  if (tiles(128, 64) >= kFill) return launch_cfg<128, 64, 2, 2, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
  return launch_cfg<64, 64, 2, 2, W4>(X, ldx, W, scale, bias, M, K, N, e, s);
}

}  // namespace

// The weight-stationary kernel for K = 256 and long row runs (int8 weights);
// the persistent kernel for whole tiles (16-byte aligned rows), K a
// power-of-two number of chunks and enough tiles for every block; otherwise
// the largest slab-pipelined tile that still gives about two blocks per CU
// (256 CUs).
hipError_t launch_gemm_split(const int8_t* X, int ldx, const int8_t* W, int M, int K, int N, int splits,
                             int32_t* part, hipStream_t s, bool w4) {
  if (M <= 0) return hipSuccess;
  if (splits < 1 || K % (splits * kBK)) return hipErrorInvalidValue;
  const EpiArgs e{MNMT_EPI_I32, part, N, 1.f, nullptr};
  return w4 ? launch_cfg<64, 64, 2, 2, true>(X, ldx, W, nullptr, nullptr, M, K, N, e, s, splits)
            : launch_cfg<64, 64, 2, 2, false>(X, ldx, W, nullptr, nullptr, M, K, N, e, s, splits);
}

hipError_t launch_gemm(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                       int N, const EpiArgs& e, hipStream_t s, bool w4) {
  if (M <= 0) return hipSuccess;
  if (K % kBK) return hipErrorInvalidValue;
  const bool int8_out = e.kind == MNMT_EPI_I8 || e.kind == MNMT_EPI_I8_RELU;
  const bool aligned = (reinterpret_cast<uintptr_t>(e.out) & 15) == 0 && e.ldo % (int8_out ? 16 : 4) == 0;
  const bool ops_aligned = ldx % 16 == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0 &&
                           (reinterpret_cast<uintptr_t>(W) & 15) == 0;
  if (!w4 && aligned && ops_aligned && K == kWsK && N % 256 == 0 && M % kWsRows == 0 &&
      e.kind != MNMT_EPI_F32_RESID) {
    const WsPlan p = ws_plan(M, N);
    if (p.steps_per_block >= kWsMinSteps) return launch_ws(X, ldx, W, scale, bias, M, e, p, s);
  }
  return w4 ? launch_tiled<true>(X, ldx, W, scale, bias, M, K, N, e, s, aligned)
            : launch_tiled<false>(X, ldx, W, scale, bias, M, K, N, e, s, aligned);
}

}  // namespace mnmt
