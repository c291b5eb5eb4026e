// decode_fused.hip -- decoder-step kernels for up to 8 rows (the batch-1
// latency path) with the element-wise work fused into the GEMVs (Section 4.2:
// everything between two GEMMs is one fused operation):
//   k_qgemv_ln : [embedding of the step's tokens |] LayerNorm | quantization
//                of the input rows, then a slice of a linear layer with a
//                requantizing (optionally ReLU) epilogue, or the tied output
//                projection with the arg-max fused.  Each block issues its
//                weight loads first and normalizes the (at most 8) input rows
//                while those loads are in flight; the rows are recomputed per
//                block, which costs less than a kernel boundary.
//   k_greedy_commit_slots : reduces the arg-max slots, records the tokens,
//                applies the end-of-sentence rule and advances the step.
// The arg-max of a row is spread over kSlots slots (block b updates slot
// b % kSlots) so that blocks do not serialize on one address; the commit
// kernel (the next launch) sees every update and clears the slots.
#include "blocks.hpp"
#include "internal.h"

namespace mnmt {
namespace {

constexpr int kRows = 8;    // rows per fused step (greedy batch <= 8)
constexpr int kSlots = 32;  // arg-max slots per row

// MR rows of input, rows of width K <= DMAX (LPR lanes per weight row, at
// most two 16-byte K chunks per lane), U row groups per wave; W4: gv.W holds
// packed 4-bit rows, widened in registers.
template <int MR, int DMAX, int U, bool W4>
__global__ __launch_bounds__(256) void k_qgemv_ln(FusedIn in, FusedGemv gv) {
  constexpr int LPR = lanes_per_row(DMAX);
  constexpr int RPI = 64 / LPR;
  __shared__ __attribute__((aligned(16))) int8_t a_lds[MR * DMAX];
  __shared__ unsigned long long wmax[4][MR];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPR, kl = lane % LPR;
  const int R = gv.R, K = gv.K, N = gv.N;
  const int row0 = (blockIdx.x * 4 + wave) * RPI * U;
  // 1. weight loads first
  WFrag<W4> wv[2][U];
#pragma unroll
  for (int ki = 0; ki < 2; ++ki) {
    const int k = kl * 16 + ki * LPR * 16;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int n = row0 + u * RPI + sub;
      wv[ki][u] = load_wfrag_if<W4>(k < K && n < N, gv.W, n, K, k);
    }
  }
  // 2. input rows while the loads are in flight
  // (at most 8 rows: two per wave, no wave loading rows past R)
  prepare_rows<(DMAX + 63) / 64, kRows / 4>(in, R, 0, K, gv.t, a_lds, K, blockIdx.x == 0);
  __syncthreads();
  // 3. dot products
  int acc[U][MR];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[u][m] = 0;
#pragma unroll
  for (int ki = 0; ki < 2; ++ki) {
    const int k = kl * 16 + ki * LPR * 16;
    if (k < K) {
#pragma unroll
      for (int m = 0; m < MR; ++m) {
        if (m < R) {
          const int4 xv = *(const int4*)(a_lds + m * K + k);
#pragma unroll
          for (int u = 0; u < U; ++u) acc[u][m] = dot16(wv[ki][u].get(), xv, acc[u][m]);
        }
      }
    }
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MR; ++m) acc[u][m] += __shfl_xor(acc[u][m], off, 64);
  if (gv.epi != EPI_LOGITS_ARGMAX) {
    if (kl != 0) return;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int n = row0 + u * RPI + sub;
      if (n >= N) continue;
#pragma unroll
      for (int m = 0; m < MR; ++m) {
        if (m < R) {
          float y = fmaf((float)acc[u][m], gv.scale[n], gv.bias[n]);
          if (gv.epi == MNMT_EPI_I8_RELU) y = fmaxf(y, 0.0f);
          ((int8_t*)gv.out)[(size_t)m * N + n] = code_of(y);
        }
      }
    }
    return;
  }
  // logits z = acc * scale[n] and the row's arg-max
#pragma unroll
  for (int m = 0; m < MR; ++m) {
    unsigned long long best = 0ull;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int n = row0 + u * RPI + sub;
      if (kl == 0 && n < N && m < R) {
        const float z = (float)acc[u][m] * gv.scale[n];
        if (gv.out) ((float*)gv.out)[(size_t)m * N + n] = z;
        const unsigned long long key = pack_argmax(z, n);
        best = key > best ? key : best;
      }
    }
    best = wave_max_u64(best);
    if (lane == 0) wmax[wave][m] = best;
  }
  __syncthreads();
  if (threadIdx.x < R) {
    const int m = threadIdx.x;
    unsigned long long b = wmax[0][m];
#pragma unroll
    for (int w = 1; w < 4; ++w) b = wmax[w][m] > b ? wmax[w][m] : b;
    if (b != 0ull) atomicMax(gv.slots + (size_t)m * gv.nslots + blockIdx.x % kSlots, b);
  }
}

__global__ __launch_bounds__(256) void k_greedy_commit_slots(FusedGemv gv) {
  __shared__ int next_tok[kRows];
  __shared__ unsigned long long wbest[4];
  const int t = gv.t, ns = gv.nslots;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int m = 0; m < gv.R; ++m) {
    // every thread reduces a stride of the row's slots and clears them
    unsigned long long b = 0ull;
    for (int i = threadIdx.x; i < ns; i += 256) {
      const unsigned long long v = gv.slots[(size_t)m * ns + i];
      b = v > b ? v : b;
    }
    for (int i = threadIdx.x; i < ns; i += 256) gv.slots[(size_t)m * ns + i] = 0ull;
    b = wave_max_u64(b);
    if (lane == 0) wbest[wave] = b;
    __syncthreads();
    if (threadIdx.x == 0) {
      b = wbest[0];
      for (int w = 1; w < 4; ++w) b = wbest[w] > b ? wbest[w] : b;
      if (gv.tagged) b = untag_key(b);  // tagged partials of a kernel chain (one step, one tag)
      const int tok = unpack_index(b);
      const int fin = gv.finished[m];
      if (t < gv.T) gv.out_tok[(size_t)t * gv.R + m] = fin ? gv.pad : tok;
      if (t < gv.T && gv.out_key) gv.out_key[(size_t)t * gv.R + m] = b;
      if (!fin && gv.stop_at_eos && tok == gv.eos) {
        gv.finished[m] = 1;
        gv.out_len[m] = t + 1;
      }
      gv.cur_tok[m] = fin ? gv.pad : tok;
      next_tok[m] = fin ? gv.pad : tok;
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; gv.zero_acc && i < gv.zero_n; i += blockDim.x) gv.zero_acc[i] = 0;
  if (threadIdx.x == 0) *gv.step = t + 1;
  // the next step's input rows: embedding of the new tokens at position t + 1
  if (gv.emb_out && t + 1 < gv.P) {
    const int d = gv.d;
    for (int e = threadIdx.x; e < gv.R * d; e += blockDim.x) {
      const int m = e / d, i = e % d;
      int tok = next_tok[m];
      tok = tok < 0 ? 0 : (tok >= gv.V ? gv.V - 1 : tok);
      gv.emb_out[e] = fmaf((float)gv.E[(size_t)tok * d + i], gv.c_emb[tok], gv.pe[(size_t)(t + 1) * d + i]);
    }
  }
}

// Row groups per wave: large layers (the output projection) get 8 so that
// one round of about one block per CU has the whole matrix in flight; small
// layers (and every packed 4-bit layer) get 1 for the most blocks.
template <int MR, int DMAX>
hipError_t launch_u(const FusedIn& in, const FusedGemv& gv, hipStream_t s) {
  constexpr int RPI = 64 / lanes_per_row(DMAX);
  const long blocks8 = ((long)gv.N + RPI * 32 - 1) / (RPI * 32);
  const long blocks1 = ((long)gv.N + RPI * 4 - 1) / (RPI * 4);
  if (gv.w4)
    hipLaunchKernelGGL((k_qgemv_ln<MR, DMAX, 1, true>), dim3((int)blocks1), dim3(256), 0, s, in, gv);
  else if (blocks8 >= 128)
    hipLaunchKernelGGL((k_qgemv_ln<MR, DMAX, 8, false>), dim3((int)blocks8), dim3(256), 0, s, in, gv);
  else
    hipLaunchKernelGGL((k_qgemv_ln<MR, DMAX, 1, false>), dim3((int)blocks1), dim3(256), 0, s, in, gv);
  return hipGetLastError();
}

template <int MR>
hipError_t launch_d(const FusedIn& in, const FusedGemv& gv, hipStream_t s) {
  switch (row_class(gv.K)) {
    case 64: return launch_u<MR, 64>(in, gv, s);
    case 128: return launch_u<MR, 128>(in, gv, s);
    case 256: return launch_u<MR, 256>(in, gv, s);
    case 384: return launch_u<MR, 384>(in, gv, s);
    case 512: return launch_u<MR, 512>(in, gv, s);
    default: return launch_u<MR, 1024>(in, gv, s);
  }
}

}  // namespace

int fused_slots_per_row(int V) { return max(kSlots, step_logits_blocks(V)); }

hipError_t launch_qgemv_ln(const FusedIn& in, const FusedGemv& gv, hipStream_t s) {
  // K chunks per lane must be at most two: K <= 32 * LPR with LPR <= 64
  if (gv.R < 1 || gv.R > kRows || gv.K > kMaxRowLen || gv.K % 16 || (gv.w4 && gv.epi == EPI_LOGITS_ARGMAX))
    return hipErrorInvalidValue;
  if (gv.R == 1) return launch_d<1>(in, gv, s);
  if (gv.R == 2) return launch_d<2>(in, gv, s);
  if (gv.R <= 4) return launch_d<4>(in, gv, s);
  return launch_d<8>(in, gv, s);
}

hipError_t launch_greedy_commit_slots(const FusedGemv& gv, hipStream_t s) {
  if (gv.R > kRows || gv.nslots < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_greedy_commit_slots, dim3(1), dim3(256), 0, s, gv);
  return hipGetLastError();
}

}  // namespace mnmt
