// encode_small.hip -- the encoder for at most 64 rows (a batch-1 source, or a
// few short ones) in 2 kernels per layer plus one for the output:
//   k_enc_attn (one block per head): [pending residual update + LayerNorm +
//       quantization of all rows] -> the head's Q, K, V rows on the matrix
//       cores -> attention within each sentence -> the head's context times
//       its columns of W_o, added to an int32 accumulator
//   k_enc_ffn (one block per 64 hidden units): [pending update + LayerNorm +
//       quantization] -> the chunk of W1 with the ReLU requantization -> the
//       chunk's columns of W2 into an int32 accumulator
//   k_enc_out (one block per 64 output columns of one decoder layer's cross
//       K|V projection): [pending update + final LayerNorm + quantization with
//       the encoder output scale] -> the cross keys and values
// As in the batch-1 decoder (decode_step.hip): integer partial sums are
// exact in any order, so the heads and FFN chunks add into shared int32
// accumulators, and the next kernel applies the residual epilogue
// x <- fma(gamma, x, fma(acc, scale, bias)) in its prologue.  Every block
// recomputes the LayerNorm of all rows (a few KB) instead of paying a kernel
// boundary; the blocks share the stores of the updated rows.  Two
// accumulators per kind alternate by layer; the blocks of the kernel after a
// buffer's consumer clear it.
//
// The blocks have 8 waves: the per-row work (LayerNorm, softmax) and the
// context sums are chains of dependent instructions, so more waves per block
// shorten the kernel even though the few blocks leave most CUs idle.
//
// Rows are r = b S + p (sentence b, position p < S, padded positions computed
// and never used); attention keys of row r are its sentence's positions below
// its length (Appendix A self-attention with the quantizer figure's
// precisions, the same canonical arithmetic as the other attention kernels).
#include "blocks.hpp"
#include "chain.hpp"
#include "internal.h"

namespace mnmt {
namespace {

constexpr int kEncRows = 64;                // rows of this path (B * S)
constexpr int kEncHeadDim = 64;             // widest head
constexpr int kEncChunk = 64;               // hidden units per k_enc_ffn block, columns per k_enc_out block
constexpr int kEncWaves = 8;                // waves per block
constexpr int kEncThreads = 64 * kEncWaves;
// LDS row strides of the int8 operands read as matrix-core fragments: 16
// bytes past the row, so that the rows of a fragment (16 rows, the same 16
// bytes of each) fall in different banks; at a stride of 256 (or 64) bytes
// every row of a 128-bit read maps to the same four banks.
template <int D>
constexpr int lds_ld() { return D + 16; }
constexpr int kHeadLd = kEncHeadDim + 16;   // q, k, context and hidden-unit rows
constexpr int kVtLd = kEncRows + 4;         // transposed values: 4-byte reads by 64 consecutive rows

// LayerNorm of G rows held by a wave (row q's element i = lane + 64 j in
// v[q][j]), each in the canonical order (as ln_row), interleaved.
template <int G, int NJ>
__device__ __forceinline__ void ln_rows(float (&v)[G][NJ], const float (&g)[NJ], const float (&b)[NJ], int d,
                                        float eps) {
  const int lane = threadIdx.x & 63;
  const float inv_d = 1.0f / (float)d;
  float p[G], mu[G], p2[G], rstd[G];
#pragma unroll
  for (int q = 0; q < G; ++q) {
    p[q] = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (lane + 64 * j < d) p[q] = p[q] + v[q][j];
  }
#pragma unroll
  for (int q = 0; q < G; ++q) mu[q] = wave_sum(p[q]) * inv_d;
#pragma unroll
  for (int q = 0; q < G; ++q) {
    p2[q] = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      if (lane + 64 * j < d) {
        v[q][j] = v[q][j] - mu[q];
        p2[q] = fmaf(v[q][j], v[q][j], p2[q]);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < G; ++q) rstd[q] = 1.0f / sqrtf(wave_sum(p2[q]) * inv_d + eps);
#pragma unroll
  for (int q = 0; q < G; ++q)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (lane + 64 * j < d) v[q][j] = fmaf(v[q][j] * rstd[q], g[j], b[j]);
}

// Clears this block's share of the accumulators whose consumers have
// finished (8-byte write-through stores; the counts are multiples of 64).
__device__ __forceinline__ void enc_clear(const EncIn& in) {
  const int b = blockIdx.x, nb = in.nblk;
  const int n0 = in.zero0_n / 4, n1 = in.zero1_n / 4;
  const int per0 = (n0 + nb - 1) / nb, per1 = (n1 + nb - 1) / nb;
  const int e0 = min(n0, (b + 1) * per0), e1 = min(n1, (b + 1) * per1);
  unsigned long long* z0 = reinterpret_cast<unsigned long long*>(in.zero0);
  unsigned long long* z1 = reinterpret_cast<unsigned long long*>(in.zero1);
  for (int i = b * per0 + threadIdx.x; i < e0; i += kEncThreads) {
    chain_store(z0 + 2 * i, 0ull);
    chain_store(z0 + 2 * i + 1, 0ull);
  }
  for (int i = b * per1 + threadIdx.x; i < e1; i += kEncThreads) {
    chain_store(z1 + 2 * i, 0ull);
    chain_store(z1 + 2 * i + 1, 0ull);
  }
}

// The sublayer input rows: the embedding or the pending residual update, the
// LayerNorm, the stores of the updated residual rows (x_out) and of the int8
// rows (q_out) (row r by block r mod nblk), and the int8 rows in a_lds (row
// stride lds_ld<D>()).  Wave w takes rows w + kEncWaves u, u < RPW, and issues all of
// their loads before it uses the first (one memory round trip, two for the
// embedding's token lookup), then calls issue_weights() to issue the
// kernel's other loads, then clears its share of the finished accumulators.
// D is the exact width, so no element needs a bounds check; EMBED is a
// template flag so that no load sits behind a run-time branch.
template <int D, bool EMBED, int RPW, class Issue>
__device__ __forceinline__ void enc_rows(const EncIn& in, int8_t* a_lds, Issue issue_weights) {
  constexpr int NJ = D / 64;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int R = in.R;
  // the kernel's own loads first (weights, scales, lengths: none written by
  // the previous kernel), then, in a kernel chain, the wait for it
  issue_weights();
  asm volatile("" ::: "memory");
  chain_wait(in.chain);
  float sc[NJ], bi[NJ], g[NJ], b[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = lane + 64 * j;
    sc[j] = in.scale[i];
    bi[j] = in.bias[i];
    g[j] = in.ln_g[i];
    b[j] = in.ln_b[i];
  }
  float x[RPW][NJ], a[RPW][NJ], ce[RPW];
  if (EMBED) {
    int tok[RPW];
#pragma unroll
    for (int u = 0; u < RPW; ++u) {
      const int t = in.tok[min(wave + kEncWaves * u, R - 1)];
      tok[u] = t < 0 ? 0 : (t >= in.V ? in.V - 1 : t);
    }
#pragma unroll
    for (int u = 0; u < RPW; ++u) {
      const int pos = min(wave + kEncWaves * u, R - 1) % in.S;
      ce[u] = in.c_emb[tok[u]];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int i = lane + 64 * j;
        x[u][j] = in.pe[pos * D + i];
        a[u][j] = (float)in.E[tok[u] * D + i];
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < RPW; ++u) {
      const int r = min(wave + kEncWaves * u, R - 1);
      ce[u] = 0.0f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int i = lane + 64 * j;
        x[u][j] = in.x_in[r * D + i];
        a[u][j] = (float)in.acc[r * D + i];
      }
    }
  }
  // every load of the kernel completes before its first store (the clears,
  // the rows): the memory counter retires in order, so a wait for one of
  // those loads placed after the stores would also wait for the stores to
  // reach the point of coherence
  __builtin_amdgcn_s_waitcnt(0);
  enc_clear(in);
  // up to four rows at a time, so that their dependent chains (butterflies,
  // square root, division) interleave
  constexpr int G = RPW < 4 ? RPW : 4;
#pragma unroll
  for (int u0 = 0; u0 < RPW; u0 += G) {
    if (wave + kEncWaves * u0 >= R) break;
    float v[G][NJ];
#pragma unroll
    for (int q = 0; q < G; ++q)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int u = u0 + q;
        if (EMBED)
          v[q][j] = fmaf(a[u][j], ce[u], x[u][j]);
        else if (in.update)
          v[q][j] = fmaf(in.gamma, x[u][j], fmaf(a[u][j], sc[j], bi[j]));
        else
          v[q][j] = x[u][j];
      }
    if (in.ln_mode == 1) ln_rows<G, NJ>(v, g, b, D, in.eps);  // post-LN: normalize the residual stream
    if (in.x_out) {
#pragma unroll
      for (int q = 0; q < G; ++q) {
        const int r = wave + kEncWaves * (u0 + q);
        if (r < R && r % in.nblk == (int)blockIdx.x)
#pragma unroll
          for (int j = 0; j < NJ; ++j) chain_store(in.x_out + r * D + lane + 64 * j, v[q][j]);
      }
    }
    if (in.ln_mode == 2) ln_rows<G, NJ>(v, g, b, D, in.eps);  // pre-LN: normalize the sublayer input
#pragma unroll
    for (int q = 0; q < G; ++q) {
      const int r = wave + kEncWaves * (u0 + q);
      if (r < R) {
        const bool qst = in.q_out && r % in.nblk == (int)blockIdx.x;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int8_t c = code_of(v[q][j] * in.inv_s);
          a_lds[r * lds_ld<D>() + lane + 64 * j] = c;
          if (qst) chain_store(in.q_out + r * D + lane + 64 * j, c);
        }
      }
    }
  }
}

// A fragment of int8 rows [rows, K] in LDS (row stride ld): rows m0 + l % 16,
// K bytes k0 + 16 (l / 16) .. + 15, zero past K.
__device__ __forceinline__ v4i lds_frag(const int8_t* base, int ld, int m0, int k0, int K) {
  const int lane = threadIdx.x & 63;
  const int k = k0 + 16 * (lane >> 4);
  return k < K ? *(const v4i*)(base + (m0 + (lane & 15)) * ld + k) : v4i{0, 0, 0, 0};
}

// int32 fragment D (rows m0 + 4 (l / 16) + i, column n) added to out[R, ld].
__device__ __forceinline__ void add_frag(int32_t* out, int ld, const v4i& acc, int m0, int n, int R) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + 4 * (lane >> 4) + i;
    if (m < R) atomicAdd(out + (size_t)m * ld + n, acc[i]);
  }
}

// One block per head.
template <int DMAX, bool EMBED, int RPW, bool W4>
__global__ __launch_bounds__(kEncThreads) void k_enc_attn(EncIn in, EncAttn at) {
  constexpr int KS = DMAX / 64;                                   // 64-deep K steps over d
  constexpr int NT = 3 * kEncHeadDim / 16;                        // projection tiles of the widest head
  constexpr int PT = (NT + kEncWaves - 1) / kEncWaves;            // projection tiles per wave
  constexpr int OT = (DMAX / 16 + kEncWaves - 1) / kEncWaves;     // W_o column tiles per wave
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kEncRows * lds_ld<DMAX>()];
  __shared__ __attribute__((aligned(16))) int8_t qk[2][kEncRows][kHeadLd];
  __shared__ __attribute__((aligned(16))) int8_t vt[kEncHeadDim][kVtLd];  // values, transposed
  __shared__ __attribute__((aligned(16))) int8_t ctx[kEncRows][kHeadLd];
  __shared__ __attribute__((aligned(16))) float sc[kEncRows][kEncRows];      // scores, then probabilities
  const int qs_n = at.qsplit, hd = blockIdx.x / qs_n, qs = blockIdx.x % qs_n;
  const int R = in.R, d = DMAX, dh = at.dh, S = in.S, ks = KS;
  const int mt_n = (R + 15) / 16;
  // this block's query rows: the 16-row tiles qs, qs + qs_n, ... (keys and
  // values of every row); row u of wave w is qrow(w + kEncWaves u)
  const int q_rows = 16 * ((mt_n - qs + qs_n - 1) / qs_n);  // rows of its tiles (the last may be partial)
  auto qrow = [&](int k) { return 16 * (qs + qs_n * (k / 16)) + (k % 16); };
  const int ntile = 3 * dh / 16;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, kq = lane >> 4;
  // 1. the rows, and behind their loads the weights (the head's Q|K|V rows
  //    and its W_o columns, with the projection's scale and bias per lane) and
  //    the lengths of the sentences of the wave's softmax rows
  WFrag<W4> wf[PT][KS];
  float e_sc[PT], e_bi[PT];
  WFrag<W4> of[OT];
  int nn[RPW];
  enc_rows<DMAX, EMBED, RPW>(in, a_lds, [&]() {
#pragma unroll
    for (int u = 0; u < PT; ++u) {
      const int j = 16 * min(wave + kEncWaves * u, ntile - 1) + l16;  // row of the head's [q | k | v]
      const int part = (j >= dh) + (j >= 2 * dh);
      const int n = part * d + hd * dh + (j - part * dh);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) wf[u][kk] = load_wfrag<W4>(at.W, n, d, 64 * kk + 16 * kq);
      e_sc[u] = at.scale[n];
      e_bi[u] = at.bias[n];
    }
#pragma unroll
    for (int u = 0; u < OT; ++u) {
      const int n = min(16 * (wave + kEncWaves * u) + l16, d - 1);
      of[u] = load_wfrag<W4>(at.Wo, n, d, hd * dh + 16 * min(kq, dh / 16 - 1));
    }
#pragma unroll
    for (int u = 0; u < RPW; ++u) nn[u] = at.len[min(qrow(min(wave + kEncWaves * u, q_rows - 1)), R - 1) / S];
  });
  lds_barrier();
  // 2. Q, K, V of the head, requantized into LDS (V transposed)
#pragma unroll
  for (int u = 0; u < PT; ++u) {
    const int tile = wave + kEncWaves * u;
    if (tile >= ntile) continue;
    const int j = 16 * tile + l16;
    const int part = (j >= dh) + (j >= 2 * dh);
    const int c = j - part * dh;
    v4i w[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) w[kk] = wf[u][kk].get();
    for (int mt = 0; mt < mt_n; ++mt) {
      if (part == 0 && mt % qs_n != qs) continue;  // queries of this block's rows only
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        if (kk < ks) acc = mfma16(lds_frag(a_lds, lds_ld<DMAX>(), 16 * mt, 64 * kk, d), w[kk], acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 16 * mt + 4 * kq + i;
        if (m < R) {
          const int8_t code = code_of(fmaf((float)acc[i], e_sc[u], e_bi[u]));
          if (part == 2) vt[c][m] = code;
          else qk[part][m][c] = code;
        }
      }
    }
  }
  lds_barrier();
  // 3. scores q . k (int32 exact) scaled by c_qk, every (query, key) pair
  const int qt_n = q_rows / 16;  // this block's query tiles
  for (int t = wave; t < qt_n * mt_n; t += kEncWaves) {
    const int mt = qs + qs_n * (t / mt_n), kt = t % mt_n;
    const v4i acc = mfma16(lds_frag(&qk[0][0][0], kHeadLd, 16 * mt, 0, dh),
                           lds_frag(&qk[1][0][0], kHeadLd, 16 * kt, 0, dh), v4i{0, 0, 0, 0});
#pragma unroll
    for (int i = 0; i < 4; ++i) sc[16 * mt + 4 * kq + i][16 * kt + l16] = (float)acc[i] * at.c_qk;
  }
  lds_barrier();
  // 4. softmax of each row over its sentence's keys (one key per lane: the
  //    canonical order), probabilities in place at sc[m][0 .. n); keys from
  //    n up to S rounded up to 4 get probability 0: fma(0, v, acc) leaves acc
  //    unchanged bit for bit, so the context loop may run over them
  {
    // rows of this wave: u < nu (the same count for every lane of the wave)
    const int nu = (q_rows - wave + kEncWaves - 1) / kEncWaves;
    float sv[RPW], ex[RPW];
#pragma unroll
    for (int u = 0; u < RPW; ++u) {
      const int m = min(qrow(min(wave + kEncWaves * u, q_rows - 1)), R - 1);
      const int b = m / S;
      nn[u] = nn[u] < 1 ? 1 : (nn[u] > S ? S : nn[u]);
      sv[u] = lane < nn[u] ? sc[m][b * S + lane] : -FLT_MAX;
    }
    float mx[RPW], inv[RPW];
#pragma unroll
    for (int u = 0; u < RPW; ++u) mx[u] = u < nu ? wave_max(sv[u]) : 0.0f;
#pragma unroll
    for (int u = 0; u < RPW; ++u) ex[u] = u < nu && lane < nn[u] ? canon_exp(sv[u] - mx[u]) : 0.0f;
#pragma unroll
    for (int u = 0; u < RPW; ++u) inv[u] = u < nu ? 1.0f / wave_sum(ex[u]) : 0.0f;
    wave_sync();  // every lane has read its scores before any probability is written
    const int s4 = (S + 3) & ~3;
#pragma unroll
    for (int u = 0; u < RPW; ++u) {
      const int k = wave + kEncWaves * u, m = qrow(k);
      if (k < q_rows && m < R && lane < s4) sc[m][lane] = lane < nn[u] ? ex[u] * inv[u] : 0.0f;
    }
  }
  lds_barrier();
  // 5. context: ascending keys, one fma each, requantized
  {
    // thread: column j = tid % dh of the block's rows qrow(g0 + groups u)
    // (g0 = tid / dh), one fma chain per row over the keys of its sentence in
    // ascending order.  With one sentence the rows share each load of four
    // values and read four probabilities at once; rows past R repeat row
    // R - 1, unstored.
    constexpr int CPT = RPW;  // rows per thread at most (kEncThreads / dh >= kEncWaves groups)
    const int groups = kEncThreads / dh;
    const int j = threadIdx.x % dh, g0 = threadIdx.x / dh;
    if (S == R) {  // one sentence
      // rows of this thread: u < cu (as many as CPT at the widest)
      const int cu = (q_rows - g0 + groups - 1) / groups;
      float acc[CPT];
#pragma unroll
      for (int u = 0; u < CPT; ++u) acc[u] = 0.0f;
      for (int t = 0; t < S; t += 4) {
        const int v4 = *(const int*)&vt[j][t];
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (float)(int)(int8_t)(v4 >> (8 * e));
#pragma unroll
        for (int u = 0; u < CPT; ++u) {
          if (u >= cu) break;
          const float4 p = *(const float4*)&sc[min(qrow(min(g0 + groups * u, q_rows - 1)), R - 1)][t];
          acc[u] = fmaf(p.x, v[0], acc[u]);
          acc[u] = fmaf(p.y, v[1], acc[u]);
          acc[u] = fmaf(p.z, v[2], acc[u]);
          acc[u] = fmaf(p.w, v[3], acc[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int k = g0 + groups * u, m = qrow(k);
        if (k < q_rows && m < R) ctx[m][j] = code_of(acc[u] * at.c_pv);
      }
    } else {
      for (int k = g0; k < q_rows; k += groups) {
        const int m = qrow(k);
        if (m >= R) break;  // rows ascend with k
        const int base = (m / S) * S;
        float acc = 0.0f;
        for (int t = 0; t < S; ++t) acc = fmaf(sc[m][t], (float)vt[j][base + t], acc);
        ctx[m][j] = code_of(acc * at.c_pv);
      }
    }
  }
  lds_barrier();
  // 6. the head's share of the output projection (K = dh), exact int32 sums
#pragma unroll
  for (int u = 0; u < OT; ++u) {
    const int n0 = 16 * (wave + kEncWaves * u);
    if (n0 >= d) continue;
    const v4i wo = of[u].get();
    for (int mt = qs; mt < mt_n; mt += qs_n) {
      const v4i acc = mfma16(lds_frag(&ctx[0][0], kHeadLd, 16 * mt, 0, dh), wo, v4i{0, 0, 0, 0});
      add_frag(at.acc_out, d, acc, 16 * mt, n0 + l16, R);
    }
  }
  chain_signal(in.chain);
}

// One block per kEncChunk hidden units: wave w computes the 16-unit W1 tile
// w % 4 for the 16-row tiles w / 4, w / 4 + 2, ...
template <int DMAX, int RPW, bool W4>
__global__ __launch_bounds__(kEncThreads) void k_enc_ffn(EncIn in, EncFfn f) {
  constexpr int KS = DMAX / 64;
  constexpr int OT = (DMAX / 16 + kEncWaves - 1) / kEncWaves;  // W2 column tiles per wave
  static_assert(kEncChunk == 64 && kEncWaves == 8, "four W1 tiles, two row-tile phases, one K step of W2");
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kEncRows * lds_ld<DMAX>()];
  __shared__ __attribute__((aligned(16))) int8_t hb[kEncRows][kHeadLd];
  const int R = in.R, d = DMAX, F = f.F, ks = KS;
  const int mt_n = (R + 15) / 16;
  const int f0 = blockIdx.x * kEncChunk;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, kq = lane >> 4;
  const int ht = wave & 3, mt0 = wave >> 2;
  const int hrow = f0 + 16 * ht + l16;  // < F (F is a multiple of kEncChunk)
  WFrag<W4> wf[KS];
  float e_sc, e_bi;
  WFrag<W4> of[OT];
  enc_rows<DMAX, false, RPW>(in, a_lds, [&]() {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) wf[kk] = load_wfrag<W4>(f.W1, hrow, d, 64 * kk + 16 * kq);
    e_sc = f.scale1[hrow];
    e_bi = f.bias1[hrow];
#pragma unroll
    for (int u = 0; u < OT; ++u) {
      const int n = min(16 * (wave + kEncWaves * u) + l16, d - 1);
      of[u] = load_wfrag<W4>(f.W2, n, F, f0 + 16 * kq);
    }
  });
  lds_barrier();
  v4i w1[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) w1[kk] = wf[kk].get();
  for (int mt = mt0; mt < mt_n; mt += 2) {
    v4i acc = {0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      if (kk < ks) acc = mfma16(lds_frag(a_lds, lds_ld<DMAX>(), 16 * mt, 64 * kk, d), w1[kk], acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 16 * mt + 4 * kq + i;
      if (m < R) hb[m][16 * ht + l16] = code_of(fmaxf(fmaf((float)acc[i], e_sc, e_bi), 0.0f));
    }
  }
  lds_barrier();
#pragma unroll
  for (int u = 0; u < OT; ++u) {
    const int n0 = 16 * (wave + kEncWaves * u);
    if (n0 >= d) continue;
    const v4i w2 = of[u].get();
    for (int mt = 0; mt < mt_n; ++mt) {
      const v4i acc = mfma16(lds_frag(&hb[0][0], kHeadLd, 16 * mt, 0, kEncChunk), w2, v4i{0, 0, 0, 0});
      add_frag(f.acc_out, d, acc, 16 * mt, n0 + l16, R);
    }
  }
  chain_signal(in.chain);
}

// One block per kEncChunk columns of one decoder layer's cross K|V
// projection: wave w computes the 16-column tile w % 4 for the 16-row tiles
// w / 4, w / 4 + 2, ...
template <int DMAX, int RPW, bool W4>
__global__ __launch_bounds__(kEncThreads) void k_enc_out(EncIn in, EncOut o) {
  constexpr int KS = DMAX / 64;
  static_assert(kEncChunk == 64 && kEncWaves == 8, "four column tiles, two row-tile phases");
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kEncRows * lds_ld<DMAX>()];
  const int R = in.R, d = DMAX, ks = KS;
  const int mt_n = (R + 15) / 16;
  const int per_layer = 2 * d / kEncChunk;
  const int layer = blockIdx.x / per_layer;
  const int c0 = (blockIdx.x - layer * per_layer) * kEncChunk;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, kq = lane >> 4;
  const EncOut::Layer& L = o.layer[layer];
  const int col = c0 + 16 * (wave & 3) + l16;  // < 2 d
  const int mt0 = wave >> 2;
  WFrag<W4> wf[KS];
  float e_sc, e_bi;
  enc_rows<DMAX, false, RPW>(in, a_lds, [&]() {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) wf[kk] = load_wfrag<W4>(L.W, col, d, 64 * kk + 16 * kq);
    e_sc = L.scale[col];
    e_bi = L.bias[col];
  });
  lds_barrier();
  v4i w[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) w[kk] = wf[kk].get();
  for (int mt = mt0; mt < mt_n; mt += 2) {
    v4i acc = {0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      if (kk < ks) acc = mfma16(lds_frag(a_lds, lds_ld<DMAX>(), 16 * mt, 64 * kk, d), w[kk], acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 16 * mt + 4 * kq + i;
      if (m < R) L.out[(size_t)m * 2 * d + col] = code_of(fmaf((float)acc[i], e_sc, e_bi));
    }
  }
  chain_signal(in.chain);
}

}  // namespace

bool enc_small_fits(int R, int S, int d, int dh, int F) {
  // (512 only up to 32 rows: with 8 rows per wave its attention kernel spills)
  const bool width = d == 64 || d == 128 || d == 192 || d == 256 || d == 384 || (d == 512 && R <= 32);
  return R >= 1 && R <= kEncRows && S <= kEncRows && width && dh % 16 == 0 && dh <= kEncHeadDim &&
         F % kEncChunk == 0;
}

// exact width x rows per wave (4 for up to 32 rows, else 8)
#define MNMT_ENC_BY_D(d, R, CALL)                        \
  switch ((d) * ((R) <= 32 ? 1 : -1)) {                 \
    case 64: CALL(64, 4); break;                         \
    case 128: CALL(128, 4); break;                       \
    case 192: CALL(192, 4); break;                       \
    case 256: CALL(256, 4); break;                       \
    case 384: CALL(384, 4); break;                       \
    case 512: CALL(512, 4); break;                       \
    case -64: CALL(64, 8); break;                        \
    case -128: CALL(128, 8); break;                      \
    case -192: CALL(192, 8); break;                      \
    case -256: CALL(256, 8); break;                      \
    case -384: CALL(384, 8); break;                      \
    default: return hipErrorInvalidValue;                \
  }

int enc_attn_qsplit(int R) { return R > 16 ? 2 : 1; }

hipError_t launch_enc_attn(const EncIn& in0, const EncAttn& at0, int heads, hipStream_t s) {
  if (!at0.W || !at0.Wo) return hipErrorInvalidValue;
  EncIn in = in0;
  EncAttn at = at0;
  at.qsplit = enc_attn_qsplit(in.R);
  const int blocks = heads * at.qsplit;
  in.nblk = blocks;
#define MNMT_EW(DM, RPW, W4)                                                                         \
  if (in.embed)                                                                                      \
    hipLaunchKernelGGL((k_enc_attn<DM, true, RPW, W4>), dim3(blocks), dim3(kEncThreads), 0, s, in, at); \
  else                                                                                                \
    hipLaunchKernelGGL((k_enc_attn<DM, false, RPW, W4>), dim3(blocks), dim3(kEncThreads), 0, s, in, at);
#define MNMT_E(DM, RPW)   \
  if (at.w4) {            \
    MNMT_EW(DM, RPW, true)  \
  } else {                \
    MNMT_EW(DM, RPW, false) \
  }
  MNMT_ENC_BY_D(in.d, in.R, MNMT_E)
#undef MNMT_E
#undef MNMT_EW
  return hipGetLastError();
}

hipError_t launch_enc_ffn(const EncIn& in0, const EncFfn& f, hipStream_t s) {
  if (!f.W1 || !f.W2) return hipErrorInvalidValue;
  const int blocks = f.F / kEncChunk;
  EncIn in = in0;
  in.nblk = blocks;
#define MNMT_E(DM, RPW)                                                                                    \
  if (f.w4) hipLaunchKernelGGL((k_enc_ffn<DM, RPW, true>), dim3(blocks), dim3(kEncThreads), 0, s, in, f);    \
  else hipLaunchKernelGGL((k_enc_ffn<DM, RPW, false>), dim3(blocks), dim3(kEncThreads), 0, s, in, f);
  MNMT_ENC_BY_D(in.d, in.R, MNMT_E)
#undef MNMT_E
  return hipGetLastError();
}

hipError_t launch_enc_out(const EncIn& in0, const EncOut& o, hipStream_t s) {
  if (o.layers < 1 || o.layers > EncOut::kMaxLayers) return hipErrorInvalidValue;
  for (int l = 0; l < o.layers; ++l)
    if (!o.layer[l].W) return hipErrorInvalidValue;
  const int blocks = o.layers * (2 * in0.d / kEncChunk);
  EncIn in = in0;
  in.nblk = blocks;
#define MNMT_E(DM, RPW)                                                                                    \
  if (o.w4) hipLaunchKernelGGL((k_enc_out<DM, RPW, true>), dim3(blocks), dim3(kEncThreads), 0, s, in, o);    \
  else hipLaunchKernelGGL((k_enc_out<DM, RPW, false>), dim3(blocks), dim3(kEncThreads), 0, s, in, o);
  MNMT_ENC_BY_D(in.d, in.R, MNMT_E)
#undef MNMT_E
  return hipGetLastError();
}

}  // namespace mnmt
