// kernels.hip -- embedding, LayerNorm + quantization, int8 attention with an
// int8 key/value cache, and the greedy / beam search bookkeeping.
// All fp32 arithmetic follows the canonical order of canon.hpp.
#include <cfloat>
#include <climits>

#include "blocks.hpp"
#include "internal.h"

namespace mnmt {
namespace {

// ---------------------------------------------------------------------------
// Embedding: x = fma(E[tok], c_emb[tok], PE[pos]).  One wave per row.
__global__ __launch_bounds__(256) void k_embed(const int32_t* __restrict__ tok, int rows, int S, const int* step,
                                               const int8_t* __restrict__ E, const float* __restrict__ c_emb,
                                               const float* __restrict__ pe, int d, int V, float* __restrict__ x) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  int t = tok[r];
  t = t < 0 ? 0 : (t >= V ? V - 1 : t);  // ids outside the vocabulary are clamped (memory safety)
  const int pos = step ? *step : r % S;
  const float c = c_emb[t];
  for (int i = lane; i < d; i += 64)
    x[(size_t)r * d + i] = fmaf((float)E[(size_t)t * d + i], c, pe[(size_t)pos * d + i]);
}

// Factorized embedding rows (one block per row): the token's Ef codes in LDS,
// thread n computes the exact int32 dot product with row n of P (4 codes per
// sdot4), then x = fma((float)acc * s_proj, c_emb[tok], PE[pos][n]).
__global__ __launch_bounds__(256) void k_embed_proj(const int32_t* __restrict__ tok, int S, const int* step,
                                                    const int8_t* __restrict__ E, int Ef, const int8_t* __restrict__ P,
                                                    float s_proj, const float* __restrict__ c_emb,
                                                    const float* __restrict__ pe, int d, int V, float* __restrict__ x) {
  __shared__ __attribute__((aligned(16))) int8_t e[kMaxEmbDim];
  const int r = blockIdx.x;
  int t = tok[r];
  t = t < 0 ? 0 : (t >= V ? V - 1 : t);
  const int pos = step ? *step : r % S;
  for (int k = threadIdx.x; k < Ef; k += blockDim.x) e[k] = E[(size_t)t * Ef + k];
  __syncthreads();
  const float c = c_emb[t];
  const int* er = reinterpret_cast<const int*>(e);
  for (int n = threadIdx.x; n < d; n += blockDim.x) {
    const int* pr = reinterpret_cast<const int*>(P + (size_t)n * Ef);
    int acc = 0;
    for (int k = 0; k < Ef / 4; ++k) acc = __builtin_amdgcn_sdot4(er[k], pr[k], acc, false);
    x[(size_t)r * d + n] = fmaf((float)acc * s_proj, c, pe[(size_t)pos * d + n]);
  }
}

// ---------------------------------------------------------------------------
// LayerNorm + quantization.  One wave per row; element i lives in lane i % 64
// (slot j = i / 64 of v) and is added to that lane's partial in ascending i
// (canonical order).  ln_quant_wave normalizes v in place (when do_ln) and
// stores the codes (q_row) and the normalized row (x_out_row), either may be
// null.
// ln_quant_wave_pre takes the LayerNorm's gain and bias already in
// registers (element lane + 64 j in slot j); ln_quant_wave loads them
// (clamped indexes, unconditional) before the reductions, so they arrive
// while the sums run.
template <int NJ>
__device__ __forceinline__ void ln_quant_wave_pre(float (&v)[NJ], int d, int do_ln, const float (&gj)[NJ],
                                                  const float (&bj)[NJ], float eps, float inv_s,
                                                  int8_t* __restrict__ q_row, float* __restrict__ x_out_row) {
  const int lane = threadIdx.x & 63;
  const int n = (d + 63) / 64;
  if (do_ln) {
    float p = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (j < n && i < d) p = p + v[j];
    }
    const float inv_d = 1.0f / (float)d;
    const float mu = wave_sum(p) * inv_d;
    float p2 = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (j < n && i < d) {
        v[j] = v[j] - mu;
        p2 = fmaf(v[j], v[j], p2);
      }
    }
    const float var = wave_sum(p2) * inv_d;
    const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (j < n && i < d) v[j] = fmaf(v[j] * rstd, gj[j], bj[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = lane + 64 * j;
    if (j < n && i < d) {
      if (q_row) q_row[i] = code_of(v[j] * inv_s);
      if (x_out_row) x_out_row[i] = v[j];
    }
  }
}

template <int NJ>
__device__ __forceinline__ void ln_consts(int d, int do_ln, const float* __restrict__ g, const float* __restrict__ b,
                                          float (&gj)[NJ], float (&bj)[NJ]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = min(lane + 64 * j, d - 1);
    gj[j] = do_ln ? g[i] : 0.0f;
    bj[j] = do_ln ? b[i] : 0.0f;
  }
}

template <int NJ>
__device__ __forceinline__ void ln_quant_wave(float (&v)[NJ], int d, int do_ln, const float* __restrict__ g,
                                              const float* __restrict__ b, float eps, float inv_s,
                                              int8_t* __restrict__ q_row, float* __restrict__ x_out_row) {
  float gj[NJ], bj[NJ];
  ln_consts<NJ>(d, do_ln, g, b, gj, bj);
  ln_quant_wave_pre<NJ>(v, d, do_ln, gj, bj, eps, inv_s, q_row, x_out_row);
}

// NJ = row_class(d) / 64; the row's loads are unconditional (clamped index).
template <int NJ>
__global__ __launch_bounds__(256) void k_ln_quant(const float* __restrict__ x, int rows, int d, int do_ln,
                                                  const float* __restrict__ g, const float* __restrict__ b,
                                                  float eps, float inv_s, int8_t* __restrict__ q,
                                                  float* __restrict__ x_out) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float* xr = x + (size_t)r * d;
  float v[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) v[j] = xr[min(lane + 64 * j, d - 1)];
  ln_quant_wave<NJ>(v, d, do_ln, g, b, eps, inv_s, q ? q + (size_t)r * d : nullptr,
                    x_out ? x_out + (size_t)r * d : nullptr);
}

// The pending residual update of a split-K layer, then k_ln_quant's row
// work: x = fma(gamma, x, fma((float)acc, scale, bias)) with acc the sum of
// the splits' int32 partials (the F32_RESID epilogue's expression), stored
// back (replace: the normalized row instead), LayerNorm, quantization.  Every
// load is issued before the first use (split indexes past the count repeat
// the last split and are not added).
template <int NJ>
__global__ __launch_bounds__(256) void k_resid_ln_quant(float* __restrict__ x, int rows, int d, ResidUpdate u,
                                                        int do_ln, const float* __restrict__ g,
                                                        const float* __restrict__ b, float eps, float inv_s,
                                                        int8_t* __restrict__ q, int replace) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  float* xr = x + (size_t)r * d;
  float v[NJ], sc[NJ], bi[NJ];
  int part[kMaxSplits][NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = min(lane + 64 * j, d - 1);
    v[j] = xr[i];
    sc[j] = u.scale[i];
    bi[j] = u.bias[i];
#pragma unroll
    for (int p = 0; p < kMaxSplits; ++p)
      part[p][j] = u.part[((size_t)min(p, u.splits - 1) * rows + r) * d + i];
  }
  float gj[NJ], bj[NJ];
  ln_consts<NJ>(d, do_ln, g, b, gj, bj);
  const int n = (d + 63) / 64;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    int acc = part[0][j];
#pragma unroll
    for (int p = 1; p < kMaxSplits; ++p) acc += p < u.splits ? part[p][j] : 0;
    v[j] = fmaf(u.gamma, v[j], fmaf((float)acc, sc[j], bi[j]));
    const int i = lane + 64 * j;
    if (!replace && j < n && i < d) xr[i] = v[j];
  }
  ln_quant_wave_pre<NJ>(v, d, do_ln, gj, bj, eps, inv_s, q + (size_t)r * d, replace ? xr : nullptr);
}

__device__ __forceinline__ int dot16v(const v4i a, const v4i b, int acc) {
  acc = __builtin_amdgcn_sdot4(a.x, b.x, acc, false);
  acc = __builtin_amdgcn_sdot4(a.y, b.y, acc, false);
  acc = __builtin_amdgcn_sdot4(a.z, b.z, acc, false);
  acc = __builtin_amdgcn_sdot4(a.w, b.w, acc, false);
  return acc;
}

// Attention for query rows that share one key/value set (the rows of one
// sentence in the encoder, the W hypotheses of one sentence over its source
// in the decoder's cross attention).  Block = (head, group): the block stages
// the group's keys and values of the head in LDS once (16-byte loads over all
// threads, issued together: positions and chunks past the valid ones repeat
// the last valid one and are never used), then each wave attends for its
// query rows, loading the next row's query while it works on the current one.
struct SharedAttn {
  const int8_t* q;       // query row r of the head at q + r * ldq + head * dh
  int ldq;
  // the fused query projection (kernel QF > 0): query row r of the head =
  // requant(a[r] . wq[head * dh + j]) with scale / bias, a [rows, d] int8,
  // wq [d, d] (QF 2: its packed 4-bit rows)
  const int8_t* a;
  const int8_t* wq;
  const float* q_scale;
  const float* q_bias;
  int ln_on;             // QF > 0: the rows a are computed from ln (LayerNorm + quantization of fp32 rows)
  FusedIn ln;
  int rows;              // query rows per group (row r = group * rows + i)
  const int8_t* kv;      // group g's key t of the head at kv + g * kv_group + k_off + t * ldkv + head * dh
  size_t kv_group;
  int ldkv, k_off, v_off;
  const int32_t* len;    // valid keys of group g: len[g] clamped to [1, S]
  int S, d, dh;
  float c_qk, c_pv;
  int8_t* ctx;           // context row r at ctx + r * d + head * dh
};

// QF 0: the query rows are read from a.q; QF 1 (int8 weights) or 2 (packed
// 4-bit weights): the block computes its group's query rows of the head
// itself (the cross-attention's Q projection, d = 64 KQ, at most 16 rows),
// on v_mfma_i32_16x16x64_i8 with the group's rows as A, wave w taking the
// 16-column fragments w, w + WAVES, ..., and the same requantization as the
// linear layer's I8 epilogue, into LDS.  With ln_on the group's A rows are
// the LayerNorm + quantization of its fp32 rows (prepare_rows, one row per
// wave at a time), computed while the weight, key and value loads are in
// flight.
template <int NMAX, int DHMAX, int WAVES, int QF = 0, int KQ = 1>
__global__ __launch_bounds__(64 * WAVES) void k_attn_shared(SharedAttn a) {
  static_assert(QF == 0 || WAVES == 4, "the row prologue runs on 4 waves");
  constexpr int DHC = DHMAX / 16, KS = DHMAX + 16, NI = NMAX / 64;
  constexpr int CH = NMAX * DHC, PER = (CH + 64 * WAVES - 1) / (64 * WAVES);
  constexpr int AL = 64 * KQ + 16;  // LDS row stride of the normalized rows
  __shared__ __attribute__((aligned(16))) int8_t kl[NMAX * KS];
  __shared__ __attribute__((aligned(16))) int8_t vl[NMAX * DHMAX];
  __shared__ __attribute__((aligned(16))) float pl[WAVES][NMAX];
  __shared__ __attribute__((aligned(16))) int8_t ql[QF ? 16 * DHMAX : 16];
  __shared__ __attribute__((aligned(16))) int8_t al[QF ? 16 * AL : 16];
  const int hd = blockIdx.x, g = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int dh = a.dh, nc = dh / 16;
  int n = a.len[g];
  n = n < 1 ? 1 : (n > a.S ? a.S : n);
  const int8_t* kb = a.kv + (size_t)g * a.kv_group + a.k_off + hd * dh;
  const int8_t* vb = a.kv + (size_t)g * a.kv_group + a.v_off + hd * dh;
  v4i kr[PER], vr[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int c = tid + u * 64 * WAVES;
    const int t = min(c / DHC, n - 1), cc = min(c % DHC, nc - 1);
    kr[u] = *(const v4i*)(kb + (size_t)t * a.ldkv + 16 * cc);
    vr[u] = *(const v4i*)(vb + (size_t)t * a.ldkv + 16 * cc);
  }
  const int rows = a.rows;
  auto qrow = [&](int i) { return a.q + ((size_t)g * rows + min(i, rows - 1)) * a.ldq + hd * dh; };
  v4i qn[DHC];
  if constexpr (QF == 0) {
#pragma unroll
    for (int c = 0; c < DHC; ++c) qn[c] = *(const v4i*)(qrow(wave) + 16 * min(c, nc - 1));
  } else {
    // the head's query rows: every operand load first, one fragment per wave
    // at a time (nc <= 8 fragments)
    constexpr bool W4 = QF == 2;
    const int d = 64 * KQ, l16 = lane & 15, koff = 16 * (lane >> 4);
    WFrag<W4> bf[KQ];
#pragma unroll
    for (int kk = 0; kk < KQ; ++kk) bf[kk] = load_wfrag_if<W4>(wave < nc, a.wq, hd * dh + 16 * wave + l16, d, 64 * kk + koff);
    v4i af[KQ];
    if (a.ln_on) {
      // one row per wave at a time: with the default four, each wave of a
      // four-row sentence loaded three clamped copies of its row as well
      // (6.98 -> 6.80 ms per mobile beam batch without them)
      prepare_rows<KQ, 1>(a.ln, rows, g * rows, d, 0, al, AL, false);
      lds_barrier();
#pragma unroll
      for (int kk = 0; kk < KQ; ++kk) af[kk] = *(const v4i*)(al + min(l16, rows - 1) * AL + 64 * kk + koff);
    } else {
      const int8_t* ar = a.a + ((size_t)g * rows + min(l16, rows - 1)) * d;
#pragma unroll
      for (int kk = 0; kk < KQ; ++kk) af[kk] = *(const v4i*)(ar + 64 * kk + koff);
    }
    for (int f = wave; f < nc; f += WAVES) {
      const int col = hd * dh + 16 * f + l16;
      if (f != wave) {
#pragma unroll
        for (int kk = 0; kk < KQ; ++kk) bf[kk] = load_wfrag<W4>(a.wq, col, d, 64 * kk + koff);
      }
      const float sc = a.q_scale[col], bi = a.q_bias[col];
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < KQ; ++kk) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[kk], bf[kk].get(), acc, 0, 0, 0);
      // element i of lane l: row 4 (l / 16) + i, column l % 16
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * (lane >> 4) + i;
        if (r < rows) ql[r * DHMAX + 16 * f + l16] = code_of(fmaf((float)acc[i], sc, bi));
      }
    }
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int c = tid + u * 64 * WAVES;
    if (c < CH) {
      const int t = c / DHC, cc = c % DHC;
      *(v4i*)(kl + t * KS + 16 * cc) = kr[u];
      *(v4i*)(vl + t * DHMAX + 16 * cc) = vr[u];
    }
  }
  lds_barrier();
  for (int i = wave; i < rows; i += WAVES) {
    v4i qv[DHC];
#pragma unroll
    for (int c = 0; c < DHC; ++c) {
      if constexpr (QF == 0) {
        qv[c] = qn[c];
        qn[c] = *(const v4i*)(qrow(i + WAVES) + 16 * min(c, nc - 1));
      } else {
        qv[c] = *(const v4i*)(ql + i * DHMAX + 16 * min(c, nc - 1));
      }
    }
    float sv[NI];
#pragma unroll
    for (int ii = 0; ii < NI; ++ii) {
      const int t = lane + 64 * ii;
      sv[ii] = 0.0f;
      if (t < n) {
        int acc = 0;
#pragma unroll
        for (int c = 0; c < DHC; ++c)
          if (c < nc) acc = dot16v(*(const v4i*)(kl + t * KS + 16 * c), qv[c], acc);
        sv[ii] = (float)acc * a.c_qk;
      }
    }
    softmax_context<NI>(sv, n, dh, a.c_pv, pl[wave], vl, DHMAX, a.ctx + ((size_t)g * rows + i) * a.d + hd * dh);
  }
}

// Decoder self-attention at position t = *step, block = row r: wave w takes
// heads w, w + WAVES, ...  It appends the row's new key and value of the head
// to the int8 cache and attends over positions 0..t (with beam search through
// the row's history of parent rows, hist[t & 1]; the key and value of
// position t are the new ones, read from qkv).  Loads are coalesced: CPP
// lanes take one position's dh codes (16 bytes each), so one load
// instruction covers 64 / CPP positions, and each position's score is the sum
// of its lanes' partial dot products (exact); the scores then pass through
// LDS into the one-key-per-lane layout of the canonical softmax.  Keys and
// values are loaded in batches of at most 8 instructions each, all of a batch
// issued together.
template <int NMAX, int DHMAX, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void k_attn_dec_self(const int8_t* __restrict__ qkv, int d, int h, int dh,
                                                              int T, const int* __restrict__ step,
                                                              int8_t* __restrict__ kcache, int8_t* __restrict__ vcache,
                                                              const int32_t* __restrict__ hist, float c_qk,
                                                              float c_pv, int8_t* __restrict__ ctx, int t_host) {
  constexpr int CPP = DHMAX / 16;  // lanes per position
  constexpr int PPI = 64 / CPP;    // positions per load instruction
  constexpr int NL = NMAX / PPI;   // load instructions per operand
  constexpr int NB = NL < 8 ? NL : 8;
  constexpr int NI = NMAX / 64;
  __shared__ AttnLdsT<NMAX, DHMAX> sh[WAVES];
  const int r = blockIdx.x, R = gridDim.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nc = dh / 16;
  const int c = lane % CPP, pp = lane / CPP, cc = min(c, nc - 1);
  int t = t_host >= 0 ? t_host : *step;
  t = t < 0 ? 0 : (t >= T ? T - 1 : t);
  const int n = t + 1;
  const int8_t* row = qkv + (size_t)r * 3 * d;
  // the rows that hold each position's key and value (beam: the parents)
  const int32_t* hr = hist ? hist + ((size_t)(t & 1) * R + r) * T : nullptr;
  int src[NL];
#pragma unroll
  for (int u = 0; u < NL; ++u) src[u] = hr ? hr[min(u * PPI + pp, t)] : r;
  for (int hd = wave; hd < h; hd += WAVES) {
    const int8_t* knew = row + d + hd * dh;
    const int8_t* vnew = row + 2 * d + hd * dh;
    const v4i qc = *(const v4i*)(row + hd * dh + 16 * cc);
    // the new key and value chunks for the cache append at the end
    const v4i kapp = *(const v4i*)(knew + 16 * min(lane, nc - 1));
    const v4i vapp = *(const v4i*)(vnew + 16 * min(lane, nc - 1));
    AttnLdsT<NMAX, DHMAX>& w = sh[wave];
#pragma unroll
    for (int u0 = 0; u0 < NL; u0 += NB) {
      v4i kr[NB], vr[NB];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int tp = min((u0 + u) * PPI + pp, t);
        const size_t off = ((size_t)src[u0 + u] * T + tp) * d + hd * dh + 16 * cc;
        kr[u] = *(const v4i*)(tp == t ? knew + 16 * cc : kcache + off);
        vr[u] = *(const v4i*)(tp == t ? vnew + 16 * cc : vcache + off);
      }
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        int acc = c < nc ? dot16v(kr[u], qc, 0) : 0;
#pragma unroll
        for (int o = 1; o < CPP; o <<= 1) acc += __shfl_xor(acc, o, 64);
        const int tp = (u0 + u) * PPI + pp;
        if (c == 0 && tp < n) w.p[tp] = (float)acc * c_qk;
        *(v4i*)&w.v[tp][16 * c] = vr[u];
      }
    }
    wave_sync();  // the scores and values visible to every lane
    float sv[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int tp = lane + 64 * i;
      sv[i] = tp < n ? w.p[tp] : 0.0f;
    }
    softmax_context<NI>(sv, n, dh, c_pv, w.p, &w.v[0][0], DHMAX, ctx + (size_t)r * d + hd * dh);
    // the new key and value into the cache, after every load of the head (no
    // other block reads position t of this step)
    if (lane < nc) {
      const size_t o = ((size_t)r * T + t) * d + hd * dh + 16 * lane;
      *(v4i*)(kcache + o) = kapp;
      *(v4i*)(vcache + o) = vapp;
    }
  }
}

// Decoder self-attention with the Q/K/V projection inside (the batched
// decoder, d = 64 KQ, heads up to 64 wide): block = (head, group of RB <= 16
// rows), 4 waves; the rows are independent (each has its own cache row and
// history), so a group may span sentences.  The block computes its rows of
// the head's q, k and v itself on v_mfma_i32_16x16x64_i8 (the rows as A, RB
// of its 16 rows real; wave w takes the 16-column fragments w, w + 4, w + 8
// of the head's 3 dh columns, q then k then v), with the linear layer's I8
// requantization, into LDS.  The input rows are int8 codes (a) or, with
// ln_on, the LayerNorm + quantization of fp32 rows that the block computes
// while its weight loads are in flight (after the pending update of a split
// W2 when ln.nparts > 0: the head-0 blocks store the updated rows to
// ln.x_out).  Wave w then attends for rows w,
// w + 4, ... as k_attn_dec_self does: cached positions 0..t-1 through the
// row's history, position t from LDS; the new key and value are appended to
// the cache after the wave's loads (no block reads position t of this step).
struct SelfQkvAttn {
  const int8_t* a;        // input rows [R, d] (ln_on == 0)
  int ln_on;
  FusedIn ln;
  const int8_t* wqkv;     // [3d, d] int8 (W4: packed 4-bit rows)
  const float* scale;     // [3d]
  const float* bias;
  int RB, R, dh, T;       // rows per block (at most 16), rows, head width, cache positions
  const int* step;
  int t_host;
  int8_t* kcache;         // [R][T][d]
  int8_t* vcache;
  const int32_t* hist;    // [2][R][T] or null
  float c_qk, c_pv;
  int8_t* ctx;            // [R, d]
};

template <int NMAX, int KQ, bool W4>
__global__ __launch_bounds__(256) void k_attn_self_qkv(SelfQkvAttn a) {
  constexpr int DHMAX = 64, CPP = DHMAX / 16, PPI = 64 / CPP, NL = NMAX / PPI, NB = NL < 8 ? NL : 8;
  constexpr int NI = NMAX / 64, D = 64 * KQ, AL = D + 16, QL = 3 * DHMAX, FPW = 3 * DHMAX / 16 / 4;
  __shared__ __attribute__((aligned(16))) int8_t al[16 * AL];
  __shared__ __attribute__((aligned(16))) int8_t ql[16 * QL];
  __shared__ AttnLdsT<NMAX, DHMAX> sh[4];
  const int hd = blockIdx.x, g = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int R = a.R, row0 = g * a.RB, rows = min(a.RB, R - row0), dh = a.dh, nc = dh / 16, T = a.T;
  const int l16 = lane & 15, koff = 16 * (lane >> 4);
  // 1. the wave's weight fragments and their requantization constants
  WFrag<W4> bf[FPW][KQ];
  float fsc[FPW], fbi[FPW];
#pragma unroll
  for (int u = 0; u < FPW; ++u) {
    const int f = wave + 4 * u;
    const bool ok = f < 3 * nc;
    const int col = ok ? (f / nc) * D + hd * dh + 16 * (f % nc) + l16 : 0;
#pragma unroll
    for (int kk = 0; kk < KQ; ++kk) bf[u][kk] = load_wfrag_if<W4>(ok, a.wqkv, col, D, 64 * kk + koff);
    fsc[u] = a.scale[col];
    fbi[u] = a.bias[col];
  }
  int t = a.t_host >= 0 ? a.t_host : *a.step;
  t = t < 0 ? 0 : (t >= T ? T - 1 : t);
  // 2. the sentence's input rows
  v4i af[KQ];
  if (a.ln_on) {
    // one row per wave (rows of more than four hypotheses take turns); the
    // head-0 blocks store the rows after a pending update
    prepare_rows<KQ, 1, true>(a.ln, rows, row0, D, 0, al, AL, hd == 0);
    lds_barrier();
#pragma unroll
    for (int kk = 0; kk < KQ; ++kk) af[kk] = *(const v4i*)(al + min(l16, rows - 1) * AL + 64 * kk + koff);
  } else {
    const int8_t* ar = a.a + ((size_t)row0 + min(l16, rows - 1)) * D;
#pragma unroll
    for (int kk = 0; kk < KQ; ++kk) af[kk] = *(const v4i*)(ar + 64 * kk + koff);
  }
  // 3. q | k | v of the rows (row i at ql + i QL: q, then k at DHMAX, v at 2 DHMAX)
#pragma unroll
  for (int u = 0; u < FPW; ++u) {
    const int f = wave + 4 * u;
    if (f < 3 * nc) {
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < KQ; ++kk) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[kk], bf[u][kk].get(), acc, 0, 0, 0);
      const int sel = f / nc, ff = f % nc;
      // element i of lane l: row 4 (l / 16) + i, column l % 16
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * (lane >> 4) + i;
        if (r < rows) ql[r * QL + sel * DHMAX + 16 * ff + l16] = code_of(fmaf((float)acc[i], fsc[u], fbi[u]));
      }
    }
  }
  lds_barrier();
  // 4. attention for the wave's rows
  const int n = t + 1, tc = t > 0 ? t - 1 : 0;  // cached positions 0..t-1 (tc: an in-bounds stand-in for t)
  const int c = lane % CPP, pp = lane / CPP, cc = min(c, nc - 1);
  AttnLdsT<NMAX, DHMAX>& w = sh[wave];
  for (int i = wave; i < rows; i += 4) {
    const int r = row0 + i;
    const int8_t* qr = ql + i * QL;
    const v4i qc = *(const v4i*)(qr + 16 * cc);
    const v4i kn = *(const v4i*)(qr + DHMAX + 16 * cc);
    const v4i vn = *(const v4i*)(qr + 2 * DHMAX + 16 * cc);
    const int32_t* hr = a.hist ? a.hist + ((size_t)(t & 1) * R + r) * T : nullptr;
    int src[NL];
#pragma unroll
    for (int u = 0; u < NL; ++u) src[u] = hr ? hr[min(u * PPI + pp, t)] : r;
#pragma unroll
    for (int u0 = 0; u0 < NL; u0 += NB) {
      v4i kr[NB], vr[NB];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int tp = min((u0 + u) * PPI + pp, t);
        const size_t off = ((size_t)src[u0 + u] * T + min(tp, tc)) * D + hd * dh + 16 * cc;
        kr[u] = *(const v4i*)(a.kcache + off);
        vr[u] = *(const v4i*)(a.vcache + off);
        if (tp == t) {
          kr[u] = kn;
          vr[u] = vn;
        }
      }
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        int acc = c < nc ? dot16v(kr[u], qc, 0) : 0;
#pragma unroll
        for (int o = 1; o < CPP; o <<= 1) acc += __shfl_xor(acc, o, 64);
        const int tp = (u0 + u) * PPI + pp;
        if (c == 0 && tp < n) w.p[tp] = (float)acc * a.c_qk;
        *(v4i*)&w.v[tp][16 * c] = vr[u];
      }
    }
    wave_sync();  // the scores and values visible to every lane
    float sv[NI];
#pragma unroll
    for (int ii = 0; ii < NI; ++ii) {
      const int tp = lane + 64 * ii;
      sv[ii] = tp < n ? w.p[tp] : 0.0f;
    }
    softmax_context<NI>(sv, n, dh, a.c_pv, w.p, &w.v[0][0], DHMAX, a.ctx + (size_t)r * D + hd * dh);
    // the new key and value into the cache, after every load of the row
    if (lane < nc) {
      const size_t o = ((size_t)r * T + t) * D + hd * dh + 16 * lane;
      *(v4i*)(a.kcache + o) = *(const v4i*)(qr + DHMAX + 16 * lane);
      *(v4i*)(a.vcache + o) = *(const v4i*)(qr + 2 * DHMAX + 16 * lane);
    }
    wave_sync();  // every lane's reads of w before the next row's writes
  }
}

// ---------------------------------------------------------------------------
// Greedy search bookkeeping.
__global__ void k_greedy_reset(unsigned long long* slots, int R, int steps, int32_t* cur_tok, int32_t* finished,
                               int32_t* out_len, int* step, int bos, unsigned long long* fslots, int n_fslots,
                               unsigned* epoch) {
  for (int r = threadIdx.x; r < R; r += blockDim.x) {
    slots[r] = 0ull;
    cur_tok[r] = bos;
    finished[r] = 0;
    out_len[r] = steps;
  }
  for (int i = threadIdx.x; i < n_fslots; i += blockDim.x) fslots[i] = 0ull;
  if (threadIdx.x == 0) {
    *step = 0;
    if (epoch) *epoch = *epoch + 1u;
  }
}

// Reads the step's arg-max slots (and clears them for the next step), records
// the tokens, applies the end-of-sentence rule and advances the step counter.
__global__ void k_greedy_commit(unsigned long long* slots, int R, int T, int32_t* cur_tok, int32_t* out_tok,
                                int32_t* finished, int32_t* out_len, int* step, int stop_at_eos, int eos,
                                int pad, unsigned long long* out_key) {
  const int t = *step;
  __syncthreads();  // every thread has read the step before it advances
  for (int r = threadIdx.x; r < R; r += blockDim.x) {
    const unsigned long long key = slots[r];
    const int tok = unpack_index(key);
    slots[r] = 0ull;
    const int fin = finished[r];
    if (t < T) out_tok[(size_t)t * R + r] = fin ? pad : tok;
    if (t < T && out_key) out_key[(size_t)t * R + r] = key;
    if (!fin && stop_at_eos && tok == eos) {
      finished[r] = 1;
      out_len[r] = t + 1;
    }
    cur_tok[r] = fin ? pad : tok;
  }
  if (threadIdx.x == 0) *step = t + 1;
}

__global__ void k_greedy_output(const int32_t* out_tok, const int32_t* out_len, int R, int T, int32_t* out,
                                int32_t* out_len_dst, const int* chain_err) {
  const int r = blockIdx.x;
  for (int t = threadIdx.x; t < T; t += blockDim.x) out[(size_t)r * T + t] = out_tok[(size_t)t * R + r];
  if (threadIdx.x == 0) out_len_dst[r] = (chain_err && *chain_err) ? -1 : out_len[r];
}

__global__ void k_fill_lp(LpTable tab, float* dst) {
  for (int i = threadIdx.x; i < tab.n; i += blockDim.x) dst[i] = tab.v[i];
}

// Arg-max of fp32 rows (smallest index among equal maxima), one wave per row.
__global__ __launch_bounds__(256) void k_row_argmax(const float* __restrict__ z, int R, int V,
                                                    unsigned long long* slots) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  unsigned long long best = 0ull;
  for (int v = lane; v < V; v += 64) {
    const unsigned long long k = pack_argmax(z[(size_t)r * V + v], v);
    best = k > best ? k : best;
  }
  best = wave_max_u64(best);
  if (lane == 0) slots[r] = best;
}

// The batch's source ids and lengths into the session, and the encoder
// chain's flag words cleared for the translation that follows.
__global__ void k_load_batch(const int32_t* src_in, const int32_t* len_in, int32_t* src, int32_t* len, int n_src,
                             int n_len, unsigned* zero, int n_zero) {
  const int stride = gridDim.x * blockDim.x;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n_src; i += stride) src[i] = src_in[i];
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n_len; i += stride) len[i] = len_in[i];
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n_zero; i += stride) zero[i] = 0u;
}

__global__ void k_copy_i32(const int32_t* src, int32_t* dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

// Fragment order (see frag_bytes): output chunk c of 16 bytes is lane
// l = c % 64 of slice j = (c / 64) % (K / 64) of tile t = c / (64 * K / 64),
// i.e. row 16t + l % 16, columns 64j + 16(l / 16) .. +15; rows past N are zero.
__global__ __launch_bounds__(256) void k_pack_fragments(const int8_t* __restrict__ W, int N, int K, size_t chunks,
                                                        int8_t* __restrict__ out) {
  const size_t c = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= chunks) return;
  const int ks = K / 64, lane = (int)(c % 64);
  const size_t j = (c / 64) % ks, t = c / (64 * (size_t)ks);
  const size_t row = 16 * t + (lane & 15);
  int4 v = {0, 0, 0, 0};
  if (row < (size_t)N) v = *(const int4*)(W + row * K + 64 * j + 16 * (lane >> 4));
  *(int4*)(out + 16 * c) = v;
}

// ---------------------------------------------------------------------------
// Beam search.  Rows r = b * W + j hold the W hypotheses of sentence b.

// Candidate order: higher score first, then smaller index.
__device__ __forceinline__ bool better(float c1, int i1, float c2, int i2) {
  return c1 > c2 || (c1 == c2 && i1 < i2);
}

// The search state before the first step, one element per thread over a
// grid that covers the [R][T] histories (consecutive threads write
// consecutive words of every array).
__global__ __launch_bounds__(256) void k_beam_reset(BeamState st, int* step) {
  const int R = st.B * st.W, T = st.T;
  const size_t RT = (size_t)R * T, stride = (size_t)blockDim.x * gridDim.x;
  const size_t i0 = threadIdx.x + (size_t)blockIdx.x * blockDim.x;
  for (size_t e = i0; e < RT; e += stride) {
    // every position points at a valid cache row: hist is [2][R][T] ...
    const int32_t rh = (int32_t)(e / T);
    st.hist[e] = rh;
    st.hist[RT + e] = rh;
    // ... the token and parent histories [T][R]
    const int32_t rt = (int32_t)(e % R);
    st.tok_hist[e] = st.pad;
    st.par_hist[e] = rt;
  }
  for (size_t r = i0; r < (size_t)R; r += stride) {
    st.score[r] = 0.0f;
    st.cur_tok[r] = st.bos;
  }
  for (size_t b = i0; b < (size_t)st.B; b += stride) {
    st.fin_count[b] = 0;
    st.done[b] = 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    *step = 0;
    *st.count = 0;
  }
}

// Per live row: log-softmax statistics of the logits (max, then the canonical
// sum of exp(z - max), lse = max + ln sum) and the row's K = 2W best
// expansions by (score + (z - lse) desc, token asc).  One wave per row.
template <int K>
__global__ __launch_bounds__(64) void k_beam_topk(const float* __restrict__ logits, BeamState st,
                                                  const int* __restrict__ step) {
  const int r = blockIdx.x;
  const int lane = threadIdx.x;
  const int t = st.t_host >= 0 ? st.t_host : *step;
  const int b = r / st.W, j = r % st.W;
  if (st.done[b] || (t == 0 && j > 0)) return;
  const int V = st.V;
  const float* z = logits + (size_t)r * V;
  float mx = -FLT_MAX;
  for (int v = lane; v < V; v += 64) mx = fmaxf(mx, z[v]);
  mx = wave_max(mx);
  // the vocabulary order (R2b): lane l holds partials 64 w + l (w = 0..7),
  // fed the four-term groups g = l, l + 64, ... (partial g mod 512)
  float pw[8];
#pragma unroll
  for (int w = 0; w < 8; ++w) pw[w] = 0.0f;
  for (int g = lane; 4 * g < V; g += 64) {
    const int wg = (g >> 6) & 7;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int v = 4 * g + q;
      if (v < V) {
        const float e = canon_exp(z[v] - mx);
#pragma unroll
        for (int w = 0; w < 8; ++w)
          if (w == wg) pw[w] = pw[w] + e;
      }
    }
  }
  float gs[8];
#pragma unroll
  for (int w = 0; w < 8; ++w) gs[w] = wave_sum(pw[w]);
  const float lse = mx + canon_log(((gs[0] + gs[1]) + (gs[2] + gs[3])) + ((gs[4] + gs[5]) + (gs[6] + gs[7])));
  const float sc = st.score[r];
  float ls[K];
  int lv[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    ls[k] = -FLT_MAX;
    lv[k] = INT_MAX;
  }
  for (int v = lane; v < V; v += 64) {
    float c = sc + (z[v] - lse);
    int cv = v;
    if (!better(c, cv, ls[K - 1], lv[K - 1])) continue;
#pragma unroll
    for (int k = 0; k < K; ++k) {  // insertion by swapping keeps the list sorted
      if (better(c, cv, ls[k], lv[k])) {
        const float tc = ls[k];
        const int tv = lv[k];
        ls[k] = c;
        lv[k] = cv;
        c = tc;
        cv = tv;
      }
    }
  }
  // Merge the 64 sorted lists: K rounds of a wave-wide maximum of the heads.
  for (int k = 0; k < K; ++k) {
    const unsigned long long mine = lv[0] == INT_MAX ? 0ull : pack_argmax(ls[0], lv[0]);
    const unsigned long long win = wave_max_u64(mine);
    if (mine == win && win != 0ull) {
#pragma unroll
      for (int i = 0; i + 1 < K; ++i) {
        ls[i] = ls[i + 1];
        lv[i] = lv[i + 1];
      }
      ls[K - 1] = -FLT_MAX;
      lv[K - 1] = INT_MAX;
    }
    if (lane == 0) {
      const int v = win ? unpack_index(win) : 0;
      st.cand_tok[(size_t)r * K + k] = v;
      st.cand_score[(size_t)r * K + k] = win ? sc + (z[v] - lse) : -FLT_MAX;
    }
  }
}

// The same statistics and candidates with one 512-thread block per row, for
// V a multiple of 4 up to kTopkMaxV: the row is loaded once into registers
// (element 4 (tid + 512 k) + q: 16 bytes per load, up to 16 per thread, all
// in flight), the maximum (order-free) taken from them, and each thread adds
// exp(z - max) of its own elements in ascending order: exactly the partials
// of the vocabulary order (R2b: 512 partials fed four consecutive terms at a
// time), so the wave butterflies and the tree of the 8 wave sums finish the
// sum with no exchange of the exponentials.  The candidates then come from a
// threshold: the score is monotone in z, so for K <= 8 the smallest of the 8
// wave maxima of z bounds at least 8 scores from below (one per wave), and
// otherwise each thread's best score is score + (its max z - lse) and the
// K-th largest of these over the lanes of a wave has at least K scores of the
// row at or above it (the largest such bound over the waves is taken).  The
// bound filters the row down to a short list (about 3K entries on real logits),
// ranked by one wave (up to 64 entries) or pairwise comparison.  If ties push
// the list past kTopkCap, per-thread sorted lists over the threads' own
// elements, merged over the block, take over.  The candidate order is total
// (score, then index), so neither the filter nor the split over threads
// changes the result.
constexpr int kTopkMaxV = 32768;
constexpr int kTopkThreads = 512, kTopkWaves = kTopkThreads / 64;
constexpr int kTopkV4 = kTopkMaxV / 4 / kTopkThreads;  // float4 per thread
constexpr int kTopkCap = 1024;                // entries of the filtered list
static_assert(kTopkThreads == 512, "the vocabulary order has 512 partials");

__device__ __forceinline__ unsigned long long block_max_u64(unsigned long long v, unsigned long long* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_max_u64(v);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  unsigned long long m = red[0];
#pragma unroll
  for (int w = 1; w < kTopkWaves; ++w) m = red[w] > m ? red[w] : m;
  __syncthreads();  // red is reused by the next call
  return m;
}

// Per-thread sorted lists over the thread's own elements (scores
// sc + (z - lse) of elements 4 (tid + 512 k) + q), merged over the block: the
// path for rows whose filtered list overflows (large groups of equal scores).
// It reads the row again from memory, in a loop that is not unrolled: the
// common path then holds neither the row's registers nor this code inline.
template <int K>
__device__ __noinline__ void topk_lists(const float4* __restrict__ z4, int n4, float sc, float lse,
                                        unsigned long long* redk, int* cand_tok, float* cand_score) {
  const int tid = threadIdx.x;
  float ls[K];
  int lv[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    ls[k] = -FLT_MAX;
    lv[k] = INT_MAX;
  }
#pragma unroll 1
  for (int k = 0; k < kTopkV4; ++k) {
    const int i = tid + kTopkThreads * k;
    if (i >= n4) continue;
    const float4 zk = z4[i];
    const float zq[4] = {zk.x, zk.y, zk.z, zk.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float c = sc + (zq[q] - lse);
      int cv = 4 * i + q;
      if (!better(c, cv, ls[K - 1], lv[K - 1])) continue;
#pragma unroll
      for (int m = 0; m < K; ++m) {  // insertion by swapping keeps the list sorted
        if (better(c, cv, ls[m], lv[m])) {
          const float tc = ls[m];
          const int tv = lv[m];
          ls[m] = c;
          lv[m] = cv;
          c = tc;
          cv = tv;
        }
      }
    }
  }
  for (int k = 0; k < K; ++k) {
    const unsigned long long mine = lv[0] == INT_MAX ? 0ull : pack_argmax(ls[0], lv[0]);
    const unsigned long long win = block_max_u64(mine, redk);
    if (mine == win && win != 0ull) {  // the owner of the winner records and drops it
      cand_tok[k] = lv[0];
      cand_score[k] = ls[0];
#pragma unroll
      for (int i = 0; i + 1 < K; ++i) {
        ls[i] = ls[i + 1];
        lv[i] = lv[i + 1];
      }
      ls[K - 1] = -FLT_MAX;
      lv[K - 1] = INT_MAX;
    }
    if (win == 0ull && tid == 0) {
      cand_tok[k] = 0;
      cand_score[k] = -FLT_MAX;
    }
  }
}

template <int K>
__global__ __launch_bounds__(kTopkThreads) void k_beam_topk_block(const float* __restrict__ logits, BeamState st,
                                                         const int* __restrict__ step) {
  // 8 entries past the cap: the ranking reads the list 8 entries at a time
  __shared__ __attribute__((aligned(16))) float list_c[kTopkCap + 8];
  __shared__ __attribute__((aligned(16))) int list_v[kTopkCap + 8];
  __shared__ float redf[kTopkWaves];
  __shared__ float reds[kTopkWaves];
  __shared__ unsigned long long redk[kTopkWaves];
  __shared__ int n_list;
  const int r = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = st.t_host >= 0 ? st.t_host : *step;
  const int b = r / st.W, j = r % st.W;
  if (st.done[b] || (t == 0 && j > 0)) return;
  const int V = st.V, n4 = V / 4;
  const float4* z4 = reinterpret_cast<const float4*>(logits + (size_t)r * V);
  int* cand_tok = st.cand_tok + (size_t)r * K;
  float* cand_score = st.cand_score + (size_t)r * K;
  const float sc = st.score[r];
  if (tid == 0) n_list = 0;
  // 1. the row in registers (element 4 (tid + kTopkThreads k) + q), the thread's
  //    maximum and the row's
  float4 zr[kTopkV4];
#pragma unroll
  for (int k = 0; k < kTopkV4; ++k) zr[k] = z4[min(tid + kTopkThreads * k, n4 - 1)];
  float tmx = -INFINITY;
#pragma unroll
  for (int k = 0; k < kTopkV4; ++k)
    if (tid + kTopkThreads * k < n4) tmx = fmaxf(tmx, fmaxf(fmaxf(zr[k].x, zr[k].y), fmaxf(zr[k].z, zr[k].w)));
  float mx = wave_max(fmaxf(tmx, -FLT_MAX));
  if (lane == 0) redf[wave] = mx;
  __syncthreads();
  mx = redf[0];
#pragma unroll
  for (int w = 1; w < kTopkWaves; ++w) mx = fmaxf(mx, redf[w]);
  // 2. the sum of exp(z - max) in the vocabulary order: the thread's partial
  //    over its elements in ascending order, the wave butterfly, the tree
  float part = 0.0f;
#pragma unroll
  for (int k = 0; k < kTopkV4; ++k) {
    if (tid + kTopkThreads * k < n4) {
      part = part + canon_exp(zr[k].x - mx);
      part = part + canon_exp(zr[k].y - mx);
      part = part + canon_exp(zr[k].z - mx);
      part = part + canon_exp(zr[k].w - mx);
    }
  }
  part = wave_sum(part);
  if (lane == 0) reds[wave] = part;
  __syncthreads();
  const float lse =
      mx + canon_log(((reds[0] + reds[1]) + (reds[2] + reds[3])) + ((reds[4] + reds[5]) + (reds[6] + reds[7])));
  // 3. the bound (scores below -FLT_MAX never qualify).  K <= 8 with every
  //    wave holding elements (V > 1792): the smallest of the 8 wave maxima
  //    (already in redf), since each wave has an element at or above it.
  //    Otherwise the K-th largest thread-best score of each wave, the largest
  //    over the waves.
  float tau;
  if (K <= kTopkWaves && n4 > kTopkThreads - 64) {
    float zmin = redf[0];
#pragma unroll
    for (int w = 1; w < kTopkWaves; ++w) zmin = fminf(zmin, redf[w]);
    tau = fmaxf(sc + (zmin - lse), -FLT_MAX);
  } else {
    const float cm = sc + (tmx - lse);
    float v = cm >= -FLT_MAX ? cm : -INFINITY;
    float kth = -INFINITY;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      kth = wave_max(v);
      const unsigned long long hold = __ballot(v == kth);
      if (lane == __ffsll((long long)hold) - 1) v = -INFINITY;  // drop one holder
    }
    __syncthreads();  // every read of redf (the maximum) is done
    if (lane == 0) redf[wave] = fmaxf(kth, -FLT_MAX);
    __syncthreads();
    tau = redf[0];
#pragma unroll
    for (int w = 1; w < kTopkWaves; ++w) tau = fmaxf(tau, redf[w]);
  }
  // 4. the filtered list: every score at or above the bound (one branch and
  //    at most one list slot reservation per 4 elements)
#pragma unroll
  for (int k = 0; k < kTopkV4; ++k) {
    const int i = tid + kTopkThreads * k;
    const float c4[4] = {sc + (zr[k].x - lse), sc + (zr[k].y - lse), sc + (zr[k].z - lse),
                         sc + (zr[k].w - lse)};
    const int m = (int)(c4[0] >= tau) + (int)(c4[1] >= tau) + (int)(c4[2] >= tau) + (int)(c4[3] >= tau);
    if (i < n4 && m > 0) {
      int pos = atomicAdd(&n_list, m);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (c4[q] >= tau) {
          if (pos < kTopkCap) {
            list_c[pos] = c4[q];
            list_v[pos] = 4 * i + q;
          }
          ++pos;
        }
      }
    }
  }
  __syncthreads();
  const int n = n_list;
  if (n <= 64) {
    // 5. up to 64 entries, one per lane of wave 0: rank = the number of
    //    lanes whose (score, -index) key is larger (keys are distinct; the
    //    order of pack_argmax is better()'s with -0 read as +0)
    if (wave == 0) {
      const bool live = lane < n;
      const float ci = live ? list_c[lane] : -FLT_MAX;
      const int vi = live ? list_v[lane] : 0;
      const unsigned long long key = live ? pack_argmax(ci == 0.0f ? 0.0f : ci, vi) : 0ull;
      const int hi = (int)(key >> 32), lo = (int)(uint32_t)key;
      int rank = 0;
#pragma unroll
      for (int o = 0; o < 64; ++o) {
        const unsigned long long ko = ((unsigned long long)(uint32_t)__builtin_amdgcn_readlane(hi, o) << 32) |
                                      (uint32_t)__builtin_amdgcn_readlane(lo, o);
        rank += ko > key ? 1 : 0;
      }
      if (live && rank < K) {
        cand_tok[rank] = vi;
        cand_score[rank] = ci;
      }
      if (!live && lane < K) {  // fewer than K scores qualify
        cand_tok[lane] = 0;
        cand_score[lane] = -FLT_MAX;
      }
    }
    return;
  }
  if (n <= kTopkCap) {
    // 5. rank = the number of list entries that beat the entry, the list
    //    read 8 entries at a time (four 16-byte reads issued together, the
    //    entries past n masked)
    for (int i = tid; i < n; i += kTopkThreads) {
      const float ci = list_c[i];
      const int vi = list_v[i];
      int rank = 0;
      for (int o0 = 0; o0 < n; o0 += 8) {
        const float4 c0 = *(const float4*)&list_c[o0], c1 = *(const float4*)&list_c[o0 + 4];
        const int4 v0 = *(const int4*)&list_v[o0], v1 = *(const int4*)&list_v[o0 + 4];
        const float co[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
        const int vo[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int u = 0; u < 8; ++u) rank += (o0 + u < n && better(co[u], vo[u], ci, vi)) ? 1 : 0;
      }
      if (rank < K) {
        cand_tok[rank] = vi;
        cand_score[rank] = ci;
      }
    }
    for (int k = n + tid; k < K; k += kTopkThreads) {  // fewer than K scores qualify
      cand_tok[k] = 0;
      cand_score[k] = -FLT_MAX;
    }
    return;
  }
  // 5'. the overflow path: per-thread sorted lists, block merge
  topk_lists<K>(z4, n4, sc, lse, redk, cand_tok, cand_score);
}

// Per sentence: merge the W rows' candidates, finish EOS hypotheses, refill
// the W live slots and advance the key/value history; then the next step's
// input rows of the sentence's slots (BeamNext), and the step counter
// (advanced by the last block).  One block per sentence: wave 0 updates the
// sentence, then wave w prepares slots w, w + kUpdWaves, ...
constexpr int kUpdWaves = 4;
// NJ = row_class(d) / 64.  Everything that does not depend on the update
// (the sentence's finished count, the length penalty, the candidates, the
// next position's row of the position table and the LayerNorm constants) is
// loaded at kernel start; the history copy runs one slot per wave.
template <int W_MAX, int NJ>
__global__ __launch_bounds__(64 * kUpdWaves) void k_beam_update(BeamState st, int* step, BeamNext nx) {
  constexpr int NC = W_MAX * 2 * W_MAX;  // candidates per sentence
  __shared__ float cs[NC];
  __shared__ int cj[NC], cv[NC];
  __shared__ int order[2 * W_MAX];
  __shared__ int new_par[W_MAX], new_tok[W_MAX];
  __shared__ float new_score[W_MAX];
  __shared__ int n_live_sh, done_sh;
  __shared__ int slot_tok[W_MAX];  // each slot's token after the update
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const bool w0 = wv == 0;  // the wave that ranks the sentence's candidates
  const int W = st.W, K = 2 * W, R = st.B * W, T = st.T, V = st.V;
  const int t = st.t_host >= 0 ? st.t_host : *step;
  const bool active = !st.done[b];
  const int pos = t + 1;
  const bool prep = pos < nx.steps && pos < nx.P;
  float pe_r[NJ], gj[NJ], bj[NJ];
  {
    const int pp = min(pos, nx.P - 1);
#pragma unroll
    for (int j = 0; j < NJ; ++j) pe_r[j] = nx.pe[(size_t)pp * nx.d + min(lane + 64 * j, nx.d - 1)];
    ln_consts<NJ>(nx.d, nx.do_ln, nx.g, nx.b, gj, bj);
  }
  const int fc0 = st.fin_count[b];
  const float lp_next = st.lp[min(t + 1, T)];
  if (threadIdx.x < W) slot_tok[threadIdx.x] = st.cur_tok[b * W + threadIdx.x];
  if (active) {
    const int n_alive = t == 0 ? 1 : W;
    const int n = n_alive * K;
    for (int i = lane; w0 && i < NC; i += 64) {
      if (i < n) {
        const int jj = i / K, k = i % K;
        const int r = b * W + jj;
        cs[i] = st.cand_score[(size_t)r * K + k];
        cv[i] = st.cand_tok[(size_t)r * K + k];
        cj[i] = jj;
      }
    }
    __syncthreads();
    // rank of each candidate = number of better candidates (flat index j*V + v breaks ties)
    if (n <= 64 && (long)W * V <= 0x7fffffffL) {
      // one candidate per lane of wave 0, each counting the larger of the 64
      // (score, -flat index) keys read across lanes (pack_argmax order, which
      // is the comparison's with -0 read as +0; dead lanes hold key 0)
      if (w0) {
        const bool live = lane < n;
        const float ci = live ? cs[lane] : 0.0f;
        const unsigned long long key = live ? pack_argmax(ci == 0.0f ? 0.0f : ci, cj[lane] * V + cv[lane]) : 0ull;
        const int hi = (int)(key >> 32), lo = (int)(uint32_t)key;
        int rank = 0;
#pragma unroll
        for (int o = 0; o < 64; ++o) {
          const unsigned long long ko = ((unsigned long long)(uint32_t)__builtin_amdgcn_readlane(hi, o) << 32) |
                                        (uint32_t)__builtin_amdgcn_readlane(lo, o);
          rank += ko > key ? 1 : 0;
        }
        if (live && rank < K) order[rank] = lane;
      }
    } else {
      for (int i = lane; w0 && i < n; i += 64) {
        int rank = 0;
        const long fi = (long)cj[i] * V + cv[i];
        for (int o = 0; o < n; ++o) {
          const long fo = (long)cj[o] * V + cv[o];
          rank += (cs[o] > cs[i] || (cs[o] == cs[i] && fo < fi)) ? 1 : 0;
        }
        if (rank < K) order[rank] = i;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int n_live = 0;
      int fc = fc0;
      const int n_top = n < K ? n : K;
      for (int rk = 0; rk < n_top && n_live < W; ++rk) {
        const int i = order[rk];
        if (cv[i] == st.eos) {
          if (rk < W && fc < W) {
            st.fin_score[b * W + fc] = cs[i] / lp_next;
            st.fin_len[b * W + fc] = t + 1;
            st.fin_row[b * W + fc] = b * W + cj[i];
            ++fc;
          }
          continue;
        }
        new_par[n_live] = b * W + cj[i];
        new_tok[n_live] = cv[i];
        new_score[n_live] = cs[i];
        ++n_live;
      }
      st.fin_count[b] = fc;
      if (fc >= W) st.done[b] = 1;
      n_live_sh = n_live;
      done_sh = fc >= W;
    }
  }
  __syncthreads();  // the selection (and each slot's current token) visible to every wave
  // One wave per slot: the slot's history copy (refilled slots) and the next
  // step's input row (what k_embed and k_ln_quant compute), all of the slot's
  // loads issued before its first store (the memory counter retires in
  // order: a load waited for after a store would also wait for the store).
  const int n_live = active && !done_sh ? n_live_sh : 0;
  const int32_t* hcur = st.hist + (size_t)(t & 1) * R * T;
  int32_t* hnext = st.hist + (size_t)((t + 1) & 1) * R * T;
  for (int s = wv; s < W; s += kUpdWaves) {
    const int p = b * W + s;
    const bool refill = s < n_live;
    const int par = refill ? new_par[s] : p;
    int tk = refill ? new_tok[s] : slot_tok[s];
    tk = tk < 0 ? 0 : (tk >= nx.V ? nx.V - 1 : tk);
    int hv[kMaxAttnLen / 64];
    if (refill) {
#pragma unroll
      for (int i = 0; i < kMaxAttnLen / 64; ++i) hv[i] = hcur[(size_t)par * T + min(lane + 64 * i, t)];
    }
    float e[NJ], c = 0.0f;
    if (prep) {
      c = nx.c_emb[tk];
#pragma unroll
      for (int j = 0; j < NJ; ++j) e[j] = (float)nx.E[(size_t)tk * nx.d + min(lane + 64 * j, nx.d - 1)];
    }
    if (refill) {
#pragma unroll
      for (int i = 0; i < kMaxAttnLen / 64; ++i) {
        const int tp = lane + 64 * i;
        if (tp <= t && tp < T) hnext[(size_t)p * T + tp] = tp < t ? hv[i] : par;
      }
      if (lane == 0) {
        st.score[p] = new_score[s];
        st.cur_tok[p] = new_tok[s];
        if (t < T) {
          st.tok_hist[(size_t)t * R + p] = new_tok[s];
          st.par_hist[(size_t)t * R + p] = par;
        }
      }
    }
    if (prep) {
      float v[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int i = lane + 64 * j;
        v[j] = fmaf(e[j], c, pe_r[j]);
        if (i < nx.d) nx.x[(size_t)p * nx.d + i] = v[j];
      }
      ln_quant_wave_pre<NJ>(v, nx.d, nx.do_ln, gj, bj, nx.eps, nx.inv_s, nx.a + (size_t)p * nx.d, nullptr);
    }
  }
  // the step counter, by the last block to get here (every block has read it)
  __syncthreads();
  if (threadIdx.x == 0 && atomicAdd(st.count, 1) == (int)gridDim.x - 1) {
    *st.count = 0;
    *step = t + 1;
  }
}

// Per sentence: finish the live hypotheses if the sentence never completed,
// pick the best normalized score (the first finished among equals: EOS
// hypotheses in the order they finished, then the live slots in slot order)
// and write its tokens.  One wave per sentence: the sentence's parent slots
// of steps 0..last go to LDS in one round of loads, lane 0 follows the
// parents back from the chosen hypothesis there, and the lanes then read the
// tokens of the path together (each step's token is that of the path's slot).
constexpr int kFinMaxSteps = 256, kFinMaxW = 8;
__global__ __launch_bounds__(64) void k_beam_finalize(BeamState st, int steps, int32_t* out, int32_t* out_len,
                                                      float* out_score, const int* chain_err) {
  __shared__ uint8_t par_s[kFinMaxSteps][kFinMaxW];  // parent slot of (step, slot)
  __shared__ uint8_t path[kFinMaxSteps];             // the hypothesis' slot at each step
  const int b = blockIdx.x, lane = threadIdx.x;
  const int W = st.W, R = st.B * W, r0 = b * W;
  int kind = -1, idx = 0;  // kind 0: finished entry idx; kind 1: live slot idx
  float best = 0.0f;
  const int fc = st.fin_count[b];
  for (int i = 0; i < fc; ++i) {
    const float v = st.fin_score[r0 + i];
    if (kind < 0 || v > best) {
      best = v;
      kind = 0;
      idx = i;
    }
  }
  if (!st.done[b]) {
    for (int s = 0; s < W; ++s) {
      const float v = st.score[r0 + s] / st.lp[steps];
      if (kind < 0 || v > best) {
        best = v;
        kind = 1;
        idx = s;
      }
    }
  }
  // the tokens of steps 0..last come from the path ending in `row`
  const int L = kind == 1 ? steps : st.fin_len[r0 + idx];
  const int last = min(kind == 1 ? steps - 1 : L - 2, steps - 1);
  const int row = kind == 1 ? r0 + idx : st.fin_row[r0 + idx];
  for (int e = lane; e < (last + 1) * W; e += 64) {
    const int t = e / W, j = e % W;
    par_s[t][j] = (uint8_t)min(max(st.par_hist[(size_t)t * R + r0 + j] - r0, 0), W - 1);
  }
  __syncthreads();
  if (lane == 0) {
    int slot = min(max(row - r0, 0), W - 1);
    for (int t = last; t >= 0; --t) {
      path[t] = (uint8_t)slot;
      slot = par_s[t][slot];
    }
  }
  __syncthreads();
  int32_t* o = out + (size_t)b * steps;
  for (int t = lane; t <= last; t += 64) o[t] = st.tok_hist[(size_t)t * R + r0 + path[t]];
  if (kind == 0 && lane == 0) o[L - 1] = st.eos;
  for (int t = L + lane; t < steps; t += 64) o[t] = st.pad;
  if (lane == 0) {
    out_len[b] = (chain_err && *chain_err) ? -1 : L;
    if (out_score) out_score[b] = best;
  }
}

// ---------------------------------------------------------------------------
// A plain read of n16 16-byte words (each block XOR-folds its share into one
// word of sink): the memory system's read bandwidth for the data's location
// (last-level cache when the buffer was just read and fits, HBM otherwise).
__global__ __launch_bounds__(256) void k_debug_read(const uint4* __restrict__ x, size_t n16, int reps,
                                                    unsigned* sink) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  uint4 acc = {0u, 0u, 0u, 0u};
  for (int rep = 0; rep < reps; ++rep) {
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
      const uint4 a = x[i], b = x[i + stride], c = x[i + 2 * stride], e = x[i + 3 * stride];
      acc.x ^= a.x ^ b.x ^ c.x ^ e.x;
      acc.y ^= a.y ^ b.y ^ c.y ^ e.y;
      acc.z ^= a.z ^ b.z ^ c.z ^ e.z;
      acc.w ^= a.w ^ b.w ^ c.w ^ e.w;
    }
    for (; i < n16; i += stride) {
      const uint4 a = x[i];
      acc.x ^= a.x;
      acc.y ^= a.y;
      acc.z ^= a.z;
      acc.w ^= a.w;
    }
    // keep each pass a real read (no folding of identical passes)
    asm volatile("" : "+v"(acc.x), "+v"(acc.y), "+v"(acc.z), "+v"(acc.w));
  }
  unsigned v = acc.x ^ acc.y ^ acc.z ^ acc.w;
  for (int off = 32; off >= 1; off /= 2) v ^= __shfl_xor(v, off);
  __shared__ unsigned part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

__global__ void k_debug_canon(int fn, const float* x, int n, float* y) {
  const int lane = threadIdx.x & 63;
  if (fn == 0 || fn == 1) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += blockDim.x * gridDim.x)
      y[i] = fn == 0 ? canon_exp(x[i]) : canon_log(x[i]);
    return;
  }
  if (blockIdx.x != 0 || threadIdx.x >= 64) return;
  if (fn == 2) {
    float p = 0.0f;
    for (int i = lane; i < n; i += 64) p = p + x[i];
    p = wave_sum(p);
    if (lane == 0) y[0] = p;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers.

hipError_t launch_embed(const int32_t* tok, int rows, int S_for_pos, const int* step, const int8_t* E,
                        const float* c_emb, const float* pe, int d, int V, float* x, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_embed, dim3((rows + 3) / 4), dim3(256), 0, s, tok, rows, S_for_pos, step, E, c_emb, pe, d, V,
                     x);
  return hipGetLastError();
}

hipError_t launch_embed_proj(const int32_t* tok, int rows, int S_for_pos, const int* step, const int8_t* E, int Ef,
                             const int8_t* P, float s_proj, const float* c_emb, const float* pe, int d, int V,
                             float* x, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (Ef < 4 || Ef % 4 || Ef > kMaxEmbDim) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed_proj, dim3(rows), dim3(256), 0, s, tok, S_for_pos, step, E, Ef, P, s_proj, c_emb, pe, d,
                     V, x);
  return hipGetLastError();
}

hipError_t launch_ln_quant(const float* x, int rows, int d, int do_ln, const float* g, const float* b, float eps,
                           float inv_s, int8_t* q, float* x_out, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d > kMaxRowLen) return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4);
#define MNMT_LNQ(NJ) \
  hipLaunchKernelGGL(k_ln_quant<NJ>, grid, dim3(256), 0, s, x, rows, d, do_ln, g, b, eps, inv_s, q, x_out)
  switch (row_class(d)) {
    case 64: MNMT_LNQ(1); break;
    case 128: MNMT_LNQ(2); break;
    case 256: MNMT_LNQ(4); break;
    case 384: MNMT_LNQ(6); break;
    case 512: MNMT_LNQ(8); break;
    default: MNMT_LNQ(16); break;
  }
#undef MNMT_LNQ
  return hipGetLastError();
}

hipError_t launch_resid_ln_quant(float* x, int rows, int d, const ResidUpdate& u, int do_ln, const float* g,
                                 const float* b, float eps, float inv_s, int8_t* q, bool post, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d > kMaxRowLen || u.splits < 1 || u.splits > kMaxSplits || !q) return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4);
#define MNMT_RLNQ(NJ)                                                                                         \
  hipLaunchKernelGGL(k_resid_ln_quant<NJ>, grid, dim3(256), 0, s, x, rows, d, u, do_ln, g, b, eps, inv_s, q, \
                     post ? 1 : 0)
  switch (row_class(d)) {
    case 64: MNMT_RLNQ(1); break;
    case 128: MNMT_RLNQ(2); break;
    case 256: MNMT_RLNQ(4); break;
    case 384: MNMT_RLNQ(6); break;
    case 512: MNMT_RLNQ(8); break;
    default: MNMT_RLNQ(16); break;
  }
#undef MNMT_RLNQ
  return hipGetLastError();
}

// Key-length class of the attention kernels (the LDS and registers they
// reserve), head-width class.
int attn_len_class(int n) { return n <= 64 ? 64 : n <= 128 ? 128 : 256; }
int attn_dh_class(int dh) { return dh <= 64 ? 64 : 128; }

template <int WAVES, int QF = 0, int KQ = 1>
hipError_t launch_shared(const SharedAttn& a, int groups, int h, hipStream_t s) {
  const dim3 grid(h, groups);
  const int nm = attn_len_class(a.S), dm = attn_dh_class(a.dh);
#define MNMT_SH(NM, DM) \
  hipLaunchKernelGGL((k_attn_shared<NM, DM, WAVES, QF, KQ>), grid, dim3(64 * WAVES), 0, s, a)
  if (dm == 64) {
    if (nm == 64) MNMT_SH(64, 64);
    else if (nm == 128) MNMT_SH(128, 64);
    else MNMT_SH(256, 64);
  } else {
    if (nm == 64) MNMT_SH(64, 128);
    else if (nm == 128) MNMT_SH(128, 128);
    else MNMT_SH(256, 128);
  }
#undef MNMT_SH
  return hipGetLastError();
}

hipError_t launch_attn_enc(const int8_t* qkv, const int32_t* len, int B, int S, int d, int h, float c_qk, float c_pv,
                           int8_t* ctx, hipStream_t s) {
  const int dh = d / h;
  if (S > kMaxAttnLen || dh > kMaxHeadDim || dh % 16 || B < 1 || S < 1) return hipErrorInvalidValue;
  SharedAttn a{};
  a.q = qkv;
  a.ldq = 3 * d;
  a.rows = S;
  a.kv = qkv;
  a.kv_group = (size_t)S * 3 * d;
  a.ldkv = 3 * d;
  a.k_off = d;
  a.v_off = 2 * d;
  a.len = len;
  a.S = S;
  a.d = d;
  a.dh = dh;
  a.c_qk = c_qk;
  a.c_pv = c_pv;
  a.ctx = ctx;
  return launch_shared<8>(a, B, h, s);
}

hipError_t launch_attn_dec_self(const int8_t* qkv, int R, int d, int h, int T, const int* step, int8_t* kcache,
                                int8_t* vcache, const int32_t* hist, float c_qk, float c_pv, int8_t* ctx,
                                hipStream_t s, int t_host) {
  const int dh = d / h;
  if (T > kMaxAttnLen || dh > kMaxHeadDim || dh % 16 || R < 1) return hipErrorInvalidValue;
  const int nm = attn_len_class(T), dm = attn_dh_class(dh);
  // a block per row, a wave per head (up to 8, fewer for the widest LDS)
#define MNMT_SELF(NM, DM, WV)                                                                                      \
  hipLaunchKernelGGL((k_attn_dec_self<NM, DM, WV>), dim3(R), dim3(64 * WV), 0, s, qkv, d, h, dh, T, step, kcache, \
                     vcache, hist, c_qk, c_pv, ctx, t_host)
#define MNMT_SELF_W(NM, DM)                  \
  if (h >= 8) MNMT_SELF(NM, DM, 8);         \
  else if (h >= 4) MNMT_SELF(NM, DM, 4);    \
  else if (h >= 2) MNMT_SELF(NM, DM, 2);    \
  else MNMT_SELF(NM, DM, 1);
  if (dm == 64) {
    if (nm == 64) { MNMT_SELF_W(64, 64) }
    else if (nm == 128) { MNMT_SELF_W(128, 64) }
    else if (h >= 4) MNMT_SELF(256, 64, 4);
    else if (h >= 2) MNMT_SELF(256, 64, 2);
    else MNMT_SELF(256, 64, 1);
  } else {
    if (nm == 64) { MNMT_SELF_W(64, 128) }
    else if (nm == 128) MNMT_SELF(128, 128, 2);
    else if (h >= 2) MNMT_SELF(256, 128, 2);
    else MNMT_SELF(256, 128, 1);
  }
#undef MNMT_SELF_W
#undef MNMT_SELF
  return hipGetLastError();
}

// d 256 only: at d 512 (the base model) each of the head x sentence blocks
// loads 32 KB of the Q weights and the batch time did not move (34.4 against
// 34.6 ms), so the separate Q projection stays.
bool attn_cross_q_fits(int W, int d) { return W >= 1 && W <= 16 && d == 256; }

hipError_t launch_attn_dec_cross_q(const int8_t* rows, const FusedIn* ln, const int8_t* wq, const float* q_scale,
                                   const float* q_bias, bool w4, int R, int W, int d, int h, const int8_t* kv, int S,
                                   const int32_t* len, float c_qk, float c_pv, int8_t* ctx, hipStream_t s) {
  const int dh = d / h;
  if (S > kMaxAttnLen || dh > kMaxHeadDim || dh % 16 || R % W || !attn_cross_q_fits(W, d) || !wq ||
      (ln ? !ln->x || ln->embed || ln->x_out : !rows))
    return hipErrorInvalidValue;
  SharedAttn a{};
  a.a = rows;
  if (ln) {
    a.ln_on = 1;
    a.ln = *ln;
  }
  a.wq = wq;
  a.q_scale = q_scale;
  a.q_bias = q_bias;
  a.rows = W;
  a.kv = kv;
  a.kv_group = (size_t)S * 2 * d;
  a.ldkv = 2 * d;
  a.k_off = 0;
  a.v_off = d;
  a.len = len;
  a.S = S;
  a.d = d;
  a.dh = dh;
  a.c_qk = c_qk;
  a.c_pv = c_pv;
  a.ctx = ctx;
  return w4 ? launch_shared<4, 2, 4>(a, R / W, h, s) : launch_shared<4, 1, 4>(a, R / W, h, s);
}

bool attn_self_qkv_fits(int W, int d, int h, int T) {
  const int dh = h > 0 ? d / h : 0;
  return W >= 1 && W <= 16 && (d == 128 || d == 256) && h * dh == d && dh >= 16 && dh <= 64 && dh % 16 == 0 &&
         T >= 1 && T <= kMaxAttnLen;
}

hipError_t launch_attn_self_qkv(const int8_t* rows, const FusedIn* ln, const int8_t* wqkv, const float* scale,
                                const float* bias, bool w4, int R, int W, int d, int h, int T, const int* step,
                                int8_t* kcache, int8_t* vcache, const int32_t* hist, float c_qk, float c_pv,
                                int8_t* ctx, hipStream_t s, int t_host) {
  if (!attn_self_qkv_fits(W, d, h, T) || R % W || !wqkv || !kcache || !vcache || !ctx ||
      (ln ? !ln->x || ln->embed || (ln->x_out && (!ln->wb_input || ln->x_out == ln->x)) ||
                (ln->nparts && (ln->nparts > kMaxSplits || !ln->part || !ln->x_out))
          : !rows))
    return hipErrorInvalidValue;
  SelfQkvAttn a{};
  a.a = rows;
  if (ln) {
    a.ln_on = 1;
    a.ln = *ln;
  }
  a.wqkv = wqkv;
  a.scale = scale;
  a.bias = bias;
  // one sentence per block: 16-row groups (four mobile sentences) measured
  // 7.73 against 6.90 ms per mobile beam batch, a quarter of the blocks each
  // attending for four rows per wave.  At d 512 (the base model) the fused
  // form lost to the separate projection with either grouping (37.4-37.6
  // against 34.1 ms per batch): each block reads a 96 KB slice of W_qkv.
  const int rb = W;
  a.RB = rb;
  a.R = R;
  a.dh = d / h;
  a.T = T;
  a.step = step;
  a.t_host = t_host;
  a.kcache = kcache;
  a.vcache = vcache;
  a.hist = hist;
  a.c_qk = c_qk;
  a.c_pv = c_pv;
  a.ctx = ctx;
  const dim3 grid(h, (R + rb - 1) / rb);
  const int nm = attn_len_class(T);
#define MNMT_SQ(NM, KQ)                                                          \
  if (w4)                                                                        \
    hipLaunchKernelGGL((k_attn_self_qkv<NM, KQ, true>), grid, dim3(256), 0, s, a); \
  else                                                                           \
    hipLaunchKernelGGL((k_attn_self_qkv<NM, KQ, false>), grid, dim3(256), 0, s, a);
#define MNMT_SQ_K(NM) \
  if (d == 128) {     \
    MNMT_SQ(NM, 2)    \
  } else {            \
    MNMT_SQ(NM, 4)    \
  }
  if (nm == 64) {
    MNMT_SQ_K(64)
  } else if (nm == 128) {
    MNMT_SQ_K(128)
  } else {
    MNMT_SQ_K(256)
  }
#undef MNMT_SQ_K
#undef MNMT_SQ
  return hipGetLastError();
}

hipError_t launch_attn_dec_cross(const int8_t* q, int R, int W, int d, int h, const int8_t* kv, int S,
                                 const int32_t* len, float c_qk, float c_pv, int8_t* ctx, hipStream_t s) {
  const int dh = d / h;
  if (S > kMaxAttnLen || dh > kMaxHeadDim || dh % 16 || W < 1 || R % W) return hipErrorInvalidValue;
  SharedAttn a{};
  a.q = q;
  a.ldq = d;
  a.rows = W;
  a.kv = kv;
  a.kv_group = (size_t)S * 2 * d;
  a.ldkv = 2 * d;
  a.k_off = 0;
  a.v_off = d;
  a.len = len;
  a.S = S;
  a.d = d;
  a.dh = dh;
  a.c_qk = c_qk;
  a.c_pv = c_pv;
  a.ctx = ctx;
  return launch_shared<4>(a, R / W, h, s);
}

hipError_t launch_greedy_reset(unsigned long long* slots, int R, int steps, int32_t* cur_tok, int32_t* finished,
                               int32_t* out_len, int* step, int bos, unsigned long long* fslots, int n_fslots,
                               unsigned* epoch, hipStream_t s) {
  hipLaunchKernelGGL(k_greedy_reset, dim3(1), dim3(256), 0, s, slots, R, steps, cur_tok, finished, out_len, step,
                     bos, fslots, n_fslots, epoch);
  return hipGetLastError();
}

hipError_t launch_greedy_commit(unsigned long long* slots, int R, int T, int32_t* cur_tok, int32_t* out_tok,
                                int32_t* finished, int32_t* out_len, int* step, int stop_at_eos, int eos, int pad,
                                unsigned long long* out_key, hipStream_t s) {
  hipLaunchKernelGGL(k_greedy_commit, dim3(1), dim3(256), 0, s, slots, R, T, cur_tok, out_tok, finished, out_len,
                     step, stop_at_eos, eos, pad, out_key);
  return hipGetLastError();
}

hipError_t launch_greedy_output(const int32_t* out_tok, const int32_t* out_len, int R, int T, int32_t* out,
                                int32_t* out_len_dst, const int* chain_err, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_greedy_output, dim3(R), dim3(64), 0, s, out_tok, out_len, R, T, out, out_len_dst, chain_err);
  return hipGetLastError();
}

hipError_t launch_fill_lp(const LpTable& tab, float* dst, hipStream_t s) {
  if (tab.n < 1 || tab.n > LpTable::kMax) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_fill_lp, dim3(1), dim3(256), 0, s, tab, dst);
  return hipGetLastError();
}

hipError_t launch_row_argmax(const float* z, int R, int V, unsigned long long* slots, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_row_argmax, dim3((R + 3) / 4), dim3(256), 0, s, z, R, V, slots);
  return hipGetLastError();
}

hipError_t launch_load_batch(const int32_t* src_in, const int32_t* len_in, int32_t* src, int32_t* len, int n_src,
                             int n_len, unsigned* zero, int n_zero, hipStream_t s) {
  const int n = max(max(n_src, n_len), n_zero);
  const int blocks = min(256, max(1, (n + 255) / 256));
  hipLaunchKernelGGL(k_load_batch, dim3(blocks), dim3(256), 0, s, src_in, len_in, src, len, n_src, n_len, zero, n_zero);
  return hipGetLastError();
}

size_t frag_bytes(int N, int K) { return N < 1 || K < 64 || K % 64 ? 0 : (size_t)((N + 15) / 16) * 16 * K; }

hipError_t launch_pack_fragments(const int8_t* W, int N, int K, int8_t* out, hipStream_t s) {
  const size_t bytes = frag_bytes(N, K);
  if (!bytes || !W || !out || reinterpret_cast<uintptr_t>(W) % 16 || reinterpret_cast<uintptr_t>(out) % 16)
    return hipErrorInvalidValue;
  const size_t chunks = bytes / 16;
  hipLaunchKernelGGL(k_pack_fragments, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s, W, N, K, chunks, out);
  return hipGetLastError();
}

hipError_t launch_copy_i32(const int32_t* src, int32_t* dst, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_i32, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_beam_reset(const BeamState& st, int* step, hipStream_t s) {
  const size_t RT = (size_t)st.B * st.W * st.T;
  const size_t nb = (RT + 255) / 256;
  const int blocks = nb < 1 ? 1 : (nb > 1024 ? 1024 : (int)nb);
  hipLaunchKernelGGL(k_beam_reset, dim3(blocks), dim3(256), 0, s, st, step);
  return hipGetLastError();
}

hipError_t launch_beam_topk(const float* logits, const BeamState& st, const int* step, hipStream_t s) {
  const int R = st.B * st.W;
  if (st.V <= kTopkMaxV && st.V % 4 == 0) {
#define MNMT_TOPK(K) hipLaunchKernelGGL(k_beam_topk_block<K>, dim3(R), dim3(kTopkThreads), 0, s, logits, st, step)
    switch (2 * st.W) {
      case 2: MNMT_TOPK(2); break;
      case 4: MNMT_TOPK(4); break;
      case 6: MNMT_TOPK(6); break;
      case 8: MNMT_TOPK(8); break;
      case 10: MNMT_TOPK(10); break;
      case 12: MNMT_TOPK(12); break;
      case 14: MNMT_TOPK(14); break;
      case 16: MNMT_TOPK(16); break;
      default: return hipErrorInvalidValue;
    }
#undef MNMT_TOPK
    return hipGetLastError();
  }
  switch (2 * st.W) {
    case 2: hipLaunchKernelGGL(k_beam_topk<2>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 4: hipLaunchKernelGGL(k_beam_topk<4>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 6: hipLaunchKernelGGL(k_beam_topk<6>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 8: hipLaunchKernelGGL(k_beam_topk<8>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 10: hipLaunchKernelGGL(k_beam_topk<10>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 12: hipLaunchKernelGGL(k_beam_topk<12>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 14: hipLaunchKernelGGL(k_beam_topk<14>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    case 16: hipLaunchKernelGGL(k_beam_topk<16>, dim3(R), dim3(64), 0, s, logits, st, step); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_beam_update(const BeamState& st, int* step, const BeamNext& nx, hipStream_t s) {
  if (st.W > 8 || nx.d < 1 || nx.d > kMaxRowLen || !nx.x || !nx.a || !st.count) return hipErrorInvalidValue;
  const dim3 grid(st.B), block(64 * kUpdWaves);
#define MNMT_UPD(NJ) hipLaunchKernelGGL((k_beam_update<8, NJ>), grid, block, 0, s, st, step, nx)
  switch (row_class(nx.d)) {
    case 64: MNMT_UPD(1); break;
    case 128: MNMT_UPD(2); break;
    case 256: MNMT_UPD(4); break;
    case 384: MNMT_UPD(6); break;
    case 512: MNMT_UPD(8); break;
    default: MNMT_UPD(16); break;
  }
#undef MNMT_UPD
  return hipGetLastError();
}

hipError_t launch_beam_finalize(const BeamState& st, int steps, int32_t* out, int32_t* out_len, float* out_score,
                                const int* chain_err, hipStream_t s) {
  if (steps < 0 || steps > kFinMaxSteps || st.W < 1 || st.W > kFinMaxW) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_beam_finalize, dim3(st.B), dim3(64), 0, s, st, steps, out, out_len, out_score, chain_err);
  return hipGetLastError();
}

hipError_t launch_debug_read(const void* x, size_t bytes, int reps, unsigned* sink, hipStream_t s) {
  if (bytes == 0 || reps < 1) return hipSuccess;
  hipLaunchKernelGGL(k_debug_read, dim3(kDebugReadBlocks), dim3(256), 0, s, static_cast<const uint4*>(x), bytes / 16,
                     reps, sink);
  return hipGetLastError();
}

hipError_t launch_debug_canon(int fn, const float* x, int n, float* y, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (fn < 0 || fn > 2) return hipErrorInvalidValue;
  const int blocks = (fn == 2) ? 1 : (n + 255) / 256 > 1024 ? 1024 : (n + 255) / 256;
  hipLaunchKernelGGL(k_debug_canon, dim3(blocks), dim3(256), 0, s, fn, x, n, y);
  return hipGetLastError();
}

}  // namespace mnmt
