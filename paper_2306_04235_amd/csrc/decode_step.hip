// decode_step.hip -- the decoder step for at most 2 rows (the batch-1 latency
// path) in 3 block roles per decoder layer plus the output projection and the
// commit, instead of one kernel per operation.  The roles run as one launch
// per layer (k_step_layer) or as three kernels:
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
//
// At one or two rows every kernel is bound by memory latency, not bandwidth,
// so each one issues all of its global loads (rows, parameters, weights, the
// attention keys and values) before it waits for the first of them: the
// kernel then pays about one memory round trip instead of one per phase.
#include <hip/hip_ext.h>

#include "blocks.hpp"
#include "chain.hpp"
#include "internal.h"

namespace mnmt {
namespace {

constexpr int kStepRows = 2;     // rows (greedy batch) of this path
constexpr int kStepMaxLen = 128; // longest self / cross attention
constexpr int kStepHeadDim = 64; // widest head
constexpr int kFfnChunk = 64;    // hidden units per k_step_ffn block


// What the wave preparing one input row loads at kernel start.
template <int NJ>
struct RowRegs {
  float x[NJ];   // residual row
  int a[NJ];     // pending accumulator
  float sc[NJ];  // pending update scale and bias
  float bi[NJ];
  float g[NJ];   // the LayerNorm's gain and bias
  float b[NJ];
};

// The loads of input row r (element i = lane + 64 j in slot j; slots past d
// repeat element d - 1 and are never used), in two parts: the constants
// (model parameters, issued before a chain wait together with the weights)
// and the row data (written by the previous kernel, issued after it).  No
// load is conditional on a lane: a branch around a load makes the compiler
// wait for it where the branches join, which would serialize the kernel's
// memory round trips.
template <int NJ>
__device__ __forceinline__ void load_row_consts(const StepIn& in, int d, RowRegs<NJ>& q) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = min(lane + 64 * j, d - 1);
    q.sc[j] = in.scale[i];
    q.bi[j] = in.bias[i];
    q.g[j] = in.ln_g[i];
    q.b[j] = in.ln_b[i];
  }
}

template <int NJ>
__device__ __forceinline__ void load_row_data(const StepIn& in, int r, int d, RowRegs<NJ>& q) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = min(lane + 64 * j, d - 1);
    q.x[j] = in.x_in[(size_t)r * d + i];
    q.a[j] = (int)(unsigned)in.acc[(size_t)r * d + i];  // the sum's low half (StepCount)
  }
}

// Counted hand-off (StepCount) words: relaxed agent-scope 64-bit atomics.
__device__ __forceinline__ unsigned long long count_load(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void tag_store(unsigned long long* p, unsigned tag, unsigned bits) {
  __hip_atomic_store(p, ((unsigned long long)tag << 32) | bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// One block's int32 partial sum into a counted word: the value (mod 2^32)
// plus one count.
__device__ __forceinline__ void count_add(unsigned long long* p, int v) {
  atomicAdd(p, (unsigned long long)(unsigned)v + kCountUnit);
}

// Row r from the previous kernel through the counted hand-off: lane l polls
// its elements' tagged row words and counted sums until every tag is `want`
// and every count in.cnt.count_in, which leaves the row and the exact sums
// in q.  Bounded like chain_wait: a poll that gives up records it in *err.
template <int NJ>
__device__ __forceinline__ void poll_row_data(const StepIn& in, int r, int d, RowRegs<NJ>& q, unsigned want) {
  const int lane = threadIdx.x & 63;
  const unsigned long long need = (unsigned long long)in.cnt.count_in;
  unsigned spins = 0;
  while (true) {
    bool ok = true;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = min(lane + 64 * j, d - 1);
      const unsigned long long wx = count_load(in.cnt.x_in64 + (size_t)r * d + i);
      const unsigned long long wa = count_load(in.acc + (size_t)r * d + i);
      ok &= (unsigned)(wx >> 32) == want && (wa >> 40) == need;
      q.x[j] = __uint_as_float((unsigned)wx);
      q.a[j] = (int)(unsigned)wa;
    }
    if (ok) break;
    if (++spins >= kChainSpinLimit) {
      if (in.chain.err) __hip_atomic_fetch_or(in.chain.err, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Every load the kernel has issued (weights, constants, the input rows)
// completes here, in every wave, before block 0 issues its first store: the
// memory counter retires in order, so a wait for one of those loads placed
// after the stores would also wait for the stores to reach the point of
// coherence (about half a microsecond), and block 0, whose partial sums the
// next kernel also waits for, would lag the other blocks by that much.
__device__ __forceinline__ void loads_done() { __builtin_amdgcn_s_waitcnt(0); }

// The arg-max partials of the previous step's logits kernel (lane i: slots
// i + 64 k, clamped to the n written ones) once every one carries `want`
// (tagged keys); bounded like chain_wait.
__device__ __forceinline__ void poll_partials(const unsigned long long* sl, int n, unsigned want, int* err,
                                              unsigned long long (&pk)[4]) {
  const int lane = threadIdx.x & 63;
  unsigned spins = 0;
  while (true) {
    bool ok = true;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      pk[k] = count_load(sl + min(lane + 64 * k, n - 1));
      ok &= key_tag(pk[k]) == want;
    }
    if (__all(ok)) break;
    if (++spins >= kChainSpinLimit) {
      if (err) __hip_atomic_fetch_or(err, 4, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Finishes row r from the loaded registers: the pending residual update, the
// LayerNorm, the store of the updated residual row (block 0: plain, or tagged
// with out_tag for the counted hand-off), and the int8 codes in a_lds + r * d.
template <int NJ>
__device__ __forceinline__ void finish_row(const StepIn& in, int r, int d, RowRegs<NJ>& q, int8_t* a_lds,
                                           unsigned out_tag, int bid) {
  const int lane = threadIdx.x & 63;
  float v[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    v[j] = in.update ? fmaf(in.gamma, q.x[j], fmaf((float)q.a[j], q.sc[j], q.bi[j])) : q.x[j];
  if (in.ln_mode == 1) ln_row<NJ>(v, q.g, q.b, d, in.eps);  // post-LN: normalize the residual stream
  if (bid == 0 && in.x_out) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (i < d) chain_store(in.x_out + (size_t)r * d + i, v[j]);
    }
  }
  if (bid == 0 && in.cnt.x_out64) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = lane + 64 * j;
      if (i < d) tag_store(in.cnt.x_out64 + (size_t)r * d + i, out_tag, __float_as_uint(v[j]));
    }
  }
  if (in.ln_mode == 2) ln_row<NJ>(v, q.g, q.b, d, in.eps);  // pre-LN: normalize the sublayer input
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = lane + 64 * j;
    if (i < d) a_lds[r * d + i] = code_of(v[j] * in.inv_s);
  }
}

constexpr int kStepThreads = 256;  // block size of every step kernel

// (The loop stride is the compile-time block size: reading blockDim.x loads
// the dispatch packet and waits for every load issued before it.)
__device__ __forceinline__ void clear_acc(const StepIn& in, int bid) {
  if (bid == 0 && in.zero_acc)
    for (int i = threadIdx.x; i < in.zero_n; i += kStepThreads) chain_store(in.zero_acc + i, 0ull);
}

// Before block 0 adds its partial sums: its clear of an accumulator must have
// landed, since the next kernel's counted poll (not a flag stored after a
// full wait) is all that orders that accumulator's next producer after it.
__device__ __forceinline__ void clear_done(const StepIn& in, int bid) {
  if (bid == 0 && in.zero_acc) __builtin_amdgcn_s_waitcnt(0);
}

// The projections run on v_mfma_i32_16x16x64_i8 even though only R <= 2 of
// the 16 rows of its A operand are real: one matrix instruction yields 16
// complete output dot products in lanes 0..15 (D[m] = row m), where the
// vector form spends tens of instructions per 4 outputs on cross-lane
// reductions, and these kernels are bound by instruction issue, not by
// memory.  Fragment layout: lane l holds 16 bytes of K at 16 (l / 16) of
// row l % 16 (of the activations for A, of the weights for B).

// One block per head.  DMAX: model width class; NI: attended positions per
// lane (n <= 64 NI).  MODE 1 (self, layer 0): the input rows are the
// embeddings of the previous step's arg-max tokens, found from cm's partials;
// MODE 2 (cross, layer 0): block 0 records those tokens.
// The attention step of block `bid` (head bid); the kernel's chain signal is
// left to the caller.
template <int DMAX, bool SELF, int NI, int MODE, bool W4>
__device__ __forceinline__ void step_attn_body(const StepIn& in, const StepAttn& at, const StepCommit& cm, int bid) {
  constexpr int NJ = DMAX / 64;
  constexpr int KS = DMAX / 64;      // 64-deep K steps of the projection
  constexpr int TPW = SELF ? 3 : 1;  // 16-row projection tiles per wave (12 or 4 per head)
  constexpr int OT = DMAX / 64;      // 16-column W_o tiles per wave (d / 16 over 4 waves)
  constexpr int HC = kStepHeadDim / 16;
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kStepRows * DMAX];
  __shared__ __attribute__((aligned(16))) int8_t qkv[3][kStepRows][kStepHeadDim];
  __shared__ __attribute__((aligned(16))) int8_t ctx[kStepRows][kStepHeadDim];
  __shared__ AttnLdsT<64 * NI, kStepHeadDim> att[kStepRows];
  const int hd = bid;
  const int R = at.R, d = DMAX, dh = at.dh, nc = dh / 16, ks = d / 64;  // DMAX is the exact width
  const int ntile = (SELF ? 3 : 1) * dh / 16;  // projection tiles of this head
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, kq = lane >> 4;
  // 1. every global load, none conditional: the projection's weight
  //    fragments with their scales and biases, the W_o fragments, the keys
  //    and values (all written before the previous kernel started), then,
  //    after the chain wait, the wave's input row
  WFrag<W4> wf[TPW][KS];
  float e_sc[TPW], e_bi[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int j = 16 * min(wave + 4 * t, ntile - 1) + l16;  // row of the head's [q | k | v]
    const int part = (j >= dh) + (j >= 2 * dh);
    const size_t n = (size_t)part * d + hd * dh + (j - part * dh);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) wf[t][kk] = load_wfrag<W4>(at.W, n, d, 64 * min(kk, ks - 1) + 16 * kq);
    e_sc[t] = at.scale[n];
    e_bi[t] = at.bias[n];
  }
  WFrag<W4> of[OT];
#pragma unroll
  for (int t = 0; t < OT; ++t) {
    const int n = min(16 * (wave + 4 * t) + l16, d - 1);
    of[t] = load_wfrag<W4>(at.Wo, n, d, hd * dh + 16 * min(kq, nc - 1));
  }
  // keys and values of row r in registers: position lane + 64 i (self: the
  // cached positions before t; cross: every source position; positions at
  // or past n_load repeat position n_load - 1, or 0, and are not used)
  const int r = min(wave, R - 1);
  const int n_load = SELF ? at.t : at.S;
  const int8_t* kbase = SELF ? at.kcache + (size_t)r * at.T * d + hd * dh : at.kv + (size_t)r * at.S * 2 * d + hd * dh;
  const int8_t* vbase = SELF ? at.vcache + (size_t)r * at.T * d + hd * dh : kbase + d;
  const size_t pstride = SELF ? (size_t)d : (size_t)2 * d;
  v4i kr[NI][HC], vr[NI][HC];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const size_t p = (size_t)max(min(lane + 64 * i, n_load - 1), 0);
#pragma unroll
    for (int c = 0; c < HC; ++c) {
      const int off = 16 * min(c, nc - 1);
      kr[i][c] = *(const v4i*)(kbase + p * pstride + off);
      vr[i][c] = *(const v4i*)(vbase + p * pstride + off);
    }
  }
  int n_att = SELF ? at.t + 1 : at.len[r];
  n_att = SELF ? n_att : (n_att < 1 ? 1 : (n_att > at.S ? at.S : n_att));
  const unsigned ep = *in.cnt.epoch;  // row tags of the counted hand-off (StepCount)
  const unsigned want = ep * kTagSpan + in.cnt.tag_in, otag = ep * kTagSpan + in.cnt.tag_out;
  RowRegs<NJ> rr;
  if (MODE == 1) {
    // the position term now, the token's embedding once the token is known
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = min(lane + 64 * j, d - 1);
      rr.x[j] = cm.pe[(size_t)cm.t * d + i];
      rr.a[j] = 0;
      rr.sc[j] = 0.0f;
      rr.bi[j] = 0.0f;
      rr.g[j] = in.ln_g[i];
      rr.b[j] = in.ln_b[i];
    }
  } else {
    load_row_consts(in, d, rr);
  }
  asm volatile("" ::: "memory");  // the loads above stay ahead of the wait
  chain_wait(in.chain);
  // MODE 1 / 2: the arg-max partials of the wave's row (lane i: slots i + 64 k)
  // and whether the row had finished
  unsigned long long pk[4] = {0ull, 0ull, 0ull, 0ull};
  int fin = 0;
  if (MODE != 0) {
    const int row = min(wave, R - 1);
    const unsigned long long* sl = cm.slots + (size_t)row * cm.nslots;
    if (cm.tagged) {
      // no flag wait: the waves that use the partials poll them until every
      // one carries step t - 1's tag
      if (wave < R && (MODE == 1 || bid == 0)) {
        poll_partials(sl, cm.nparts, step_tag(ep, cm.t - 1), in.chain.err, pk);
        fin = __hip_atomic_load(cm.finished + row, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) pk[k] = sl[min(lane + 64 * k, cm.nslots - 1)];
      fin = cm.finished[row];
    }
  }
  if (MODE != 1) {
    if (in.cnt.count_in > 0) {
      if (wave < R) poll_row_data(in, wave, d, rr, want);
      lds_barrier();  // the accumulator clear below comes after every wave's poll
    } else {
      load_row_data(in, min(wave, R - 1), d, rr);
    }
  }
  if (MODE == 1) {
    unsigned long long key = pk[0];
#pragma unroll
    for (int k = 1; k < 4; ++k) key = pk[k] > key ? pk[k] : key;
    const unsigned long long kmax = wave_max_u64(key);
    const int tok = cm.tagged ? tagged_index(kmax) : unpack_index(kmax);
    // x = E[tok] c_emb[tok] + PE[t] (padding after the end of the sentence)
    int te = fin ? cm.pad : tok;
    te = te < 0 ? 0 : (te >= cm.V ? cm.V - 1 : te);
    const float ce = cm.c_emb[te];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = min(lane + 64 * j, d - 1);
      rr.x[j] = fmaf((float)cm.E[(size_t)te * d + i], ce, rr.x[j]);
    }
  }
  // 2. the rows
  // (the clear after the row: its stores must not sit in the in-order
  // memory counter ahead of the row data that finish_row waits for)
  loads_done();
  if (wave < R) finish_row(in, wave, d, rr, a_lds, otag, bid);
  clear_acc(in, bid);

  lds_barrier();
  // 3. Q (K, V) of the head on the matrix cores, requantized into LDS
  {
    const int arow = l16 < R ? l16 : 0;
    v4i af[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) af[kk] = *(const v4i*)(a_lds + arow * d + 64 * kk + 16 * kq);
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = wave + 4 * t;
      if (tile < ntile) {
        v4i acc = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
          if (kk < ks) acc = mfma16(af[kk], wf[t][kk].get(), acc);
        if (lane < 16) {
          const int j = 16 * tile + lane;
          const int part = (j >= dh) + (j >= 2 * dh);
#pragma unroll
          for (int m = 0; m < kStepRows; ++m)
            if (m < R) qkv[part][m][j - part * dh] = code_of(fmaf((float)acc[m], e_sc[t], e_bi[t]));
        }
      }
    }
  }
  lds_barrier();
  // 4. attention of row `wave` (Appendix A with the quantizer figure's
  //    precisions): int8 scores, fp32 softmax in the canonical order, context
  //    accumulated over ascending positions with one fma each, requantized
  if (wave < R) {
    AttnLdsT<64 * NI, kStepHeadDim>& sh = att[r];
    const int8_t* knew = qkv[1][r];
    const int8_t* vnew = qkv[2][r];
    if (SELF) {
      int8_t* kc = at.kcache + ((size_t)r * at.T + at.t) * d + hd * dh;
      int8_t* vc = at.vcache + ((size_t)r * at.T + at.t) * d + hd * dh;
      for (int j = lane; j < dh; j += 64) {
        chain_store(kc + j, knew[j]);
        chain_store(vc + j, vnew[j]);
      }
    }
    int4 qv[HC], kn[HC];
#pragma unroll
    for (int c = 0; c < HC; ++c) {
      qv[c] = c < nc ? *(const int4*)(qkv[0][r] + 16 * c) : make_int4(0, 0, 0, 0);
      kn[c] = c < nc ? *(const int4*)(knew + 16 * c) : make_int4(0, 0, 0, 0);
    }
    int s_new = 0;  // score of the position appended at this step
#pragma unroll
    for (int c = 0; c < HC; ++c) s_new = dot16(kn[c], qv[c], s_new);
    float sv[NI];
    float mx = -FLT_MAX;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int p = lane + 64 * i;
      sv[i] = 0.0f;
      if (p < n_att) {
        const bool cur = SELF && p == at.t;
        int acc = 0;
#pragma unroll
        for (int c = 0; c < HC; ++c) {
          const int4 kk = make_int4(kr[i][c].x, kr[i][c].y, kr[i][c].z, kr[i][c].w);
          acc = dot16(kk, qv[c], acc);
        }
        if (!cur)
#pragma unroll
          for (int c = 0; c < HC; ++c)
            if (c < nc) *(v4i*)&sh.v[p][16 * c] = vr[i][c];
        sv[i] = (float)(cur ? s_new : acc) * at.c_qk;
        mx = fmaxf(mx, sv[i]);
      }
    }
    if (SELF)
      for (int j = lane; j < dh; j += 64) sh.v[at.t][j] = vnew[j];
    mx = wave_max(mx);
    float part = 0.0f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      if (lane + 64 * i < n_att) {
        sv[i] = canon_exp(sv[i] - mx);
        part = part + sv[i];
      }
    }
    const float inv = 1.0f / wave_sum(part);
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (lane + 64 * i < n_att) sh.p[lane + 64 * i] = sv[i] * inv;
    wave_sync();  // p and v visible to every lane of this wave
    for (int j = lane; j < dh; j += 64) {
      float acc = 0.0f;
      int p = 0;
      for (; p + 4 <= n_att; p += 4) {
        const float p0 = sh.p[p], p1 = sh.p[p + 1], p2 = sh.p[p + 2], p3 = sh.p[p + 3];
        const float v0 = sh.v[p][j], v1 = sh.v[p + 1][j], v2 = sh.v[p + 2][j], v3 = sh.v[p + 3][j];
        acc = fmaf(p0, v0, acc);
        acc = fmaf(p1, v1, acc);
        acc = fmaf(p2, v2, acc);
        acc = fmaf(p3, v3, acc);
      }
      for (; p < n_att; ++p) acc = fmaf(sh.p[p], (float)sh.v[p][j], acc);
      ctx[r][j] = code_of(acc * at.c_pv);
    }
  }
  lds_barrier();
  // 5. this head's share of the output projection (K = dh), exact int32
  //    partial sums added to the accumulator
  // Block 0: its accumulator clear must have landed before it adds (see
  // clear_done).  Self-attention blocks: their key/value appends must have
  // landed before their partial sums, which the rest of the step waits on:
  // this layer's launch of the next step reads the cache before its own wait
  // and starts only once the launch after this one has finished, which
  // cannot finish before these sums have landed.
  if (SELF) __builtin_amdgcn_s_waitcnt(0);
  else clear_done(in, bid);
  {
    const int crow = l16 < R ? l16 : 0;
    const v4i cf = kq < nc ? *(const v4i*)(ctx[crow] + 16 * kq) : v4i{0, 0, 0, 0};
#pragma unroll
    for (int t = 0; t < OT; ++t) {
      const int n0 = 16 * (wave + 4 * t);
      if (n0 < d) {
        const v4i acc = mfma16(cf, of[t].get(), v4i{0, 0, 0, 0});
        if (lane < 16)
#pragma unroll
          for (int m = 0; m < kStepRows; ++m)
            if (m < R) count_add(at.acc_out + (size_t)m * d + n0 + lane, acc[m]);
      }
    }
  }
  if (MODE == 2 && bid == 0) {
    // step t - 1's token (off the critical path, at the end): output, end of
    // sentence, current token, step counter
    unsigned long long key = pk[0];
#pragma unroll
    for (int k = 1; k < 4; ++k) key = pk[k] > key ? pk[k] : key;
    const unsigned long long kmax = wave_max_u64(key);
    const unsigned long long best = cm.tagged ? untag_key(kmax) : kmax;
    const int tok = unpack_index(best);
    if (wave < R && lane == 0) {
      const int tc = cm.t - 1;
      if (tc < cm.T) chain_store(cm.out_tok + (size_t)tc * R + wave, fin ? cm.pad : tok);
      if (cm.out_key && tc < cm.T) cm.out_key[(size_t)tc * R + wave] = best;
      if (!fin && cm.stop_at_eos && tok == cm.eos) {
        chain_store(cm.finished + wave, 1);
        chain_store(cm.out_len + wave, tc + 1);
      }
      chain_store(cm.cur_tok + wave, fin ? cm.pad : tok);
      if (wave == 0) chain_store(cm.step, cm.t);
    }
  }
}

template <int DMAX, bool SELF, int NI, int MODE, bool W4>
__global__ __launch_bounds__(kStepThreads) void k_step_attn(StepIn in, StepAttn at, StepCommit cm) {
  step_attn_body<DMAX, SELF, NI, MODE, W4>(in, at, cm, blockIdx.x);
  chain_signal(in.chain);
}

// One block per kFfnChunk hidden units (one 16-row W1 tile per wave): ReLU
// requantization of the chunk, then the chunk's W2 columns (K = 64) into the
// int32 accumulator.
template <int DMAX, bool W4>
__device__ __forceinline__ void step_ffn_body(const StepIn& in, const StepFfn& f, int bid) {
  constexpr int NJ = DMAX / 64;
  constexpr int KS = DMAX / 64;
  constexpr int OT = DMAX / 64;
  static_assert(kFfnChunk == 64, "one W1 tile per wave and one K step of W2");
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kStepRows * DMAX];
  __shared__ __attribute__((aligned(16))) int8_t h[kStepRows][kFfnChunk];
  const int R = f.R, d = DMAX, F = f.F, ks = d / 64;  // DMAX is the exact width
  const int f0 = bid * kFfnChunk;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, kq = lane >> 4;
  const size_t hrow = (size_t)min(f0 + 16 * wave + l16, F - 1);
  WFrag<W4> wf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) wf[kk] = load_wfrag<W4>(f.W1, hrow, d, 64 * min(kk, ks - 1) + 16 * kq);
  const float e_sc = f.scale1[hrow], e_bi = f.bias1[hrow];
  WFrag<W4> of[OT];
#pragma unroll
  for (int t = 0; t < OT; ++t) {
    const int n = min(16 * (wave + 4 * t) + l16, d - 1);
    of[t] = load_wfrag<W4>(f.W2, n, F, f0 + 16 * kq);
  }
  const unsigned ep = *in.cnt.epoch;  // row tags of the counted hand-off (StepCount)
  const unsigned want = ep * kTagSpan + in.cnt.tag_in, otag = ep * kTagSpan + in.cnt.tag_out;
  RowRegs<NJ> rr;
  load_row_consts(in, d, rr);
  asm volatile("" ::: "memory");  // the weight loads stay ahead of the wait
  chain_wait(in.chain);
  if (in.cnt.count_in > 0) {
    if (wave < R) poll_row_data(in, wave, d, rr, want);
    lds_barrier();  // the accumulator clear below comes after every wave's poll
  } else {
    load_row_data(in, min(wave, R - 1), d, rr);
  }
  // (the clear after the row: its stores must not sit in the in-order
  // memory counter ahead of the row data that finish_row waits for)
  loads_done();
  if (wave < R) finish_row(in, wave, d, rr, a_lds, otag, bid);
  clear_acc(in, bid);
  lds_barrier();
  {
    const int arow = l16 < R ? l16 : 0;
    v4i acc = {0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      if (kk < ks) acc = mfma16(*(const v4i*)(a_lds + arow * d + 64 * kk + 16 * kq), wf[kk].get(), acc);
    if (lane < 16)
#pragma unroll
      for (int m = 0; m < kStepRows; ++m)
        if (m < R) h[m][16 * wave + lane] = code_of(fmaxf(fmaf((float)acc[m], e_sc, e_bi), 0.0f));
  }
  lds_barrier();
  clear_done(in, bid);
  {
    const int hr = l16 < R ? l16 : 0;
    const v4i hf = *(const v4i*)(h[hr] + 16 * kq);
#pragma unroll
    for (int t = 0; t < OT; ++t) {
      const int n0 = 16 * (wave + 4 * t);
      if (n0 < d) {
        const v4i acc = mfma16(hf, of[t].get(), v4i{0, 0, 0, 0});
        if (lane < 16)
#pragma unroll
          for (int m = 0; m < kStepRows; ++m)
            if (m < R) count_add(f.acc_out + (size_t)m * d + n0 + lane, acc[m]);
      }
    }
  }
}

template <int DMAX, bool W4>
__global__ __launch_bounds__(kStepThreads) void k_step_ffn(StepIn in, StepFfn f) {
  step_ffn_body<DMAX, W4>(in, f, blockIdx.x);
  chain_signal(in.chain);
}

// One decoder layer of the step in one launch: blocks [0, heads) run the
// self-attention step (head = block), blocks [heads, 2 heads) the
// cross-attention step, the rest the FFN chunks; the phases hand off through
// the counted words inside the launch, exactly as separate kernels would.  A
// layer costs one kernel node instead of three (the decode graph shrinks by
// two thirds).  FOLD: the first layer of a folded step (the self-attention
// blocks embed the previous step's token, the first cross-attention block
// records it).
// Block b of a decoder layer's launch (or of its share of the step's
// launch): its role, then its flag (when the next role waits on flags).
template <int DMAX, int NIS, int NIC, bool FOLD, bool W4>
__device__ __forceinline__ void step_layer_body(const StepIn& ia, const StepAttn& sa, const StepIn& ib,
                                                const StepAttn& ca, const StepIn& ic, const StepFfn& f,
                                                const StepCommit& cm, int b, int nblk) {
  const int heads = sa.d / sa.dh;
  if (b < heads)
    step_attn_body<DMAX, true, NIS, FOLD ? 1 : 0, W4>(ia, sa, cm, b);
  else if (b < 2 * heads)
    step_attn_body<DMAX, false, NIC, FOLD ? 2 : 0, W4>(ib, ca, cm, b - heads);
  else
    step_ffn_body<DMAX, W4>(ic, f, b - 2 * heads);
  chain_signal_as(ic.chain, b, nblk);  // every block (when the next role waits on flags)
}

template <int DMAX, int NIS, int NIC, bool FOLD, bool W4>
__global__ __launch_bounds__(kStepThreads) void k_step_layer(StepIn ia, StepAttn sa, StepIn ib, StepAttn ca,
                                                             StepIn ic, StepFfn f, StepCommit cm) {
  step_layer_body<DMAX, NIS, NIC, FOLD, W4>(ia, sa, ib, ca, ic, f, cm, blockIdx.x, gridDim.x);
}

// Output projection over the shared embedding with the fused arg-max: each
// wave takes TPW tiles of 16 vocabulary rows (kLogitsTiles alone, more in a
// kernel chain, where the weights load while the previous kernel runs and
// fewer blocks mean fewer flags to store and to wait for).  RAW: the rows are
// int8 codes already (g.x_i8) instead of the residual stream.  FRAG: the
// embedding in fragment order (launch_pack_fragments), so that each of a
// wave's weight loads reads one contiguous kilobyte; row-major, each load
// gathers 64-byte pieces of 16 rows.
constexpr int kLogitsTiles = 2;
// in a chain: 4 tiles per wave once that still leaves about 100 blocks
__host__ inline int chain_logits_tiles(int V) { return V >= 4 * 4 * 16 * 96 ? 4 : kLogitsTiles; }
// bid / nblk: the block's index among the role's blocks and their number
// (the whole grid as a kernel of its own).
template <int DMAX, bool RAW, int TPW, bool FRAG>
__device__ __forceinline__ void step_logits_body(const StepIn& in, const StepLogits& g, int bid, int nblk) {
  constexpr int NJ = DMAX / 64;
  constexpr int KS = DMAX / 64;
  __shared__ __attribute__((aligned(16))) int8_t a_lds[kStepRows * DMAX];
  __shared__ unsigned long long wmax[4][kStepRows];
  const int R = g.R, d = DMAX, N = g.V, ks = d / 64;  // DMAX is the exact width
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, kq = lane >> 4;
  const int row0 = (bid * 4 + wave) * TPW * 16;
  v4i xr = {0, 0, 0, 0};
  if (RAW) xr = *(const v4i*)(g.x_i8 + (size_t)min(wave, R - 1) * d + 16 * min(lane, d / 16 - 1));
  v4i wf[TPW][KS];
  float co[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const size_t n = (size_t)min(row0 + 16 * t + l16, N - 1);
    const size_t tile = (size_t)min(row0 / 16 + t, (N - 1) / 16);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      if (FRAG) wf[t][kk] = *(const v4i*)(g.E + ((tile * KS + kk) * 64 + lane) * 16);
      else wf[t][kk] = *(const v4i*)(g.E + n * d + 64 * min(kk, ks - 1) + 16 * kq);
    }
    co[t] = g.c_out[n];
  }
  const unsigned tag = (!RAW && g.tagged) ? step_tag(*g.epoch, g.t) : 0u;
  RowRegs<NJ> rr;
  if (!RAW) {
    load_row_consts(in, d, rr);
    asm volatile("" ::: "memory");  // the weight loads stay ahead of the wait
    chain_wait(in.chain);
    load_row_data(in, min(wave, R - 1), d, rr);
  }
  if (!RAW) {
    loads_done();
    if (wave < R) finish_row(in, wave, d, rr, a_lds, 0u, bid);
    clear_acc(in, bid);
  } else if (wave < R && lane < d / 16) {
    *(v4i*)(a_lds + wave * d + 16 * lane) = xr;
  }
  lds_barrier();
  const int arow = l16 < R ? l16 : 0;
  v4i af[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) af[kk] = *(const v4i*)(a_lds + arow * d + 64 * kk + 16 * kq);
  unsigned long long best[kStepRows] = {0ull, 0ull};
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    v4i acc = {0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      if (kk < ks) acc = mfma16(af[kk], wf[t][kk], acc);
    const int n = row0 + 16 * t + lane;
    if (lane < 16 && n < N) {
#pragma unroll
      for (int m = 0; m < kStepRows; ++m) {
        if (m < R) {
          const float z = (float)acc[m] * co[t];
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
  // a tagged partial is the hand-off itself: block 0's accumulator clear
  // (every wave's share) must have landed before it is stored
  if (!RAW && g.tagged && bid == 0 && in.zero_acc) __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  if (threadIdx.x < R) {
    const int m = threadIdx.x;
    unsigned long long b = wmax[0][m];
#pragma unroll
    for (int w = 1; w < 4; ++w) b = wmax[w][m] > b ? wmax[w][m] : b;
    unsigned long long* slot = g.slots + (size_t)m * g.nslots;
    if (g.nslots >= nblk) {
      // one partial per block: a plain store, no atomic (atomics on one
      // address serialize), reduced by the consumer
      if (RAW) {
        slot[bid] = b;  // read after the launch, not by a chained kernel
      } else if (g.tagged) {
        chain_store(slot + bid, tagged_key(b, tag));
      } else {
        chain_store(slot + bid, b);
      }
    } else {
      // few slots: most blocks find a larger key already there, and the
      // test spares them the serialized atomic
      slot += bid % g.nslots;
      if (b > __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) atomicMax(slot, b);
    }
  }
  if (!RAW) chain_signal_as(in.chain, bid, nblk);
}

template <int DMAX, bool RAW, int TPW, bool FRAG>
__global__ __launch_bounds__(kStepThreads) void k_step_logits(StepIn in, StepLogits g) {
  step_logits_body<DMAX, RAW, TPW, FRAG>(in, g, blockIdx.x, gridDim.x);
}

// The whole decode step in one launch (two decoder layers, then the output
// projection with the fused arg-max): blocks [0, L) and [L, 2 L) run the two
// layers' roles (L = step_layer_blocks), the rest the logits kernel's blocks
// (4 tiles of 16 vocabulary rows per wave).  The hand-offs are the ones the
// separate launches use: counted words into each layer and between the
// layers, the last layer's flags for the logits blocks, tagged partials (or
// the logits blocks' flags) for the next step.  Every consumer role has
// higher block indices than its producers, and blocks are dispatched in
// index order, so producers never wait behind their consumers.
template <int DMAX, bool FOLD, bool W4>
__global__ __launch_bounds__(kStepThreads) void k_step_all(StepAll p) {
  const int L = p.layer_blocks;
  const int b = blockIdx.x;
  if (b < L)
    step_layer_body<DMAX, 1, 1, FOLD, W4>(p.ia[0], p.sa[0], p.ib[0], p.ca[0], p.ic[0], p.f[0], p.cm, b, L);
  else if (b < 2 * L)
    step_layer_body<DMAX, 1, 1, false, W4>(p.ia[1], p.sa[1], p.ib[1], p.ca[1], p.ic[1], p.f[1], StepCommit{}, b - L,
                                           L);
  else
    step_logits_body<DMAX, false, 4, true>(p.lin, p.g, b - 2 * L, (int)gridDim.x - 2 * L);
}

}  // namespace

bool step_path_fits(int R, int d, int dh, int F, int T, int S) {
  return R >= 1 && R <= kStepRows && d <= 512 && d % 64 == 0 && dh <= kStepHeadDim && dh % 16 == 0 &&
         F % kFfnChunk == 0 && T <= kStepMaxLen && S <= kStepMaxLen;
}

bool step_logits_fits(int R, int d) { return R >= 1 && R <= kStepRows && d % 64 == 0 && d >= 64 && d <= 512; }

int step_logits_blocks(int V) {
  const int rpb = 4 * kLogitsTiles * 16;  // rows per block
  return (V + rpb - 1) / rpb;
}

int step_logits_blocks_chained(int V, int d) {
  (void)d;
  const int rpb = 4 * chain_logits_tiles(V) * 16;
  return (V + rpb - 1) / rpb;
}

// Kernels are instantiated on the exact width (a multiple of 64 up to 512),
// so the row code carries no bounds checks.
#define MNMT_BY_D(d, CALL)            \
  switch (d) {                        \
    case 64: CALL(64); break;         \
    case 128: CALL(128); break;       \
    case 192: CALL(192); break;       \
    case 256: CALL(256); break;       \
    case 320: CALL(320); break;       \
    case 384: CALL(384); break;       \
    case 448: CALL(448); break;       \
    case 512: CALL(512); break;       \
    default: return hipErrorInvalidValue; \
  }

hipError_t launch_step_attn(const StepIn& in, const StepAttn& at, int self, int heads, hipStream_t s,
                            const StepCommit* cm) {
  // positions attended: self t + 1 <= T, cross at most S
  const int n_max = self ? at.t + 1 : at.S;
  if (cm && (cm->nslots < 1 || cm->nslots > 256 || cm->t < 1)) return hipErrorInvalidValue;
  if (!at.W || !at.Wo) return hipErrorInvalidValue;  // (a weight without the form this launch reads)
  const StepCommit c = cm ? *cm : StepCommit{};
#define MNMT_ATTN_W(DM, SELF, NI, W4)                                                                           \
  do {                                                                                                           \
    if (!cm)                                                                                                     \
      hipLaunchKernelGGL((k_step_attn<DM, SELF, NI, 0, W4>), dim3(heads), dim3(kStepThreads), 0, s, in, at, c); \
    else                                                                                                         \
      hipLaunchKernelGGL((k_step_attn<DM, SELF, NI, SELF ? 1 : 2, W4>), dim3(heads), dim3(kStepThreads), 0, s, in, \
                         at, c);                                                                                 \
  } while (0)
#define MNMT_ATTN_NI(DM, SELF, NI)             \
  do {                                         \
    if (at.w4) MNMT_ATTN_W(DM, SELF, NI, true);  \
    else MNMT_ATTN_W(DM, SELF, NI, false);       \
  } while (0)
#define MNMT_ATTN(DM)                                   \
  if (self) {                                           \
    if (n_max <= 64) MNMT_ATTN_NI(DM, true, 1);         \
    else MNMT_ATTN_NI(DM, true, 2);                     \
  } else {                                              \
    if (n_max <= 64) MNMT_ATTN_NI(DM, false, 1);        \
    else MNMT_ATTN_NI(DM, false, 2);                    \
  }
  MNMT_BY_D(at.d, MNMT_ATTN)
#undef MNMT_ATTN
#undef MNMT_ATTN_NI
#undef MNMT_ATTN_W
  return hipGetLastError();
}

int step_layer_blocks(int heads, int F) { return 2 * heads + F / kFfnChunk; }

hipError_t launch_step_layer(const StepIn& ia, const StepAttn& sa, const StepIn& ib, const StepAttn& ca,
                             const StepIn& ic, const StepFfn& f, hipStream_t s, const StepCommit* cm) {
  const int heads = sa.d / sa.dh;
  if (sa.w4 != ca.w4 || sa.w4 != f.w4) return hipErrorInvalidValue;  // one weight form per launch
  if (!sa.W || !sa.Wo || !ca.W || !ca.Wo || !f.W1 || !f.W2) return hipErrorInvalidValue;
  if (cm && (cm->nslots < 1 || cm->nslots > 256 || cm->t < 1)) return hipErrorInvalidValue;
  const StepCommit c = cm ? *cm : StepCommit{};
  const int blocks = step_layer_blocks(heads, f.F);
  const int ns = sa.t + 1 <= 64 ? 1 : 2, nc = ca.S <= 64 ? 1 : 2;
#define MNMT_LAYER_K(DM, NS, NC, FO, W)                                                                       \
  hipLaunchKernelGGL((k_step_layer<DM, NS, NC, FO, W>), dim3(blocks), dim3(kStepThreads), 0, s, ia, sa, ib, ca, \
                     ic, f, c)
#define MNMT_LAYER_W(DM, NS, NC, FO)               \
  if (sa.w4) MNMT_LAYER_K(DM, NS, NC, FO, true);   \
  else MNMT_LAYER_K(DM, NS, NC, FO, false);
#define MNMT_LAYER_F(DM, NS, NC)       \
  if (cm) {                            \
    MNMT_LAYER_W(DM, NS, NC, true)     \
  } else {                             \
    MNMT_LAYER_W(DM, NS, NC, false)    \
  }
#define MNMT_LAYER(DM)                                              \
  if (ns == 1 && nc == 1) {                                         \
    MNMT_LAYER_F(DM, 1, 1)                                          \
  } else if (ns == 1) {                                             \
    MNMT_LAYER_F(DM, 1, 2)                                          \
  } else if (nc == 1) {                                             \
    MNMT_LAYER_F(DM, 2, 1)                                          \
  } else {                                                          \
    MNMT_LAYER_F(DM, 2, 2)                                          \
  }
  MNMT_BY_D(sa.d, MNMT_LAYER)
#undef MNMT_LAYER
#undef MNMT_LAYER_F
#undef MNMT_LAYER_W
#undef MNMT_LAYER_K
  return hipGetLastError();
}

hipError_t launch_step_ffn(const StepIn& in, const StepFfn& f, hipStream_t s) {
  if (!f.W1 || !f.W2) return hipErrorInvalidValue;
  const int blocks = (f.F + kFfnChunk - 1) / kFfnChunk;
#define MNMT_FFN(DM)                                                                               \
  if (f.w4) hipLaunchKernelGGL((k_step_ffn<DM, true>), dim3(blocks), dim3(kStepThreads), 0, s, in, f); \
  else hipLaunchKernelGGL((k_step_ffn<DM, false>), dim3(blocks), dim3(kStepThreads), 0, s, in, f);
  MNMT_BY_D(f.d, MNMT_FFN)
#undef MNMT_FFN
  return hipGetLastError();
}

bool step_all_fits(int n_dec, int d, int heads, int F, int T, int S, int V) {
  return n_dec == 2 && d == 256 && d % heads == 0 && d / heads <= kStepHeadDim && F % kFfnChunk == 0 &&
         T <= 64 && S <= 64 && V <= kTagMaxV && chain_logits_tiles(V) == 4 &&
         step_layer_blocks(heads, F) <= kChainMaxBlocks && step_logits_blocks_chained(V, d) <= kChainMaxBlocks;
}

hipError_t launch_step_all(const StepAll& p, bool fold, hipStream_t s) {
  const int heads = p.sa[0].d / p.sa[0].dh;
  const bool w4 = p.sa[0].w4;
  for (int l = 0; l < 2; ++l)
    if (p.sa[l].w4 != w4 || p.ca[l].w4 != w4 || p.f[l].w4 != w4 || !p.sa[l].W || !p.ca[l].W || !p.f[l].W1)
      return hipErrorInvalidValue;
  if (p.layer_blocks != step_layer_blocks(heads, p.f[0].F) || p.f[1].F != p.f[0].F || !p.g.frag || !p.g.tagged ||
      !step_all_fits(2, p.g.d, heads, p.f[0].F, p.sa[0].t + 1, p.ca[0].S, p.g.V))
    return hipErrorInvalidValue;
  if (fold && (p.cm.nslots < 1 || p.cm.nslots > 256 || p.cm.t < 1)) return hipErrorInvalidValue;
  const int blocks = 2 * p.layer_blocks + step_logits_blocks_chained(p.g.V, p.g.d);
  if (chain_logits_tiles(p.g.V) != 4) return hipErrorInvalidValue;
#define MNMT_ALL(DM, FO, W) hipLaunchKernelGGL((k_step_all<DM, FO, W>), dim3(blocks), dim3(kStepThreads), 0, s, p)
#define MNMT_ALL_D(DM)                         \
  if (fold) {                                  \
    if (w4) MNMT_ALL(DM, true, true);          \
    else MNMT_ALL(DM, true, false);            \
  } else {                                     \
    if (w4) MNMT_ALL(DM, false, true);         \
    else MNMT_ALL(DM, false, false);           \
  }
  MNMT_ALL_D(256)
#undef MNMT_ALL_D
#undef MNMT_ALL
  return hipGetLastError();
}

hipError_t launch_step_logits(const StepIn& in, const StepLogits& g, hipStream_t s, hipEvent_t ev_start,
                              hipEvent_t ev_stop) {
  const int blocks = step_logits_blocks(g.V);
  const int cblocks = step_logits_blocks_chained(g.V, g.d);
  if (in.chain.done && g.nslots < cblocks) return hipErrorInvalidValue;
  // tagged partials: the chained grid (whose block count the consumers poll)
  if (g.tagged && (!in.chain.done || g.V > kTagMaxV || !g.epoch)) return hipErrorInvalidValue;
  if (!g.x_i8 && !g.frag) return hipErrorInvalidValue;  // the decoder reads the fragment-order copy
#define MNMT_RAW(DM, FR)                                                                                          \
  if (ev_start || ev_stop)                                                                                        \
    hipExtLaunchKernelGGL((k_step_logits<DM, true, kLogitsTiles, FR>), dim3(blocks), dim3(kStepThreads), 0, s,    \
                          ev_start, ev_stop, 0, in, g);                                                           \
  else                                                                                                            \
    hipLaunchKernelGGL((k_step_logits<DM, true, kLogitsTiles, FR>), dim3(blocks), dim3(kStepThreads), 0, s, in, g);
#define MNMT_LOGITS(DM)                                                                                         \
  if (g.x_i8 && g.frag) {                                                                                       \
    MNMT_RAW(DM, true)                                                                                          \
  } else if (g.x_i8) {                                                                                          \
    MNMT_RAW(DM, false)                                                                                         \
  } else if (in.chain.done && chain_logits_tiles(g.V) == 4) {                                                   \
    hipLaunchKernelGGL((k_step_logits<DM, false, 4, true>), dim3(cblocks), dim3(kStepThreads), 0, s, in, g);    \
  } else {                                                                                                      \
    hipLaunchKernelGGL((k_step_logits<DM, false, kLogitsTiles, true>), dim3(blocks), dim3(kStepThreads), 0, s, in, \
                       g);                                                                                      \
  }
  MNMT_BY_D(g.d, MNMT_LOGITS)
#undef MNMT_LOGITS
#undef MNMT_RAW
  return hipGetLastError();
}

}  // namespace mnmt
