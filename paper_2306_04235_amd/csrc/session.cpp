// session.cpp -- workspace plan, encoder / decoder drivers, greedy and beam
// search loops, and hipGraph capture of a whole search.
//
// Workspace plan (Section 4.2: buffers shared by operations that never live
// at the same time): the encoder's activations (fp32 residual, int8 LN/context
// buffer, int8 QKV, int8 FFN hidden, int8 output) share one region with the
// decoder's fp32 logits, which are only needed after encoding has finished.
// Each layer reuses the same few buffers: one fp32 residual stream and int8
// buffers for the sublayer input, attention context and FFN hidden layer.
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <string>
#include <utility>

#include "internal.h"

namespace mnmt {
namespace {

struct Bump {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = (off + 255) / 256 * 256;
    off = o + bytes;
    return o;
  }
};

constexpr size_t kEncAccRows = 64;  // rows of the small-batch encoder path

struct Plan {
  size_t src, len, region, enc_x, enc_x2, enc_a, enc_qkv, enc_h, enc_out, logits;
  std::vector<size_t> cross_kv, kc, vc;
  size_t dec_x, dec_x2, dec_a, dec_qkv, dec_q, dec_h, dec_u, dec_part, fslots, enc_acc;
  size_t cur_tok, step, slots, out_tok, finished, out_len, out_key, lp;
  size_t score, cand_score, cand_tok, tok_hist, par_hist, hist, fin_score, fin_len, fin_row, fin_count, done;
  size_t chain_err, enc_chain, beam_count, epoch, step_x64;
  size_t total;
};

int validate_cfg(const mnmt_model* m, const mnmt_session_cfg* c) {
  if (!m || !c) return set_error(MNMT_E_INVALID_ARG, "null model or session config");
  const int P = m->info.max_pos;
  if (c->max_batch < 1 || c->max_batch > 65536 || c->max_src_len < 1 || c->max_src_len > 256 ||
      c->max_src_len > P || c->max_tgt_len < 1 || c->max_tgt_len > 256 || c->max_tgt_len > P || c->beam < 1 ||
      c->beam > 8 || 2 * c->beam > m->info.vocab)
    return set_error(MNMT_E_INVALID_ARG,
                     "session config out of range: need max_batch >= 1, 1 <= max_src_len, max_tgt_len <= "
                     "min(256, max_pos), 1 <= beam <= 8 and 2*beam <= vocab");
  return MNMT_OK;
}

size_t enc_acc_bytes(size_t d) { return 4 * kEncAccRows * d * sizeof(int32_t); }

// The chain's flag words: one slot of kChainSlotWords per kernel of a step
// (self-attention, cross-attention, FFN per layer, then the logits).
size_t chain_words(const mnmt_model* m) { return (3 * (size_t)m->info.n_dec + 1) * kChainSlotWords; }

// 8-byte words cleared by the greedy reset: the fused arg-max slots, the
// decode-step accumulators and the chain's flag words, which follow each other.
int fslots_words(const mnmt_model* m) {
  return 8 * fused_slots_per_row(m->info.vocab) + 3 * 2 * m->info.d_model + (int)(chain_words(m) / 2);
}

Plan make_plan(const mnmt_model* m, const mnmt_session_cfg& c) {
  Plan p{};
  Bump b;
  const size_t d = m->info.d_model, F = m->info.d_ffn, V = m->info.vocab, Ld = m->info.n_dec;
  const size_t B = c.max_batch, S = c.max_src_len, T = c.max_tgt_len, W = c.beam, R = B * W, BS = B * S;
  p.src = b.take(4 * BS);
  p.len = b.take(4 * B);
  // shared region: encoder scratch | decoder logits
  Bump r;
  p.enc_x = r.take(4 * BS * d);
  p.enc_a = r.take(BS * d);
  p.enc_qkv = r.take(BS * 3 * d);
  p.enc_h = r.take(BS * F);
  p.enc_out = r.take(BS * d);
  p.enc_x2 = r.take(4 * BS * d);
  const size_t enc_bytes = r.off;
  const size_t logit_bytes = 4 * R * V;
  p.region = b.take(enc_bytes > logit_bytes ? enc_bytes : logit_bytes);
  p.enc_x += p.region;
  p.enc_a += p.region;
  p.enc_qkv += p.region;
  p.enc_h += p.region;
  p.enc_out += p.region;
  p.enc_x2 += p.region;
  p.logits = p.region;
  for (size_t l = 0; l < Ld; ++l) p.cross_kv.push_back(b.take(BS * 2 * d));
  // int32 split-K accumulators of the small-batch encoder: W_o and W2 sums,
  // two of each (zero at creation; every encode leaves them zero)
  p.enc_acc = b.take(enc_acc_bytes(d));
  p.dec_x = b.take(4 * R * d);
  p.dec_x2 = b.take(4 * R * d);
  // fused arg-max slots, the decode-step int32 accumulators and the chain's
  // flag words (cleared together)
  p.fslots = b.take(8 * 8 * (size_t)fused_slots_per_row(m->info.vocab) + 8 * 3 * 2 * d + 4 * chain_words(m));
  p.dec_a = b.take(R * d);
  p.dec_qkv = b.take(R * 3 * d);
  p.dec_q = b.take(R * d);
  p.dec_h = b.take(R * F);
  p.dec_u = b.take(R * d);  // factorized embedding: emb_dim <= d codes per row
  p.dec_part = b.take(4 * kMaxSplits * R * d);  // split-K partial sums of the long-K decoder layers
  for (size_t l = 0; l < Ld; ++l) {
    p.kc.push_back(b.take(R * T * d));
    p.vc.push_back(b.take(R * T * d));
  }
  p.cur_tok = b.take(4 * R);
  p.step = b.take(4);
  p.slots = b.take(8 * R);
  p.out_tok = b.take(4 * T * R);
  p.finished = b.take(4 * R);
    p.out_len = b.take(4 * R);
  p.out_key = b.take(8 * T * R);
  p.lp = b.take(4 * (T + 1));
  p.score = b.take(4 * R);
  p.cand_score = b.take(4 * R * 2 * W);
  p.cand_tok = b.take(4 * R * 2 * W);
  p.tok_hist = b.take(4 * T * R);
  p.par_hist = b.take(4 * T * R);
  p.hist = b.take(4 * 2 * R * T);
  p.fin_score = b.take(4 * B * W);
  p.fin_len = b.take(4 * B * W);
  p.fin_row = b.take(4 * B * W);
  p.fin_count = b.take(4 * B);
  p.done = b.take(4 * B);
  p.chain_err = b.take(4);
  p.beam_count = b.take(4);
  p.enc_chain = b.take(4 * 2 * (size_t)m->info.n_enc * kChainSlotWords);
  p.epoch = b.take(4);
  p.step_x64 = b.take(8 * 3 * Ld * 2 * d);
  p.total = (b.off + 255) / 256 * 256;
  return p;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

#define LAUNCH(x)                                                   \
  do {                                                              \
    hipError_t _e = (x);                                            \
    if (_e != hipSuccess) return hip_error(_e, #x);                 \
  } while (0)

int qlin(const LinearDev& L, const int8_t* X, int M, int kind, void* out, float gamma, hipStream_t s,
         unsigned long long* argmax = nullptr) {
  EpiArgs e{kind, out, L.N, gamma, argmax};
  const int8_t* w;
  const bool w4 = batched_weights(L, w);
  LAUNCH(launch_qlinear(X, L.K, w, L.scale, L.bias, M, L.K, L.N, e, s, w4));
  return MNMT_OK;
}

// A factorized embedding (Section 2.1) runs on the general decode paths only:
// the fused batch-1 kernels embed and project over rows of the model width.
bool factored(const mnmt_model* m) { return m->info.emb_dim > 0; }

// Embedding rows x [rows, d] of tok (position r % S_for_pos, or *step).
int embed_rows(const mnmt_session* S, const int32_t* tok, int rows, int S_for_pos, const int* step, float* x,
               hipStream_t s) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, V = m->info.vocab;
  if (factored(m))
    LAUNCH(launch_embed_proj(tok, rows, S_for_pos, step, m->E, m->info.emb_dim, m->proj, m->s_proj, m->c_emb, m->pe,
                             d, V, x, s));
  else
    LAUNCH(launch_embed(tok, rows, S_for_pos, step, m->E, m->c_emb, m->pe, d, V, x, s));
  return MNMT_OK;
}

// The int8 rows [R, K] the tied output projection takes: the final rows a
// [R, d], or for a factorized embedding their projection back to emb_dim.
int logits_input(mnmt_session* S, int R, const int8_t** X, int* K, hipStream_t s) {
  const mnmt_model* m = S->m;
  *X = S->dec_a;
  *K = m->info.d_model;
  if (!factored(m)) return MNMT_OK;
  const int rc = qlin(m->proj_out, S->dec_a, R, MNMT_EPI_I8, S->dec_u, 1.f, s);
  *X = S->dec_u;
  *K = m->info.emb_dim;
  return rc;
}

// Encoder for at most 64 rows (the batch-1 latency path): the embedding and
// every LayerNorm run in the prologue of the matrix-core GEMM that consumes
// them; per layer [LN + QKV] [attention] [W_o + residual] [LN + W1 + ReLU]
// [W2 + residual].  Post-LN models alternate between two residual buffers.
int run_encoder_small(mnmt_session* S, hipStream_t s) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, rows = S->B * S->S;
  const bool post = m->info.ln_post;
  float* xc = S->enc_x;
  float* xo = S->enc_x2;
  auto input = [&](bool embed, bool do_ln, const LnDev& ln, float inv_s, bool write_norm) {
    FusedIn in{};
    in.x = xc;
    in.embed = embed;
    in.tok = S->src;
    in.E = m->E;
    in.c_emb = m->c_emb;
    in.pe = m->pe;
    in.V = m->info.vocab;
    in.S_pos = S->S;
    in.do_ln = do_ln;
    in.g = ln.g;
    in.b = ln.b;
    in.eps = m->info.ln_eps;
    in.inv_s = inv_s;
    if (embed) {
      in.x_out = xc;
      in.wb_input = 1;
    } else if (write_norm) {
      in.x_out = xo;
    }
    return in;
  };
  auto small = [&](const FusedIn* in, const int8_t* X, const LinearDev& L, int kind, void* out, float gamma) {
    EpiArgs e{kind, out, L.N, gamma, nullptr};
    const int8_t* w;
    const bool w4 = batched_weights(L, w);
    return launch_qgemm_small(in, X, L.K, w, L.scale, L.bias, rows, L.K, L.N, e, s, w4);
  };
  for (size_t l = 0; l < m->enc.size(); ++l) {
    const LayerDev& L = m->enc[l];
    const bool embed = l == 0;
    FusedIn in = input(embed, post ? !embed : true, post ? (embed ? L.sa_ln : m->enc[l - 1].ff_ln) : L.sa_ln,
                       L.qkv.inv_in, post && !embed);
    LAUNCH(small(&in, nullptr, L.qkv, MNMT_EPI_I8, S->enc_qkv, 1.f));
    if (post && !embed) std::swap(xc, xo);
    LAUNCH(launch_attn_enc(S->enc_qkv, S->len, S->B, S->S, d, m->info.n_heads, L.sa_cqk, L.sa_cpv, S->enc_a, s));
    LAUNCH(small(nullptr, S->enc_a, L.o, MNMT_EPI_F32_RESID, xc, L.sa_gamma));
    in = input(false, true, post ? L.sa_ln : L.ff_ln, L.w1.inv_in, post);
    LAUNCH(small(&in, nullptr, L.w1, MNMT_EPI_I8_RELU, S->enc_h, 1.f));
    if (post) std::swap(xc, xo);
    LAUNCH(small(nullptr, S->enc_h, L.w2, MNMT_EPI_F32_RESID, xc, L.ff_gamma));
  }
  const LnDev& lnf = post ? m->enc.back().ff_ln : m->enc_ln;
  LAUNCH(launch_ln_quant(xc, rows, d, 1, lnf.g, lnf.b, m->info.ln_eps, m->inv_enc, S->enc_out, nullptr, s));
  for (size_t l = 0; l < m->dec.size(); ++l)
    LAUNCH(small(nullptr, S->enc_out, m->dec[l].ckv, MNMT_EPI_I8, S->cross_kv[l], 1.f));
  return MNMT_OK;
}

// Encoder for at most 64 rows in 2 kernels per layer (encode_small.hip):
// [attention block] [FFN block] per layer, then [final LayerNorm + encoder
// output + every decoder layer's cross K|V].  Each kernel applies the
// previous sublayer's residual update in its prologue; the W_o and W2 int32
// accumulators alternate by layer parity and are cleared by the kernel after
// their consumer, so that all four are zero again when the encode ends.
// Host state of a translation's kernel chain: kernel j runs on stream j mod 2,
// after kernel j - 2 (stream order), and waits on the flags of kernel j - 1.
struct Chain {
  hipStream_t st[2];
  unsigned* flags;
  int* err;
  long j = 0;  // kernels launched so far
  int prev_slot = 0, prev_blocks = 0;
  unsigned prev_val = 0;
  // The chain arguments of the next kernel (flag slot, block count, the value
  // its blocks store) and the stream it goes on.
  hipStream_t next(StepChain& c, int slot, int blocks, unsigned val, bool signal = true) {
    c.wait = j > 0 ? flags + (size_t)prev_slot * kChainSlotWords : nullptr;
    c.nwait = prev_blocks;
    c.want = prev_val;
    c.done = signal ? flags + (size_t)slot * kChainSlotWords : nullptr;
    c.val = val;
    c.err = err;
    prev_slot = slot;
    prev_blocks = blocks;
    prev_val = val;
    return st[j++ & 1];
  }
  hipStream_t last() const { return st[(j - 1) & 1]; }
};

int run_encoder_blocks(mnmt_session* S, hipStream_t s, Chain* ch = nullptr) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, h = m->info.n_heads, R = S->B * S->S;
  const int L = (int)m->enc.size();
  const bool post = m->info.ln_post;
  int32_t* acc_o[2] = {S->enc_acc, S->enc_acc + kEncAccRows * d};
  int32_t* acc_f[2] = {S->enc_acc + 2 * kEncAccRows * d, S->enc_acc + 3 * kEncAccRows * d};
  const int n = R * d;
  float* xa = S->enc_x;
  float* xb = S->enc_x2;
  const float* any_d = m->enc[0].sa_ln.g;  // a valid float[d] for operands a kernel does not use
  auto base = [&](float inv_s) {
    EncIn in{};
    in.R = R;
    in.d = d;
    in.S = S->S;
    in.tok = S->src;
    in.E = m->E;
    in.c_emb = m->c_emb;
    in.pe = m->pe;
    in.V = m->info.vocab;
    in.x_in = xa;
    in.x_out = xb;
    in.acc = acc_o[0];
    in.scale = any_d;
    in.bias = any_d;
    in.gamma = 1.0f;
    in.ln_g = any_d;
    in.ln_b = any_d;
    in.eps = m->info.ln_eps;
    in.inv_s = inv_s;
    return in;
  };
  // the residual update of the sublayer whose partial sums are in acc (and
  // its post-LN LayerNorm in post-LN models), then the next pre-LN LayerNorm
  auto rows = [&](EncIn& in, const int32_t* acc, const LinearDev* Lp, float gamma, const LnDev& post_ln,
                  const LnDev& pre_ln) {
    if (acc) {
      in.acc = acc;
      in.scale = Lp->scale;
      in.bias = Lp->bias;
      in.gamma = gamma;
      in.update = 1;
    }
    const LnDev& ln = post ? post_ln : pre_ln;
    if (ln.g && (acc || !post)) {
      in.ln_g = ln.g;
      in.ln_b = ln.b;
      in.ln_mode = post ? 1 : 2;
    }
  };
  const LnDev none{};
  for (int l = 0; l < L; ++l) {
    const LayerDev& Ly = m->enc[l];
    {  // self-attention block
      EncIn in = base(Ly.qkv.inv_in);
      if (l == 0) {
        in.embed = 1;  // the embeddings become the residual stream
        rows(in, nullptr, nullptr, 1.0f, none, Ly.sa_ln);
        in.zero1 = acc_f[0];
        in.zero1_n = n;
      } else {
        const LayerDev& P = m->enc[l - 1];
        rows(in, acc_f[(l - 1) & 1], &P.w2, P.ff_gamma, P.ff_ln, Ly.sa_ln);
      }
      in.zero0 = acc_o[(l + 1) & 1];
      in.zero0_n = n;
      EncAttn at{};
      at.dh = m->dh;
      at.w4 = pick_weights(Ly.qkv, Ly.o, at.W, at.Wo);
      at.scale = Ly.qkv.scale;
      at.bias = Ly.qkv.bias;
      at.len = S->len;
      at.c_qk = Ly.sa_cqk;
      at.c_pv = Ly.sa_cpv;
      at.acc_out = acc_o[l & 1];
      const hipStream_t ks = ch ? ch->next(in.chain, 2 * l, h * enc_attn_qsplit(R), 1) : s;
      LAUNCH(launch_enc_attn(in, at, h, ks));
      std::swap(xa, xb);
    }
    {  // FFN block
      EncIn in = base(Ly.w1.inv_in);
      rows(in, acc_o[l & 1], &Ly.o, Ly.sa_gamma, Ly.sa_ln, Ly.ff_ln);
      in.zero0 = acc_f[(l + 1) & 1];
      in.zero0_n = n;
      EncFfn f{};
      f.F = Ly.w1.N;
      f.w4 = pick_weights(Ly.w1, Ly.w2, f.W1, f.W2);
      f.scale1 = Ly.w1.scale;
      f.bias1 = Ly.w1.bias;
      f.acc_out = acc_f[l & 1];
      const hipStream_t ks = ch ? ch->next(in.chain, 2 * l + 1, f.F / 64, 1) : s;
      LAUNCH(launch_enc_ffn(in, f, ks));
      std::swap(xa, xb);
    }
  }
  // final LayerNorm (post-LN: the last layer's), the int8 encoder output and
  // the cross keys and values of every decoder layer
  const LayerDev& last = m->enc.back();
  EncIn in = base(m->inv_enc);
  in.x_out = nullptr;
  rows(in, acc_f[(L - 1) & 1], &last.w2, last.ff_gamma, last.ff_ln, m->enc_ln);
  in.q_out = S->enc_out;
  in.zero0 = acc_o[(L - 1) & 1];
  in.zero0_n = n;
  EncOut o{};
  o.layers = (int)m->dec.size();
  o.w4 = true;  // packed 4-bit rows when every layer has them
  for (int l = 0; l < o.layers; ++l) o.w4 = o.w4 && m->dec[l].ckv.w4;
  for (int l = 0; l < o.layers; ++l) {
    o.layer[l].W = o.w4 ? reinterpret_cast<const int8_t*>(m->dec[l].ckv.w4) : m->dec[l].ckv.w;
    o.layer[l].scale = m->dec[l].ckv.scale;
    o.layer[l].bias = m->dec[l].ckv.bias;
    o.layer[l].out = S->cross_kv[l];
  }
  // the last kernel of the chain: no flag (the caller joins the streams)
  const hipStream_t ks = ch ? ch->next(in.chain, 0, o.layers * 2 * d / 64, 1, false) : s;
  LAUNCH(launch_enc_out(in, o, ks));
  return MNMT_OK;
}

// Encoder over the session's current batch (rows = B * S, padded rows are
// computed and ignored), then every decoder layer's cross keys/values.
int run_encoder(mnmt_session* S, hipStream_t s) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, rows = S->B * S->S;
  const bool post = m->info.ln_post;
  const float eps = m->info.ln_eps;
  if (!factored(m) && enc_small_fits(rows, S->S, d, m->dh, m->info.d_ffn) && (int)m->dec.size() <= EncOut::kMaxLayers) {
    if (!S->chain_on || m->info.n_heads > kChainCopyStride || m->info.d_ffn / 64 > kChainCopyStride)
      return run_encoder_blocks(S, s);
    // the encoder's kernels as a chain over the two streams (see Chain)
    MNMT_HIP(hipEventRecord(S->fork_ev, s));
    MNMT_HIP(hipStreamWaitEvent(S->side_stream, S->fork_ev, 0));
    Chain ch{{s, S->side_stream}, S->enc_chain, S->chain_err};
    const int rc = run_encoder_blocks(S, s, &ch);
    MNMT_HIP(hipEventRecord(S->join_ev, S->side_stream));
    MNMT_HIP(hipStreamWaitEvent(s, S->join_ev, 0));
    return rc;
  }
  if (!factored(m) && qgemm_small_fits(rows, d) && qgemm_small_fits(rows, m->info.d_ffn))
    return run_encoder_small(S, s);
  int rc0 = embed_rows(S, S->src, rows, S->S, nullptr, S->enc_x, s);
  if (rc0) return rc0;
  const LayerDev& L0 = m->enc[0];
  LAUNCH(launch_ln_quant(S->enc_x, rows, d, !post, L0.sa_ln.g, L0.sa_ln.b, eps, L0.qkv.inv_in, S->enc_a, nullptr, s));
  for (size_t l = 0; l < m->enc.size(); ++l) {
    const LayerDev& L = m->enc[l];
    int rc;
    if ((rc = qlin(L.qkv, S->enc_a, rows, MNMT_EPI_I8, S->enc_qkv, 1.f, s))) return rc;
    LAUNCH(launch_attn_enc(S->enc_qkv, S->len, S->B, S->S, d, m->info.n_heads, L.sa_cqk, L.sa_cpv, S->enc_a, s));
    if ((rc = qlin(L.o, S->enc_a, rows, MNMT_EPI_F32_RESID, S->enc_x, L.sa_gamma, s))) return rc;
    // input of the FFN: pre-LN normalizes with the FFN's LayerNorm; post-LN
    // normalizes the residual with the attention sublayer's LayerNorm.
    const LnDev& ln1 = post ? L.sa_ln : L.ff_ln;
    LAUNCH(launch_ln_quant(S->enc_x, rows, d, 1, ln1.g, ln1.b, eps, L.w1.inv_in, S->enc_a, post ? S->enc_x : nullptr, s));
    if ((rc = qlin(L.w1, S->enc_a, rows, MNMT_EPI_I8_RELU, S->enc_h, 1.f, s))) return rc;
    if ((rc = qlin(L.w2, S->enc_h, rows, MNMT_EPI_F32_RESID, S->enc_x, L.ff_gamma, s))) return rc;
    const bool last = l + 1 == m->enc.size();
    int8_t* dst = last ? S->enc_out : S->enc_a;
    const float inv = last ? m->inv_enc : m->enc[l + 1].qkv.inv_in;
    const LnDev& ln2 = post ? L.ff_ln : (last ? m->enc_ln : m->enc[l + 1].sa_ln);
    LAUNCH(launch_ln_quant(S->enc_x, rows, d, 1, ln2.g, ln2.b, eps, inv, dst, post ? S->enc_x : nullptr, s));
  }
  for (size_t l = 0; l < m->dec.size(); ++l) {
    int rc;
    if ((rc = qlin(m->dec[l].ckv, S->enc_out, rows, MNMT_EPI_I8, S->cross_kv[l], 1.f, s))) return rc;
  }
  return MNMT_OK;
}

// One decoder step for R rows (W hypotheses per sentence); ends with the
// final sublayer input in dec_a, ready for the output projection.
// rows_ready: dec_x and dec_a already hold the step's input rows (written by
// the previous step's beam update).
// t_host: the step index when known at enqueue (>= 0), else -1 (the kernels
// read the device step counter).
int run_decoder_layers(mnmt_session* S, int R, int W, bool beam, hipStream_t s, bool rows_ready = false,
                       int t_host = -1) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, h = m->info.n_heads, T = S->cfg.max_tgt_len;
  const bool post = m->info.ln_post;
  const float eps = m->info.ln_eps;
  const LayerDev& L0 = m->dec[0];
  float* xc = S->dec_x;
  if (!rows_ready) {
    const int rc0 = embed_rows(S, S->cur_tok, R, 1, S->step, S->dec_x, s);
    if (rc0) return rc0;
    LAUNCH(launch_ln_quant(S->dec_x, R, d, !post, L0.sa_ln.g, L0.sa_ln.b, eps, L0.qkv.inv_in, S->dec_a, nullptr, s));
  }
  // a residual update left pending by a split-K layer (splits > 0), applied
  // by the next LayerNorm kernel or in the prologue of the fused
  // self-attention kernel
  ResidUpdate pend{};
  float* const xbuf[2] = {S->dec_x, S->dec_x2};
  // LayerNorm + quantization of the rows with L's input scale into dec_a
  // (post-LN: the normalized rows also replace x)
  auto ln_rows = [&](const LnDev& ln, float inv_s, bool replace) -> int {
    if (pend.splits) {
      LAUNCH(launch_resid_ln_quant(xc, R, d, pend, 1, ln.g, ln.b, eps, inv_s, S->dec_a, replace, s));
      pend.splits = 0;
    } else {
      LAUNCH(launch_ln_quant(xc, R, d, 1, ln.g, ln.b, eps, inv_s, S->dec_a, replace ? xc : nullptr, s));
    }
    return MNMT_OK;
  };
  // the linear layer L over the rows LN(x) quantized with L's input scale;
  // pre-LN rows that the one-round-trip GEMM takes above 64 rows are
  // normalized in its prologue (each 16x64 block its 16 rows) instead of by a
  // kernel of their own
  auto ln_linear = [&](const LinearDev& L, const LnDev& ln, int kind, void* out) -> int {
    if (S->ln_fused_on && !post && !pend.splits && R > 64 && qgemm_rows_fit(R, L.K, L.N) && L.K == d) {
      FusedIn in{};
      in.x = xc;
      in.do_ln = 1;
      in.g = ln.g;
      in.b = ln.b;
      in.eps = eps;
      in.inv_s = L.inv_in;
      const int8_t* w;
      const bool w4 = batched_weights(L, w);
      const EpiArgs e{kind, out, L.N, 1.f, nullptr};
      LAUNCH(launch_qgemm_small(&in, nullptr, 0, w, L.scale, L.bias, R, L.K, L.N, e, s, w4));
      return MNMT_OK;
    }
    const int rc = ln_rows(ln, L.inv_in, post);
    return rc ? rc : qlin(L, S->dec_a, R, kind, out, 1.f, s);
  };
  for (size_t l = 0; l < m->dec.size(); ++l) {
    const LayerDev& L = m->dec[l];
    int rc;
    if (S->qkv_fused_on && S->ln_fused_on && beam && !post && R > 64 && attn_self_qkv_fits(W, d, h, T) &&
        (l > 0 || !pend.splits)) {
      // the Q/K/V projection inside the self-attention kernel (one block per
      // head and sentence), from the step's int8 input rows (layer 0) or the
      // LayerNorm each block computes (later layers, after the pending update
      // of a split W2: the head-0 blocks store the updated rows into the
      // other residual buffer, since the other blocks still read the old
      // ones); the context goes to dec_q (other blocks of a sentence still
      // read its rows of dec_a)
      FusedIn in{};
      float* xn = xc;
      if (l > 0) {
        in.x = xc;
        in.do_ln = 1;
        in.g = L.sa_ln.g;
        in.b = L.sa_ln.b;
        in.eps = eps;
        in.inv_s = L.qkv.inv_in;
        if (pend.splits) {
          in.part = pend.part;
          in.nparts = pend.splits;
          in.part_stride = (size_t)R * d;
          in.pscale = pend.scale;
          in.pbias = pend.bias;
          in.pgamma = pend.gamma;
          in.x_out = xn = xc == xbuf[0] ? xbuf[1] : xbuf[0];
          in.wb_input = 1;
          pend.splits = 0;
        }
      }
      const int8_t* w;
      const bool w4 = batched_weights(L.qkv, w);
      LAUNCH(launch_attn_self_qkv(l > 0 ? nullptr : S->dec_a, l > 0 ? &in : nullptr, w, L.qkv.scale, L.qkv.bias, w4,
                                  R, W, d, h, T, S->step, S->kcache[l], S->vcache[l], S->beam.hist, L.sa_cqk,
                                  L.sa_cpv, S->dec_q, s, t_host));
      xc = xn;
      if ((rc = qlin(L.o, S->dec_q, R, MNMT_EPI_F32_RESID, xc, L.sa_gamma, s))) return rc;
    } else {
      if (l == 0)  // the step's input rows, quantized by the embedding step or the beam update
        rc = qlin(L.qkv, S->dec_a, R, MNMT_EPI_I8, S->dec_qkv, 1.f, s);
      else  // pre-LN: the layer's own LayerNorm; post-LN: the previous FFN's
        rc = ln_linear(L.qkv, post ? m->dec[l - 1].ff_ln : L.sa_ln, MNMT_EPI_I8, S->dec_qkv);
      if (rc) return rc;
      LAUNCH(launch_attn_dec_self(S->dec_qkv, R, d, h, T, S->step, S->kcache[l], S->vcache[l],
                                  beam ? S->beam.hist : nullptr, L.sa_cqk, L.sa_cpv, S->dec_a, s, t_host));
      if ((rc = qlin(L.o, S->dec_a, R, MNMT_EPI_F32_RESID, xc, L.sa_gamma, s))) return rc;
    }
    int8_t* cctx = S->dec_a;  // the cross-attention context rows
    if (attn_cross_q_fits(W, d)) {
      // the Q projection inside the attention kernel, from the LayerNorm'd
      // rows in dec_a; the context goes to dec_q (other blocks of a sentence
      // still read its rows of dec_a)
      // (pre-LN: each block normalizes its sentence's rows itself)
      const bool own_ln = S->ln_fused_on && !post && !pend.splits;
      FusedIn in{};
      if (own_ln) {
        in.x = xc;
        in.do_ln = 1;
        in.g = L.ca_ln.g;
        in.b = L.ca_ln.b;
        in.eps = eps;
        in.inv_s = L.cq.inv_in;
      } else if ((rc = ln_rows(post ? L.sa_ln : L.ca_ln, L.cq.inv_in, post))) {
        return rc;
      }
      const int8_t* wq;
      const bool w4 = batched_weights(L.cq, wq);
      cctx = S->dec_q;
      LAUNCH(launch_attn_dec_cross_q(own_ln ? nullptr : S->dec_a, own_ln ? &in : nullptr, wq, L.cq.scale, L.cq.bias,
                                     w4, R, W, d, h, S->cross_kv[l], S->S, S->len, L.ca_cqk, L.ca_cpv, cctx, s));
    } else {
      if ((rc = ln_linear(L.cq, post ? L.sa_ln : L.ca_ln, MNMT_EPI_I8, S->dec_q))) return rc;
      LAUNCH(launch_attn_dec_cross(S->dec_q, R, W, d, h, S->cross_kv[l], S->S, S->len, L.ca_cqk, L.ca_cpv, cctx, s));
    }
    if ((rc = qlin(L.co, cctx, R, MNMT_EPI_F32_RESID, xc, L.ca_gamma, s))) return rc;
    if ((rc = ln_linear(L.w1, post ? L.ca_ln : L.ff_ln, MNMT_EPI_I8_RELU, S->dec_h))) return rc;
    if (const int sp = qgemm_splits(R, L.w2.K, L.w2.N)) {  // long K: partial sums, update pending
      const int8_t* w;
      const bool w4 = batched_weights(L.w2, w);
      LAUNCH(launch_qgemm_split(S->dec_h, L.w2.K, w, R, L.w2.K, L.w2.N, S->dec_part, s, w4));
      pend = ResidUpdate{S->dec_part, sp, L.w2.scale, L.w2.bias, L.ff_gamma};
    } else if ((rc = qlin(L.w2, S->dec_h, R, MNMT_EPI_F32_RESID, xc, L.ff_gamma, s))) {
      return rc;
    }
  }
  // the final LayerNorm (post-LN: the last FFN's) into dec_a for the output
  // projection
  const LayerDev& last = m->dec.back();
  return ln_rows(post ? last.ff_ln : m->dec_ln, m->inv_fin, false);
}

// Greedy step: layers, tied output projection with fused arg-max (batch <= 8)
// or logits + row arg-max, then bookkeeping.  logits_out: optional [R, V].
int greedy_step(mnmt_session* S, int R, int stop_at_eos, float* logits_out, hipStream_t s) {
  const mnmt_model* m = S->m;
  int rc = run_decoder_layers(S, R, 1, false, s);
  if (rc) return rc;
  const int V = m->info.vocab;
  const int8_t* X;
  int K;
  if ((rc = logits_input(S, R, &X, &K, s))) return rc;
  if (R <= 8) {
    EpiArgs e{EPI_LOGITS_ARGMAX, logits_out, V, 1.f, S->slots};
    LAUNCH(launch_qlinear(X, K, m->E, m->c_out, nullptr, R, K, V, e, s));
  } else {
    float* z = logits_out ? logits_out : S->logits;
    EpiArgs e{MNMT_EPI_LOGITS, z, V, 1.f, nullptr};
    LAUNCH(launch_qlinear(X, K, m->E, m->c_out, nullptr, R, K, V, e, s));
    LAUNCH(launch_row_argmax(z, R, V, S->slots, s));
  }
    LAUNCH(launch_greedy_commit(S->slots, R, S->cfg.max_tgt_len, S->cur_tok, S->out_tok, S->finished, S->out_len,
                              S->step, stop_at_eos, m->info.eos_id, m->info.pad_id, S->out_key, s));
  return MNMT_OK;
}

// Greedy step for at most 8 rows with LayerNorm (and the embedding) fused into
// the GEMV that consumes it, per decoder layer:
//   [LN + QKV] [self-attention] [W_o + residual] [LN + Q] [cross-attention]
//   [W_oc + residual] [LN + W1 + ReLU] [W2 + residual]
// then [LN + logits + arg-max] and [commit].  Post-LN models alternate between
// two residual buffers: block 0 writes the normalized rows while the other
// blocks still read the un-normalized ones.
int greedy_step_fused(mnmt_session* S, int R, int t, int stop_at_eos, float* logits_out, hipStream_t s) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, h = m->info.n_heads, T = S->cfg.max_tgt_len;
  const bool post = m->info.ln_post;
  float* xc = S->dec_x;
  float* xo = S->dec_x2;
  auto input = [&](bool embed, bool do_ln, const LnDev& ln, float inv_s, bool write_norm) {
    FusedIn in{};
    in.x = xc;
    in.embed = embed;
    in.tok = S->cur_tok;
    in.E = m->E;
    in.c_emb = m->c_emb;
    in.pe = m->pe;
    in.V = m->info.vocab;
    in.do_ln = do_ln;
    in.g = ln.g;
    in.b = ln.b;
    in.eps = m->info.ln_eps;
    in.inv_s = inv_s;
    if (embed) {
      in.x_out = xc;  // the embedding becomes the residual stream
      in.wb_input = 1;
    } else if (write_norm) {
      in.x_out = xo;  // post-LN: the normalized rows become the residual stream
      in.wb_input = 0;
    }
    return in;
  };
  auto gemv = [&](const LinearDev& L, int epi, void* out) {
    FusedGemv gv{};
    gv.R = R;
    gv.K = L.K;
    gv.N = L.N;
    gv.t = t;
    gv.epi = epi;
    gv.w4 = batched_weights(L, gv.W);
    gv.scale = L.scale;
    gv.bias = L.bias;
    gv.out = out;
    return gv;
  };
  int rc;
  for (size_t l = 0; l < m->dec.size(); ++l) {
    const LayerDev& L = m->dec[l];
    {
      const bool embed = l == 0;
      const LnDev& ln = post ? (embed ? L.sa_ln : m->dec[l - 1].ff_ln) : L.sa_ln;
      LAUNCH(launch_qgemv_ln(input(embed, post ? !embed : true, ln, L.qkv.inv_in, post && !embed),
                             gemv(L.qkv, MNMT_EPI_I8, S->dec_qkv), s));
      if (post && !embed) std::swap(xc, xo);
    }
    LAUNCH(launch_attn_dec_self(S->dec_qkv, R, d, h, T, S->step, S->kcache[l], S->vcache[l], nullptr, L.sa_cqk,
                                L.sa_cpv, S->dec_a, s));
    if ((rc = qlin(L.o, S->dec_a, R, MNMT_EPI_F32_RESID, xc, L.sa_gamma, s))) return rc;
    LAUNCH(launch_qgemv_ln(input(false, true, post ? L.sa_ln : L.ca_ln, L.cq.inv_in, post),
                           gemv(L.cq, MNMT_EPI_I8, S->dec_q), s));
    if (post) std::swap(xc, xo);
    LAUNCH(launch_attn_dec_cross(S->dec_q, R, 1, d, h, S->cross_kv[l], S->S, S->len, L.ca_cqk, L.ca_cpv, S->dec_a, s));
    if ((rc = qlin(L.co, S->dec_a, R, MNMT_EPI_F32_RESID, xc, L.ca_gamma, s))) return rc;
    LAUNCH(launch_qgemv_ln(input(false, true, post ? L.ca_ln : L.ff_ln, L.w1.inv_in, post),
                           gemv(L.w1, MNMT_EPI_I8_RELU, S->dec_h), s));
    if (post) std::swap(xc, xo);
    if ((rc = qlin(L.w2, S->dec_h, R, MNMT_EPI_F32_RESID, xc, L.ff_gamma, s))) return rc;
  }
  // output projection over the shared embedding with the arg-max, then commit
  LinearDev out_proj{m->E, nullptr, m->c_out, nullptr, m->info.vocab, d, 0.f};
  FusedGemv gv = gemv(out_proj, EPI_LOGITS_ARGMAX, logits_out);
  gv.slots = S->fslots;
  gv.nslots = fused_slots_per_row(m->info.vocab);
  gv.step = S->step;
  gv.out_tok = S->out_tok;
  gv.cur_tok = S->cur_tok;
  gv.finished = S->finished;
    gv.out_len = S->out_len;
  gv.out_key = S->out_key;
  gv.T = T;
  gv.stop_at_eos = stop_at_eos;
  gv.eos = m->info.eos_id;
  gv.pad = m->info.pad_id;
  LAUNCH(launch_qgemv_ln(input(false, true, post ? m->dec.back().ff_ln : m->dec_ln, m->inv_fin, false), gv, s));
  LAUNCH(launch_greedy_commit_slots(gv, s));
  return MNMT_OK;
}

// Greedy step for at most 2 rows in 3 kernels per layer (decode_step.hip):
// [attention block, self] [attention block, cross] [FFN block] per layer,
// then [output projection + arg-max] and [commit].  The step's input rows
// (the embeddings of the current tokens) are in dec_x on entry; the commit
// writes the next step's.  Each kernel applies the previous sublayer's
// residual update in its prologue; the three int32 accumulators (W_o, W_oc,
// W2 partial sums) are cleared by the kernel after their consumer, and the
// residual rows alternate between two buffers.
// The commit folds into the next step when every row's partials fit one
// wave's four loads per lane.
bool fold_ok(const mnmt_model* m) { return fused_slots_per_row(m->info.vocab) <= 256; }

// Every kernel of the 1-2 row step fits the flag slots.
bool chain_ok(const mnmt_model* m) {
  return fold_ok(m) && m->info.n_heads <= kChainMaxBlocks && m->info.d_ffn / 64 <= kChainMaxBlocks &&
         step_logits_blocks_chained(m->info.vocab, m->info.d_model) <= kChainMaxBlocks;
}

// fold (a whole translation's steps): step t > 0 embeds and records step t -
// 1's token inside its first layer instead of a commit kernel after step t -
// 1; the last step commits as usual.
int greedy_step_v3(mnmt_session* S, int R, int t, int stop_at_eos, float* logits_out, hipStream_t s, bool fold,
                   bool last_step, Chain* ch) {
  const mnmt_model* m = S->m;
  const int d = m->info.d_model, h = m->info.n_heads, T = S->cfg.max_tgt_len;
  const bool post = m->info.ln_post;
  unsigned long long* acc_o = S->step_acc;
  unsigned long long* acc_oc = S->step_acc + 2 * d;
  unsigned long long* acc_w2 = S->step_acc + 4 * d;
  const int nacc = R * d;
  float* xa = S->dec_x;
  float* xb = S->dec_x2;
  // a row input with no pending update and no LayerNorm; the pointers of the
  // unused operands only need to be valid
  auto base = [&](float inv_s) {
    StepIn in{};
    in.x_in = xa;
    in.x_out = xb;
    in.acc = acc_o;
    in.scale = m->dec_ln.g ? m->dec_ln.g : m->dec[0].sa_ln.g;
    in.bias = in.scale;
    in.gamma = 1.0f;
    in.ln_g = in.scale;
    in.ln_b = in.scale;
    in.eps = m->info.ln_eps;
    in.inv_s = inv_s;
    return in;
  };
  // the residual update of the sublayer whose partial sums are in acc (its
  // post-LN LayerNorm in post-LN models), and the pre-LN LayerNorm of the next
  auto rows = [&](StepIn& in, const unsigned long long* acc, const LinearDev* L, float gamma, const LnDev& post_ln,
                  const LnDev& pre_ln) {
    if (acc) {
      in.acc = acc;
      in.scale = L->scale;
      in.bias = L->bias;
      in.gamma = gamma;
      in.update = 1;
    }
    const LnDev& ln = post ? post_ln : pre_ln;
    if (ln.g && (acc || !post)) {
      in.ln_g = ln.g;
      in.ln_b = ln.b;
      in.ln_mode = post ? 1 : 2;
    }
  };
  auto attn = [&](const LayerDev& L, bool self, unsigned long long* acc_out) {
    StepAttn at{};
    at.R = R;
    at.d = d;
    at.dh = m->dh;
    at.T = T;
    at.S = S->S;
    at.t = t;
    const LinearDev& P = self ? L.qkv : L.cq;
    at.w4 = pick_weights(P, self ? L.o : L.co, at.W, at.Wo);
    at.scale = P.scale;
    at.bias = P.bias;
    at.len = S->len;
    at.c_qk = self ? L.sa_cqk : L.ca_cqk;
    at.c_pv = self ? L.sa_cpv : L.ca_cpv;
    at.acc_out = acc_out;
    return at;
  };
  const LnDev none{};
  // Counted hand-off (StepCount) between the step's kernels: kernel k of the
  // step (3 per layer, then the logits) polls kernel k - 1's counted sums and
  // tagged rows (0 < k < 3 L) and leaves its own the same way (k < 3 L - 1);
  // the last FFN still stores its rows plainly and flags its blocks, since
  // the logits kernel's hundred-odd blocks would all poll the same words, and
  // the step's first kernel waits on the logits kernel's flags.
  const int nk = 3 * (int)m->dec.size();
  const bool counted = S->counted_on && nk < 32;  // tag offsets t * 32 + k
  int prev_blocks = 0;
  auto count_io = [&](StepIn& in, int k, int blocks) {
    in.cnt.epoch = S->epoch;
    if (counted) {
      if (k > 0) {
        in.cnt.count_in = prev_blocks;
        in.cnt.x_in64 = S->step_x64 + (size_t)(k - 1) * 2 * d;
        in.cnt.tag_in = (unsigned)(t * 32 + k - 1);
        in.chain.wait = nullptr;
        in.chain.nwait = 0;
      }
      if (k < nk - 1) {
        in.cnt.x_out64 = S->step_x64 + (size_t)k * 2 * d;
        in.cnt.tag_out = (unsigned)(t * 32 + k);
        in.x_out = nullptr;
        in.chain.done = nullptr;
      }
    }
    prev_blocks = blocks;
  };
  const bool folded = fold && t > 0 && fold_ok(m);
  // Tagged arg-max partials (chained, counted steps): the logits kernel's
  // partials carry a tag of (translation, step), and the next step's layer-0
  // blocks poll them instead of waiting on the logits kernel's flags.
  const int V = m->info.vocab;
  const int lblocks = step_logits_blocks_chained(V, d);
  const bool tagged = ch && counted && S->tagged_on && fold && fold_ok(m) && V <= kTagMaxV &&
                      lblocks <= fused_slots_per_row(V) && lblocks <= 256;
  StepCommit cm{};
  if (folded) {
    cm.slots = S->fslots;
    cm.nslots = fused_slots_per_row(m->info.vocab);
    cm.E = m->E;
    cm.c_emb = m->c_emb;
    cm.pe = m->pe;
    cm.V = m->info.vocab;
    cm.t = t;
    cm.finished = S->finished;
    cm.out_tok = S->out_tok;
    cm.out_len = S->out_len;
    cm.out_key = S->out_key;
    cm.cur_tok = S->cur_tok;
    cm.step = S->step;
    cm.T = T;
    cm.stop_at_eos = stop_at_eos;
    cm.eos = m->info.eos_id;
    cm.pad = m->info.pad_id;
    cm.tagged = tagged;
    cm.nparts = lblocks;
    cm.epoch = S->epoch;
  }
  // merged: each layer's three phases in one launch (launch_step_layer), the
  // phases handing off through the counted words inside it
  // (the logits kernel's 256 threads poll one flag word per block of the
  // last layer's launch)
  const bool merged = S->merged_on && counted && step_layer_blocks(h, m->info.d_ffn) <= 256;
  // single: the two layers and the logits in one launch (k_step_all), whose
  // arguments are collected here; the chain then advances once per step
  const bool single = merged && tagged && S->single_on &&
                      step_all_fits((int)m->dec.size(), d, h, m->info.d_ffn, T, S->S, m->info.vocab);
  StepAll all{};
  for (size_t l = 0; l < m->dec.size(); ++l) {
    const LayerDev& L = m->dec[l];
    const StepCommit* cml = folded && l == 0 ? &cm : nullptr;
    StepIn ia{}, ib{}, ic{};
    StepAttn sa{}, ca{};
    StepFfn f{};
    {  // self-attention block
      StepIn in = base(L.qkv.inv_in);
      if (l == 0) {
        // the embeddings are the residual stream as they are (folded: the
        // kernel computes them and block 0 stores them for the next kernel)
        if (!cml) in.x_out = nullptr;
        rows(in, nullptr, nullptr, 1.0f, none, L.sa_ln);
      } else {
        const LayerDev& P = m->dec[l - 1];
        rows(in, acc_w2, &P.w2, P.ff_gamma, P.ff_ln, L.sa_ln);
        in.zero_acc = acc_oc;
        in.zero_n = nacc;
      }
      StepAttn at = attn(L, true, acc_o);
      at.kcache = S->kcache[l];
      at.vcache = S->vcache[l];
      if (merged) {
        count_io(in, 3 * (int)l, h);
        ia = in;
        sa = at;
      } else {
        const hipStream_t ks = ch ? ch->next(in.chain, 3 * (int)l, h, t + 1) : s;
        count_io(in, 3 * (int)l, h);
        if (cml && tagged) in.chain.wait = nullptr;  // polls the tagged partials instead
        LAUNCH(launch_step_attn(in, at, 1, h, ks, cml));
      }
      if (in.x_out) std::swap(xa, xb);
    }
    {  // cross-attention block
      StepIn in = base(L.cq.inv_in);
      rows(in, acc_o, &L.o, L.sa_gamma, L.sa_ln, L.ca_ln);
      in.zero_acc = acc_w2;
      in.zero_n = nacc;
      StepAttn at = attn(L, false, acc_oc);
      at.kv = S->cross_kv[l];
      if (merged) {
        count_io(in, 3 * (int)l + 1, h);
        ib = in;
        ca = at;
      } else {
        const hipStream_t ks = ch ? ch->next(in.chain, 3 * (int)l + 1, h, t + 1) : s;
        count_io(in, 3 * (int)l + 1, h);
        LAUNCH(launch_step_attn(in, at, 0, h, ks, cml));
      }
      std::swap(xa, xb);
    }
    {  // FFN block
      StepIn in = base(L.w1.inv_in);
      rows(in, acc_oc, &L.co, L.ca_gamma, L.ca_ln, L.ff_ln);
      in.zero_acc = acc_o;
      in.zero_n = nacc;
      f.R = R;
      f.d = d;
      f.F = L.w1.N;
      f.w4 = pick_weights(L.w1, L.w2, f.W1, f.W2);
      f.scale1 = L.w1.scale;
      f.bias1 = L.w1.bias;
      f.acc_out = acc_w2;
      if (merged) {
        count_io(in, 3 * (int)l + 2, f.F / 64);
        ic = in;
      } else {
        const hipStream_t ks = ch ? ch->next(in.chain, 3 * (int)l + 2, f.F / 64, t + 1) : s;
        count_io(in, 3 * (int)l + 2, f.F / 64);
        LAUNCH(launch_step_ffn(in, f, ks));
      }
      std::swap(xa, xb);
    }
    if (single) {
      // the arguments of this layer's share of the step's launch; the last
      // layer flags its blocks for the logits blocks (the chain's waits and
      // errors are set with the launch)
      all.ia[l] = ia;
      all.sa[l] = sa;
      all.ib[l] = ib;
      all.ca[l] = ca;
      all.ic[l] = ic;
      all.f[l] = f;
      if (l + 1 == m->dec.size()) {
        all.ic[l].chain.done = S->chain + (size_t)(3 * l) * kChainSlotWords;
        all.ic[l].chain.val = (unsigned)(t + 1);
      }
      if (cml) all.cm = *cml;
    } else if (merged) {
      // the launch's chain: in the first layer the self- and cross-attention
      // blocks wait on the previous kernel's flags (the cross blocks of a
      // folded step read the previous step's arg-max partials, which only
      // that wait orders after the logits kernel that writes them; as
      // separate kernels, stream order did); every block of the last layer
      // flags its end for the logits kernel (the next layer instead polls the
      // counted words); polls that give up report through err
      const bool last = l + 1 == m->dec.size();
      StepChain c{};
      const hipStream_t ks = ch ? ch->next(c, 3 * (int)l, step_layer_blocks(h, L.w1.N), t + 1, last) : s;
      if (l == 0 && !(cml && tagged)) {  // (tagged: layer 0 polls the partials instead)
        for (StepIn* p : {&ia, &ib}) {
          p->chain.wait = c.wait;
          p->chain.nwait = c.nwait;
          p->chain.want = c.want;
        }
      }
      ia.chain.err = ib.chain.err = ic.chain.err = c.err;
      ic.chain.done = c.done;
      ic.chain.val = c.val;
      LAUNCH(launch_step_layer(ia, sa, ib, ca, ic, f, ks, cml));
    }
  }
  const LayerDev& last = m->dec.back();
  StepIn in = base(m->inv_fin);
  in.x_out = nullptr;
  rows(in, acc_w2, &last.w2, last.ff_gamma, last.ff_ln, m->dec_ln);
  in.zero_acc = acc_oc;
  in.zero_n = nacc;
  StepLogits g{};
  g.R = R;
  g.d = d;
  g.V = m->info.vocab;
  g.E = m->E_frag;
  g.frag = true;
  g.c_out = m->c_out;
  g.logits = logits_out;
  g.slots = S->fslots;
  g.nslots = fused_slots_per_row(m->info.vocab);
  g.tagged = tagged;
  g.epoch = S->epoch;
  g.t = t;
  const hipStream_t ks =
      ch ? ch->next(in.chain, 3 * (int)m->dec.size(), step_logits_blocks_chained(g.V, d), t + 1) : s;
  if (single) {
    // one launch for the step: the logits blocks wait on the last layer's
    // flags inside it; the step's first layer waits as the launch (tagged:
    // it polls the previous step's partials instead)
    all.layer_blocks = step_layer_blocks(h, m->info.d_ffn);
    const int lastl = (int)m->dec.size() - 1;
    for (int l = 0; l <= lastl; ++l) all.ia[l].chain.err = all.ib[l].chain.err = all.ic[l].chain.err = in.chain.err;
    all.lin = in;
    all.lin.chain.wait = all.ic[lastl].chain.done;
    all.lin.chain.nwait = all.layer_blocks;
    all.lin.chain.want = (unsigned)(t + 1);
    all.g = g;
    LAUNCH(launch_step_all(all, folded, ks));
  } else {
    LAUNCH(launch_step_logits(in, g, ks));
  }
  FusedGemv gv{};
  gv.R = R;
  gv.t = t;
  gv.slots = S->fslots;
  gv.nslots = fused_slots_per_row(m->info.vocab);
  gv.tagged = tagged;
  gv.step = S->step;
  gv.out_tok = S->out_tok;
  gv.cur_tok = S->cur_tok;
  gv.finished = S->finished;
    gv.out_len = S->out_len;
  gv.out_key = S->out_key;
  gv.T = T;
  gv.stop_at_eos = stop_at_eos;
  gv.eos = m->info.eos_id;
  gv.pad = m->info.pad_id;
  gv.zero_acc = reinterpret_cast<int32_t*>(acc_w2);  // cleared as 2 nacc int32 words
  gv.zero_n = 2 * nacc;
  gv.emb_out = S->dec_x;
  gv.E = m->E;
  gv.c_emb = m->c_emb;
  gv.pe = m->pe;
  gv.d = d;
  gv.V = m->info.vocab;
  gv.P = m->info.max_pos;
  if (fold && !last_step && fold_ok(m)) return MNMT_OK;  // the next step's first layer commits
  LAUNCH(launch_greedy_commit_slots(gv, ch ? ch->last() : s));  // after the logits on their stream
  return MNMT_OK;
}

bool step_path_used(const mnmt_session* S, int R) {
  const mnmt_model* m = S->m;
  return !factored(m) && step_path_fits(R, m->info.d_model, m->dh, m->info.d_ffn, S->cfg.max_tgt_len, S->S);
}

// The 1-2 row path's input rows: embeddings of cur_tok at the position held
// by the device step counter.
int embed_step_input(mnmt_session* S, int R, hipStream_t s) {
  const mnmt_model* m = S->m;
  LAUNCH(launch_embed(S->cur_tok, R, 1, S->step, m->E, m->c_emb, m->pe, m->info.d_model, m->info.vocab, S->dec_x, s));
  return MNMT_OK;
}

// The greedy step for R rows on the fastest path that fits.
// On the 1-2 row path the input rows must be in dec_x (embed_step_input).
int greedy_step_any(mnmt_session* S, int R, int t, int stop_at_eos, float* logits_out, hipStream_t s,
                    bool fold = false, bool last = false, Chain* ch = nullptr) {
  if (step_path_used(S, R)) return greedy_step_v3(S, R, t, stop_at_eos, logits_out, s, fold, last, ch);
  if (R <= 8 && !factored(S->m)) return greedy_step_fused(S, R, t, stop_at_eos, logits_out, s);
  return greedy_step(S, R, stop_at_eos, logits_out, s);
}

// Step t of `steps`: from the second step on, the input rows come from the
// previous step's beam update, which also prepares them for the next one.
int beam_step(mnmt_session* S, int R, int W, int t, int steps, hipStream_t s) {
  const mnmt_model* m = S->m;
  // factorized embeddings embed their rows in the decoder (the beam update
  // prepares rows of the model width only)
  int rc = run_decoder_layers(S, R, W, true, s, t > 0 && !factored(m), t);
  if (rc) return rc;
  const int d = m->info.d_model, V = m->info.vocab;
  const int8_t* X;
  int K;
  if ((rc = logits_input(S, R, &X, &K, s))) return rc;
  EpiArgs e{MNMT_EPI_LOGITS, S->logits, V, 1.f, nullptr};
  LAUNCH(launch_qlinear(X, K, m->E, m->c_out, nullptr, R, K, V, e, s));
  BeamState st = S->beam;
  st.t_host = t;  // the graph replays the steps in this order
  LAUNCH(launch_beam_topk(S->logits, st, S->step, s));
  const LayerDev& L0 = m->dec[0];
  BeamNext nx{};
  nx.x = S->dec_x;
  nx.a = S->dec_a;
  nx.E = m->E;
  nx.c_emb = m->c_emb;
  nx.pe = m->pe;
  nx.d = d;
  nx.V = V;
  nx.P = m->info.max_pos;
  nx.steps = factored(m) ? 0 : steps;
  nx.do_ln = !m->info.ln_post;
  nx.g = L0.sa_ln.g;
  nx.b = L0.sa_ln.b;
  nx.eps = m->info.ln_eps;
  nx.inv_s = L0.qkv.inv_in;
  LAUNCH(launch_beam_update(st, S->step, nx, s));
  return MNMT_OK;
}

// All device work of a translate call after the inputs are in the session.
int enqueue_search(mnmt_session* S, const mnmt_search_cfg& sc, hipStream_t s) {
  int rc = run_encoder(S, s);
  if (rc) return rc;
  const mnmt_model* m = S->m;
  if (sc.beam == 1) {
    const int R = S->B;
    LAUNCH(launch_greedy_reset(S->slots, R, sc.max_steps, S->cur_tok, S->finished, S->out_len, S->step,
                               m->info.bos_id, S->fslots, fslots_words(m), S->epoch, s));
    if (step_path_used(S, R) && (rc = embed_step_input(S, R, s))) return rc;
    if (step_path_used(S, R) && chain_ok(m) && S->chain_on) {
      // the step kernels alternate between the caller's stream and the side
      // stream, each loading its weights while its predecessor runs
      MNMT_HIP(hipEventRecord(S->fork_ev, s));
      MNMT_HIP(hipStreamWaitEvent(S->side_stream, S->fork_ev, 0));
      Chain ch{{s, S->side_stream}, S->chain, S->chain_err};
      for (int t = 0; t < sc.max_steps && !rc; ++t)
        rc = greedy_step_any(S, R, t, sc.stop_at_eos, nullptr, s, true, t + 1 == sc.max_steps, &ch);
      // join the side stream whatever happened, so a capture can end cleanly
      MNMT_HIP(hipEventRecord(S->join_ev, S->side_stream));
      MNMT_HIP(hipStreamWaitEvent(s, S->join_ev, 0));
      if (rc) return rc;
    } else {
      for (int t = 0; t < sc.max_steps; ++t)
        if ((rc = greedy_step_any(S, R, t, sc.stop_at_eos, nullptr, s, true, t + 1 == sc.max_steps))) return rc;
    }
  } else {
    const int R = S->B * sc.beam;
    LAUNCH(launch_beam_reset(S->beam, S->step, s));
    for (int t = 0; t < sc.max_steps; ++t)
      if ((rc = beam_step(S, R, sc.beam, t, sc.max_steps, s))) return rc;
  }
  return MNMT_OK;
}

int check_ptr(const void* p, const char* what) {
  if (!p) return set_error(MNMT_E_INVALID_ARG, std::string(what) + " is null");
  if (reinterpret_cast<uintptr_t>(p) % 16) return set_error(MNMT_E_INVALID_ARG, std::string(what) + " is not 16-byte aligned");
  return MNMT_OK;
}

int load_batch(mnmt_session* S, const int32_t* d_src, const int32_t* d_len, int B, int S_max, hipStream_t s) {
  if (!S || !S->m) return set_error(MNMT_E_INVALID_ARG, "null session");
  int rc;
  if ((rc = check_ptr(d_src, "d_src")) || (rc = check_ptr(d_len, "d_len"))) return rc;
  if (B < 1 || S_max < 1) return set_error(MNMT_E_INVALID_ARG, "batch and source length must be positive");
  if (B > S->cfg.max_batch || S_max > S->cfg.max_src_len)
    return set_error(MNMT_E_CAPACITY, "batch or source length exceeds the session capacity");
  S->B = B;
  S->S = S_max;
  LAUNCH(launch_load_batch(d_src, d_len, S->src, S->len, B * S_max, B, S->enc_chain,
                           2 * S->m->info.n_enc * kChainSlotWords, s));
  return MNMT_OK;
}

}  // namespace
}  // namespace mnmt

using namespace mnmt;

extern "C" int mnmt_session_bytes(const mnmt_model* model, const mnmt_session_cfg* cfg, size_t* bytes) {
  int rc = validate_cfg(model, cfg);
  if (rc) return rc;
  if (!bytes) return set_error(MNMT_E_INVALID_ARG, "bytes is null");
  *bytes = make_plan(model, *cfg).total;
  return MNMT_OK;
}

extern "C" int mnmt_session_create(const mnmt_model* model, const mnmt_session_cfg* cfg, void* d_ws, size_t ws_bytes,
                                   mnmt_session** out) {
  int rc = validate_cfg(model, cfg);
  if (rc) return rc;
  if (!out) return set_error(MNMT_E_INVALID_ARG, "out is null");
  if (!d_ws || reinterpret_cast<uintptr_t>(d_ws) % 256)
    return set_error(MNMT_E_INVALID_ARG, "workspace must be non-null and 256-byte aligned");
  const Plan p = make_plan(model, *cfg);
  if (ws_bytes < p.total) return set_error(MNMT_E_INVALID_ARG, "workspace smaller than mnmt_session_bytes");
  auto* S = new mnmt_session();
  S->m = model;
  S->cfg = *cfg;
  S->R = cfg->max_batch * cfg->beam;
  uint8_t* base = static_cast<uint8_t*>(d_ws);
  auto at = [&](size_t off) { return static_cast<void*>(base + off); };
  const size_t d = model->info.d_model, BS = (size_t)cfg->max_batch * cfg->max_src_len, R = S->R,
               T = cfg->max_tgt_len, V = model->info.vocab;
  S->src = (int32_t*)at(p.src);
  S->len = (int32_t*)at(p.len);
  S->enc_x = (float*)at(p.enc_x);
  S->enc_a = (int8_t*)at(p.enc_a);
  S->enc_qkv = (int8_t*)at(p.enc_qkv);
  S->enc_h = (int8_t*)at(p.enc_h);
  S->enc_out = (int8_t*)at(p.enc_out);
  S->enc_x2 = (float*)at(p.enc_x2);
  S->logits = (float*)at(p.logits);
  for (size_t l = 0; l < p.cross_kv.size(); ++l) S->cross_kv.push_back((int8_t*)at(p.cross_kv[l]));
  S->dec_x = (float*)at(p.dec_x);
  S->dec_x2 = (float*)at(p.dec_x2);
  S->fslots = (unsigned long long*)at(p.fslots);
  S->enc_acc = (int32_t*)at(p.enc_acc);
  S->step_acc = (unsigned long long*)(S->fslots + 8 * (size_t)fused_slots_per_row((int)V));
  S->chain = (unsigned*)(S->step_acc + 3 * 2 * d);
  S->chain_err = (int*)at(p.chain_err);
  S->epoch = (unsigned*)at(p.epoch);
  S->step_x64 = (unsigned long long*)at(p.step_x64);
  S->enc_chain = (unsigned*)at(p.enc_chain);
  S->dec_a = (int8_t*)at(p.dec_a);
  S->dec_qkv = (int8_t*)at(p.dec_qkv);
  S->dec_q = (int8_t*)at(p.dec_q);
  S->dec_h = (int8_t*)at(p.dec_h);
  S->dec_u = (int8_t*)at(p.dec_u);
  S->dec_part = (int32_t*)at(p.dec_part);
  for (size_t l = 0; l < p.kc.size(); ++l) {
    S->kcache.push_back((int8_t*)at(p.kc[l]));
    S->vcache.push_back((int8_t*)at(p.vc[l]));
  }
  S->cur_tok = (int32_t*)at(p.cur_tok);
  S->step = (int*)at(p.step);
  S->slots = (unsigned long long*)at(p.slots);
  S->out_tok = (int32_t*)at(p.out_tok);
  S->finished = (int32_t*)at(p.finished);
    S->out_len = (int32_t*)at(p.out_len);
  S->out_key = (unsigned long long*)at(p.out_key);
  S->lp = (float*)at(p.lp);
  BeamState& st = S->beam;
  st.B = cfg->max_batch;
  st.W = cfg->beam;
  st.V = model->info.vocab;
  st.T = cfg->max_tgt_len;
  st.score = (float*)at(p.score);
  st.cand_score = (float*)at(p.cand_score);
  st.cand_tok = (int32_t*)at(p.cand_tok);
  st.tok_hist = (int32_t*)at(p.tok_hist);
  st.par_hist = (int32_t*)at(p.par_hist);
  st.hist = (int32_t*)at(p.hist);
  st.fin_score = (float*)at(p.fin_score);
  st.fin_len = (int32_t*)at(p.fin_len);
  st.fin_row = (int32_t*)at(p.fin_row);
  st.fin_count = (int32_t*)at(p.fin_count);
  st.done = (int32_t*)at(p.done);
  st.count = (int32_t*)at(p.beam_count);
  st.cur_tok = S->cur_tok;
  st.lp = S->lp;
  st.eos = model->info.eos_id;
  st.pad = model->info.pad_id;
  st.bos = model->info.bos_id;
  S->named["enc_out"] = {S->enc_out, BS * d};
  S->named["dec_x"] = {S->dec_x, 4 * R * d};
  S->named["logits"] = {S->logits, 4 * R * V};
  S->named["step"] = {S->step, 4};
  S->named["cur_tok"] = {S->cur_tok, 4 * R};
    S->named["chain_err"] = {S->chain_err, 4};
  S->named["out_key"] = {S->out_key, 8 * T * R};
  for (size_t l = 0; l < p.cross_kv.size(); ++l) {
    S->named["cross_kv." + std::to_string(l)] = {S->cross_kv[l], BS * 2 * d};
    S->named["kcache." + std::to_string(l)] = {S->kcache[l], R * T * d};
    S->named["vcache." + std::to_string(l)] = {S->vcache[l], R * T * d};
  }
  if (hipStreamCreateWithFlags(&S->capture_stream, hipStreamNonBlocking) != hipSuccess ||
      hipStreamCreateWithFlags(&S->side_stream, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&S->fork_ev, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&S->join_ev, hipEventDisableTiming) != hipSuccess) {
    mnmt_session_free(S);
    return set_error(MNMT_E_HIP, "could not create the session's streams and events");
  }
  // Tools that serialize kernel dispatches (a kernel tracer may) would leave
  // each chained kernel polling for a predecessor queued behind it until its
  // wait gives up; MNMT_SERIAL_STEPS=1 runs the steps in one stream instead.
  const char* serial = std::getenv("MNMT_SERIAL_STEPS");
  S->chain_on = !(serial && std::atoi(serial) != 0);
  // MNMT_COUNTED=0: flags and one-word accumulators between all the 1-2 row
  // step kernels instead of the counted hand-off (for comparison)
  const char* counted = std::getenv("MNMT_COUNTED");
  S->counted_on = !(counted && std::atoi(counted) == 0);
  // MNMT_MERGED_LAYERS=0: three launches per decoder layer of the 1-2 row
  // step instead of one (for comparison)
  const char* merged = std::getenv("MNMT_MERGED_LAYERS");
  S->merged_on = !(merged && std::atoi(merged) == 0);
  // MNMT_TAGGED=0: the step's first layer waits on the logits kernel's flags
  // instead of polling its tagged arg-max partials
  const char* tagged = std::getenv("MNMT_TAGGED");
  S->tagged_on = !(tagged && std::atoi(tagged) == 0);
  // MNMT_STEP_LAUNCH=1: the whole step of a two-layer decoder in one launch
  // instead of a launch per decoder layer and one for the logits (measured
  // slower: its logits blocks poll from the start of the step)
  const char* single = std::getenv("MNMT_STEP_LAUNCH");
  S->single_on = single && std::atoi(single) != 0;
  // MNMT_LN_FUSED=0: the batched decoder's pre-LN LayerNorms as kernels of
  // their own instead of in the prologue of the linear layer they feed
  const char* lnf = std::getenv("MNMT_LN_FUSED");
  S->ln_fused_on = !(lnf && std::atoi(lnf) == 0);
  // MNMT_QKV_FUSED=0: the batched pre-LN decoder's Q/K/V projection as a
  // GEMM of its own instead of inside the self-attention kernel
  const char* qkvf = std::getenv("MNMT_QKV_FUSED");
  S->qkv_fused_on = !(qkvf && std::atoi(qkvf) == 0);
  // the encoder accumulators start at zero (each encode leaves them so), the
  // chain error word too
  hipError_t h = hipMemsetAsync(S->enc_acc, 0, enc_acc_bytes(d), S->capture_stream);
  if (h == hipSuccess) h = hipMemsetAsync(S->chain_err, 0, sizeof(int), S->capture_stream);
  // row tags start at epoch 1, so the zeroed words never match
  if (h == hipSuccess) h = hipMemsetAsync(S->epoch, 0, sizeof(unsigned), S->capture_stream);
  if (h == hipSuccess)
    h = hipMemsetAsync(S->step_x64, 0, 8 * 3 * (size_t)model->info.n_dec * 2 * d, S->capture_stream);
  if (h == hipSuccess) h = hipStreamSynchronize(S->capture_stream);
  if (h != hipSuccess) {
    mnmt_session_free(S);
    return hip_error(h, "clearing the encoder accumulators");
  }
  *out = S;
  return MNMT_OK;
}

extern "C" void mnmt_session_free(mnmt_session* S) {
  if (!S) return;
  for (auto& g : S->graphs) (void)hipGraphExecDestroy(g.second);
  if (S->capture_stream) (void)hipStreamDestroy(S->capture_stream);
  if (S->side_stream) (void)hipStreamDestroy(S->side_stream);
  if (S->fork_ev) (void)hipEventDestroy(S->fork_ev);
  if (S->join_ev) (void)hipEventDestroy(S->join_ev);
  delete S;
}

extern "C" int mnmt_session_status(mnmt_session* S, void* stream) {
  if (!S) return set_error(MNMT_E_INVALID_ARG, "null session");
  hipStream_t s = as_stream(stream);
  int err = 0;
  MNMT_HIP(hipMemcpyAsync(&err, S->chain_err, sizeof(int), hipMemcpyDeviceToHost, s));
  MNMT_HIP(hipStreamSynchronize(s));
  if (!err) return MNMT_OK;
  MNMT_HIP(hipMemsetAsync(S->chain_err, 0, sizeof(int), s));
  MNMT_HIP(hipStreamSynchronize(s));
  return set_error(MNMT_E_TIMEOUT,
                   "a kernel of a chained batch-1 translation gave up waiting for its predecessor; the results "
                   "since the last status check are invalid (their lengths read -1)");
}

extern "C" int mnmt_session_tensor(const mnmt_session* S, const char* name, void** d_ptr, size_t* bytes) {
  if (!S || !name || !d_ptr) return set_error(MNMT_E_INVALID_ARG, "null argument");
  auto it = S->named.find(name);
  if (it == S->named.end()) return set_error(MNMT_E_INVALID_ARG, std::string("no session tensor ") + name);
  *d_ptr = it->second.first;
  if (bytes) *bytes = it->second.second;
  return MNMT_OK;
}

extern "C" int mnmt_encode(mnmt_session* S, const int32_t* d_src, const int32_t* d_len, int B, int S_max,
                           void* stream) {
  hipStream_t s = as_stream(stream);
  int rc = load_batch(S, d_src, d_len, B, S_max, s);
  if (rc) return rc;
  S->W = 1;
  if ((rc = run_encoder(S, s))) return rc;
  const mnmt_model* m = S->m;
  LAUNCH(launch_greedy_reset(S->slots, B, S->cfg.max_tgt_len, S->cur_tok, S->finished, S->out_len, S->step,
                             m->info.bos_id, S->fslots, fslots_words(m), S->epoch, s));
  S->encoded = true;
  S->host_step = 0;
  return MNMT_OK;
}

extern "C" int mnmt_decode_step(mnmt_session* S, const int32_t* d_prev, int32_t* d_next, float* d_logits,
                                void* stream) {
    if (!S) return set_error(MNMT_E_INVALID_ARG, "null session");
  if (S->cfg.beam > 1)
    return set_error(MNMT_E_UNSUPPORTED, "decode_step is the greedy step; beam sessions search through mnmt_translate");
  if (!S->encoded) return set_error(MNMT_E_INVALID_ARG, "decode_step needs a session after mnmt_encode");
  if (S->host_step >= S->cfg.max_tgt_len) return set_error(MNMT_E_CAPACITY, "decode step beyond max_tgt_len");
  int rc;
  if (d_prev && (rc = check_ptr(d_prev, "d_prev"))) return rc;
  if ((rc = check_ptr(d_next, "d_next"))) return rc;
  if (d_logits && (rc = check_ptr(d_logits, "d_logits"))) return rc;
  hipStream_t s = as_stream(stream);
  const int R = S->B;
  if (d_prev) LAUNCH(launch_copy_i32(d_prev, S->cur_tok, R, s));
  if (step_path_used(S, R) && (rc = embed_step_input(S, R, s))) return rc;
  if ((rc = greedy_step_any(S, R, S->host_step, 0, d_logits, s))) return rc;
  LAUNCH(launch_copy_i32(S->cur_tok, d_next, R, s));
  ++S->host_step;
  return MNMT_OK;
}

extern "C" int mnmt_translate(mnmt_session* S, const int32_t* d_src, const int32_t* d_len, int B, int S_max,
                              const mnmt_search_cfg* sc, int32_t* d_out, int32_t* d_out_len, float* d_score,
                              void* stream) {
  if (!S || !sc) return set_error(MNMT_E_INVALID_ARG, "null session or search config");
  int rc;
  if ((rc = check_ptr(d_out, "d_out")) || (rc = check_ptr(d_out_len, "d_out_len"))) return rc;
  if (d_score && (rc = check_ptr(d_score, "d_score"))) return rc;
  if (sc->beam < 1 || sc->beam > S->cfg.beam || sc->max_steps < 1 || sc->max_steps > S->cfg.max_tgt_len)
    return set_error(MNMT_E_CAPACITY, "beam or max_steps exceeds the session capacity");
  if (sc->beam > 1 && sc->beam != S->cfg.beam)
    return set_error(MNMT_E_UNSUPPORTED, "beam search runs at the session's beam width");
  if (sc->beam > 1 && !std::isfinite(sc->len_penalty_alpha))
    return set_error(MNMT_E_INVALID_ARG, "length penalty exponent must be finite");
  hipStream_t s = as_stream(stream);
  if ((rc = load_batch(S, d_src, d_len, B, S_max, s))) return rc;
  S->W = sc->beam;
  S->encoded = false;  // decode_step state is not kept across a translate
  if (sc->beam > 1) {
    S->beam.B = B;  // sentences of this call
    // length penalties ((5 + L) / 6)^alpha for L = 0..max_tgt_len, in double,
    // handed to the device in a kernel's arguments (no copy, no host wait)
    LpTable lp{};
    lp.n = S->cfg.max_tgt_len + 1;
    for (int L = 0; L < lp.n; ++L)
      lp.v[L] = (float)std::pow((5.0 + (double)L) / 6.0, (double)sc->len_penalty_alpha);
    LAUNCH(launch_fill_lp(lp, S->lp, s));
  }
  if (sc->use_graph) {
    const std::string key = std::to_string(B) + "," + std::to_string(S_max) + "," + std::to_string(sc->beam) + "," +
                            std::to_string(sc->max_steps) + "," + std::to_string(sc->stop_at_eos);
    auto it = S->graphs.find(key);
    if (it == S->graphs.end()) {
      MNMT_HIP(hipStreamBeginCapture(S->capture_stream, hipStreamCaptureModeRelaxed));
      rc = enqueue_search(S, *sc, S->capture_stream);
      hipGraph_t graph = nullptr;
      const hipError_t ec = hipStreamEndCapture(S->capture_stream, &graph);
      if (rc != MNMT_OK) {
        if (graph) (void)hipGraphDestroy(graph);
        return rc;
      }
      if (ec != hipSuccess) return hip_error(ec, "hipStreamEndCapture");
      hipGraphExec_t exec = nullptr;
      const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (ei != hipSuccess) return hip_error(ei, "hipGraphInstantiate");
      // the executable's device-side state now, not at its first launch
      const hipError_t eu = hipGraphUpload(exec, s);
      if (eu != hipSuccess) {
        (void)hipGraphExecDestroy(exec);
        return hip_error(eu, "hipGraphUpload");
      }
      it = S->graphs.emplace(key, exec).first;
    }
    MNMT_HIP(hipGraphLaunch(it->second, s));
  } else {
    if ((rc = enqueue_search(S, *sc, s))) return rc;
  }
  if (sc->beam == 1) {
    LAUNCH(launch_greedy_output(S->out_tok, S->out_len, B, sc->max_steps, d_out, d_out_len, S->chain_err, s));
  } else {
    LAUNCH(launch_beam_finalize(S->beam, sc->max_steps, d_out, d_out_len, d_score, S->chain_err, s));
  }
  return MNMT_OK;
}
