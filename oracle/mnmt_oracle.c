/*
 * mnmt_oracle.c -- plain, slow, scalar CPU oracle for the INT8
 * encoder-decoder inference path of MobileNMT (arXiv 2306.04235).
 *
 * TEST INFRASTRUCTURE: only the tests, the smoke check and the benchmark's
 * CPU-baseline leg call this code.  It is independent of the GPU library.
 *
 * What is computed, and where the paper states it:
 *   - Transformer encoder-decoder: self-attention, cross-attention and a ReLU
 *     FFN with residual connections (Appendix A, the self-weight, self-sum and
 *     FFN equations); layer normalization at the sublayer input (Appendix A
 *     and Appendix D, "Setups"), or after the residual add for post-LN models.
 *   - One shared vocabulary embedding for source input, target input and the
 *     output projection (Appendix D; "Embed x1" in the model-settings tables).
 *   - Quantizers (Section 3.2, quantizer figure): int8 inputs of every linear
 *     layer (LN output, attention context, ReLU output), int8 weights, int8
 *     Q/K/V; biases, residual stream, attention scores and softmax output in
 *     full precision; a learnable weight gamma on each sublayer's residual.
 *   - 8-bit integer GEMM (Section 4.1).
 *   - Cross-layer parameter sharing (Section 2.2, Encoder/Decoder
 *     Compression) and embedding factorization (Section 2.1, Embedding
 *     Compression) as model-file options.
 *   - Greedy search as used by the paper's engine (Appendix D); beam search
 *     as the paper's default evaluation decoder (ablation table).
 *
 * Where the paper is silent the readings below are used; each is listed with
 * its justification in the project's design notes:
 *   R1  fp32 everywhere outside the integer GEMMs; RNE; no contraction.
 *   R2  every fp32 sum over n terms is "wave64 order": 64 interleaved partial
 *       sums (term i goes to partial i mod 64, ascending i, starting at +0),
 *       then combined by halving: p[l] += p[l + off] for off = 32..1 --
 *       except the sum over the vocabulary in beam search's log-sum-exp
 *       (R2b, orc_canon_vocab_sum): 512 partials fed four consecutive terms
 *       at a time, halving within each run of 64, then a fixed tree of 8.
 *   R3  quantize: q = clamp(rint(y * (1/s)), -127, 127), 1/s rounded once.
 *   R4  folded constants computed in double, rounded once to fp32.
 *   R5  LayerNorm: biased variance, eps from the model file, affine g/b.
 *   R6  attention scale 1/sqrt(d_head); masked keys are skipped.
 *   R7  exp/log from Cody-Waite reduction + truncated series (orc_exp/orc_log).
 *   R8  beam search rules in translate_one_beam().
 *   R9  4-bit weights (the paper's W-E-A 4-8-8 setting, Table on quantization
 *       bit widths): per-row symmetric codes in [-7, 7], stored packed in the
 *       model file and unpacked here to the same int8 codes, so the integer
 *       GEMM and everything after it are unchanged.
 */
#include "mnmt_oracle.h"

#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Canonical fp32 primitives                                                 */
/* ------------------------------------------------------------------------- */

/* R2: the one summation order used for every fp32 sum. */
float orc_canon_sum(const float* x, int n) {
  float p[64];
  for (int l = 0; l < 64; ++l) p[l] = 0.0f;
  for (int i = 0; i < n; ++i) p[i % 64] = p[i % 64] + x[i];
  for (int off = 32; off >= 1; off /= 2)
    for (int l = 0; l < off; ++l) p[l] = p[l] + p[l + off];
  return p[0];
}

/* Sum of squares in the same order; each partial accumulates with one fma. */
float orc_canon_sum_squares(const float* x, int n) {
  float p[64];
  for (int l = 0; l < 64; ++l) p[l] = 0.0f;
  for (int i = 0; i < n; ++i) p[i % 64] = fmaf(x[i], x[i], p[i % 64]);
  for (int off = 32; off >= 1; off /= 2)
    for (int l = 0; l < off; ++l) p[l] = p[l] + p[l + off];
  return p[0];
}

/* R2b: the sum over the vocabulary in the log-sum-exp of beam search.  The
 * terms are dealt to 512 partial sums in groups of four consecutive terms
 * (term i goes to partial (i / 4) mod 512, ascending i, partials start at
 * +0); each run of 64 partials (64 w .. 64 w + 63) is combined by halving as
 * in R2, giving g_w; then ((g0 + g1) + (g2 + g3)) + ((g4 + g5) + (g6 + g7)). */
float orc_canon_vocab_sum(const float* x, int n) {
  float p[512];
  for (int j = 0; j < 512; ++j) p[j] = 0.0f;
  for (int i = 0; i < n; ++i) p[(i / 4) % 512] = p[(i / 4) % 512] + x[i];
  float g[8];
  for (int w = 0; w < 8; ++w) {
    float* q = p + 64 * w;
    for (int off = 32; off >= 1; off /= 2)
      for (int l = 0; l < off; ++l) q[l] = q[l] + q[l + off];
    g[w] = q[0];
  }
  return ((g[0] + g[1]) + (g[2] + g[3])) + ((g[4] + g[5]) + (g[6] + g[7]));
}

/* R3: uniform symmetric 8-bit quantization (Section 3.2; rounding to the
 * nearest integer as in the quantization equation of Appendix B, with ties to
 * even).  Codes are limited to [-127, 127]. */
int8_t orc_quantize(float y, float inv_s) {
  float r = rintf(y * inv_s);
  if (r < -127.0f) r = -127.0f;
  if (r > 127.0f) r = 127.0f;
  return (int8_t)r;
}

/* R7: e^x for x <= 0.  x = k ln2 + r with k = rint(x log2 e) and r formed by a
 * two-part (Cody-Waite) reduction; e^r from its Taylor series truncated after
 * the r^7 term, in Horner form; e^x = 2^k e^r.  Inputs below -87 give 0. */
float orc_exp(float x) {
  const float log2e = 1.44269504088896341f;
  const float ln2_hi = 0x1.62e400p-1f; /* ln 2 with its low 12 bits cleared */
  const float ln2_lo = (float)(0.69314718055994530942 - 0.693145751953125);
  if (x < -87.0f) return 0.0f;
  float k = rintf(x * log2e);
  float r = fmaf(-k, ln2_hi, x);
  r = fmaf(-k, ln2_lo, r);
  float p = (float)(1.0 / 5040.0);
  p = fmaf(p, r, (float)(1.0 / 720.0));
  p = fmaf(p, r, (float)(1.0 / 120.0));
  p = fmaf(p, r, (float)(1.0 / 24.0));
  p = fmaf(p, r, (float)(1.0 / 6.0));
  p = fmaf(p, r, 0.5f);
  p = fmaf(p, r, 1.0f);
  p = fmaf(p, r, 1.0f);
  return ldexpf(p, (int)k);
}

/* R7: ln x for normal x > 0.  x = m 2^e with m in [sqrt(1/2), sqrt(2));
 * ln m = 2 atanh(f), f = (m - 1)/(m + 1), from the odd series
 * 2f (1 + f^2/3 + f^4/5 + f^6/7 + f^8/9); ln x = e ln2 + ln m. */
float orc_log(float x) {
  const float ln2_hi = 0x1.62e400p-1f;
  const float ln2_lo = (float)(0.69314718055994530942 - 0.693145751953125);
  int e;
  float m = frexpf(x, &e); /* m in [0.5, 1) */
  if (m < 0.70710678118654752f) {
    m = m * 2.0f;
    e = e - 1;
  }
  float f = (m - 1.0f) / (m + 1.0f);
  float s = f * f;
  float p = (float)(1.0 / 9.0);
  p = fmaf(p, s, (float)(1.0 / 7.0));
  p = fmaf(p, s, (float)(1.0 / 5.0));
  p = fmaf(p, s, (float)(1.0 / 3.0));
  p = fmaf(p, s, 1.0f);
  float ln_m = (2.0f * f) * p;
  float ef = (float)e;
  return fmaf(ef, ln2_hi, fmaf(ef, ln2_lo, ln_m));
}

/* Apply orc_exp (fn 0) or orc_log (fn 1) to an array (for exhaustive sweeps). */
int orc_map(int fn, const float* x, int n, float* y) {
  if (fn < 0 || fn > 1 || n < 0) return ORC_E_ARG;
  for (int i = 0; i < n; ++i) y[i] = fn == 0 ? orc_exp(x[i]) : orc_log(x[i]);
  return ORC_OK;
}

/* GNMT-style length penalty ((5 + L) / 6)^alpha, computed in double. */
float orc_length_penalty(int L, float alpha) {
  return (float)pow((5.0 + (double)L) / 6.0, (double)alpha);
}

/* ------------------------------------------------------------------------- */
/* Integer GEMM and linear-layer epilogues (Section 4.1; quantizer figure)   */
/* ------------------------------------------------------------------------- */

/* Y[m][n] = sum_k X[m][k] * W[n][k], exact in int32 (|Y| <= 127^2 K). */
int orc_qgemm_i32(const int8_t* X, const int8_t* W, int M, int K, int N, int32_t* Y) {
  if (M < 0 || K <= 0 || N <= 0 || K > 65536) return ORC_E_ARG;
  for (int m = 0; m < M; ++m)
    for (int n = 0; n < N; ++n) {
      int32_t acc = 0;
      for (int k = 0; k < K; ++k) acc += (int32_t)X[(size_t)m * K + k] * (int32_t)W[(size_t)n * K + k];
      Y[(size_t)m * N + n] = acc;
    }
  return ORC_OK;
}

/* Linear layer with one of the epilogues of the quantizer figure:
 *   I32:       Y = acc
 *   I8:        Y = quant(fma(acc, scale[n], bias[n]))   (requant, folded scales)
 *   I8_RELU:   Y = quant(max(fma(acc, scale[n], bias[n]), 0))
 *   F32:       Y = fma(acc, scale[n], bias[n])          (dequant + full-precision bias)
 *   F32_RESID: Y = fma(gamma, Y, fma(acc, scale[n], bias[n]))  (gamma-weighted residual)
 *   LOGITS:    Y = acc * scale[n]                       (tied embedding, no bias)
 * For the I8 forms quant(y) = clamp(rint(y), -127, 127): the folded scale
 * already divides by the output scale. */
int orc_qlinear(const int8_t* X, const int8_t* W, int M, int K, int N, const float* scale,
                const float* bias, float gamma, int epilogue, void* Y) {
  if (M < 0 || K <= 0 || N <= 0) return ORC_E_ARG;
  for (int m = 0; m < M; ++m)
    for (int n = 0; n < N; ++n) {
      int32_t acc = 0;
      for (int k = 0; k < K; ++k) acc += (int32_t)X[(size_t)m * K + k] * (int32_t)W[(size_t)n * K + k];
      size_t o = (size_t)m * N + n;
      float a = (float)acc;
      switch (epilogue) {
        case ORC_EPI_I32: ((int32_t*)Y)[o] = acc; break;
        case ORC_EPI_I8: ((int8_t*)Y)[o] = orc_quantize(fmaf(a, scale[n], bias[n]), 1.0f); break;
        case ORC_EPI_I8_RELU: {
          float y = fmaf(a, scale[n], bias[n]);
          if (y < 0.0f) y = 0.0f;
          ((int8_t*)Y)[o] = orc_quantize(y, 1.0f);
          break;
        }
        case ORC_EPI_F32: ((float*)Y)[o] = fmaf(a, scale[n], bias[n]); break;
        case ORC_EPI_F32_RESID: {
          float* y = (float*)Y + o;
          *y = fmaf(gamma, *y, fmaf(a, scale[n], bias[n]));
          break;
        }
        case ORC_EPI_LOGITS: ((float*)Y)[o] = a * scale[n]; break;
        default: return ORC_E_ARG;
      }
    }
  return ORC_OK;
}

/* R4: folded requantization constants.  With x = s_in X, w = s_w W and an
 * output quantized by s_out, (x w + b) / s_out = acc (s_in s_w / s_out) + b / s_out. */
int orc_fold_requant(float s_in, const float* s_w, const float* b, float s_out, int N, float* scale,
                     float* bias) {
  for (int n = 0; n < N; ++n) {
    scale[n] = (float)((double)s_in * (double)s_w[n] / (double)s_out);
    bias[n] = (float)((double)b[n] / (double)s_out);
  }
  return ORC_OK;
}

/* R4: dequantization constant s_in s_w for full-precision outputs. */
int orc_fold_dequant(float s_in, const float* s_w, int N, float* scale) {
  for (int n = 0; n < N; ++n) scale[n] = (float)((double)s_in * (double)s_w[n]);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* LayerNorm (Appendix A: the sublayer input is layer-normalized)            */
/* ------------------------------------------------------------------------- */

/* R5: y = (x - mean) / sqrt(var + eps) * g + b, biased variance, evaluated as
 * delta = x - mu; y = fma(delta * rstd, g, b). */
static void layer_norm_row(const float* x, int d, const float* g, const float* b, float eps, float* y) {
  float* delta = (float*)malloc(sizeof(float) * (size_t)d);
  float inv_d = 1.0f / (float)d;
  float mu = orc_canon_sum(x, d) * inv_d;
  for (int i = 0; i < d; ++i) delta[i] = x[i] - mu;
  float var = orc_canon_sum_squares(delta, d) * inv_d;
  float rstd = 1.0f / sqrtf(var + eps);
  for (int i = 0; i < d; ++i) y[i] = fmaf(delta[i] * rstd, g[i], b[i]);
  free(delta);
}

int orc_layernorm_quant(const float* x, int rows, int d, const float* g, const float* b, float eps,
                        float inv_s, int8_t* q, float* y) {
  if (rows < 0 || d <= 0) return ORC_E_ARG;
  float* t = (float*)malloc(sizeof(float) * (size_t)d);
  for (int r = 0; r < rows; ++r) {
    layer_norm_row(x + (size_t)r * d, d, g, b, eps, t);
    for (int i = 0; i < d; ++i) {
      if (q) q[(size_t)r * d + i] = orc_quantize(t[i], inv_s);
      if (y) y[(size_t)r * d + i] = t[i];
    }
  }
  free(t);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Attention for one query row and one head (Appendix A, self-weight and     */
/* self-sum equations; quantizer figure (b))                                 */
/* ------------------------------------------------------------------------- */

/* q: [dh] codes; key t at K + t*ldk, value t at V + t*ldk (codes), t < n.
 *   s_t  = (q . k_t) * c_qk           c_qk = s_q s_k / sqrt(dh)
 *   p    = softmax(s) in fp32         (max-shifted, orc_exp, canonical sum)
 *   c_j  = sum_t p_t v_tj             ascending t, one fma per term
 *   out  = quant(c_j, c_pv)           c_pv = s_v / s_ctx                     */
int orc_attend(const int8_t* q, const int8_t* K, const int8_t* V, int n, int dh, int ldk,
               float c_qk, float c_pv, int8_t* out) {
  if (n <= 0 || dh <= 0) return ORC_E_ARG;
  float* s = (float*)malloc(sizeof(float) * (size_t)n);
  float* e = (float*)malloc(sizeof(float) * (size_t)n);
  for (int t = 0; t < n; ++t) {
    int32_t acc = 0;
    for (int j = 0; j < dh; ++j) acc += (int32_t)q[j] * (int32_t)K[(size_t)t * ldk + j];
    s[t] = (float)acc * c_qk;
  }
  float mx = s[0];
  for (int t = 1; t < n; ++t)
    if (s[t] > mx) mx = s[t];
  for (int t = 0; t < n; ++t) e[t] = orc_exp(s[t] - mx);
  float inv = 1.0f / orc_canon_sum(e, n);
  for (int t = 0; t < n; ++t) e[t] = e[t] * inv; /* p_t */
  for (int j = 0; j < dh; ++j) {
    float c = 0.0f;
    for (int t = 0; t < n; ++t) c = fmaf(e[t], (float)V[(size_t)t * ldk + j], c);
    out[j] = orc_quantize(c, c_pv);
  }
  free(s);
  free(e);
  return ORC_OK;
}

/* log-sum-exp of a row: max m, then m + ln(sum_v e^(z_v - m)), the sum over
 * the vocabulary in the R2b order. */
int orc_log_softmax_stats(const float* z, int n, float* max_out, float* lse_out) {
  if (n <= 0) return ORC_E_ARG;
  float mx = z[0];
  for (int v = 1; v < n; ++v)
    if (z[v] > mx) mx = z[v];
  float* e = (float*)malloc(sizeof(float) * (size_t)n);
  for (int v = 0; v < n; ++v) e[v] = orc_exp(z[v] - mx);
  float sum = orc_canon_vocab_sum(e, n);
  free(e);
  if (max_out) *max_out = mx;
  if (lse_out) *lse_out = mx + orc_log(sum);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Model file                                                                */
/* ------------------------------------------------------------------------- */

typedef struct {
  const int8_t* w; /* [N, K] */
  int8_t* w_own;   /* unpacked 4-bit weights (owned), else NULL */
  int N, K;
  const float* s_w;
  const float* b;
  float s_in, inv_in;
  float* scale; /* folded per-channel constants */
  float* bias;
} linear_t;

typedef struct {
  const float* g;
  const float* b;
} ln_t;

typedef struct {
  ln_t ln;
  linear_t qkv, o; /* self-attention: qkv [3d, d], o [d, d] */
  linear_t q, kv;  /* cross-attention: q [d, d], kv [2d, d] */
  float gamma, c_qk, c_pv;
} attn_t;

typedef struct {
  ln_t ln;
  linear_t w1, w2;
  float gamma;
} ffn_t;

typedef struct {
  attn_t sa, ca;
  ffn_t ff;
  int alias; /* this layer reuses another layer's parameters (owns nothing) */
} layer_t;

struct orc_model {
  int d, h, dh, F, Le, Ld, V, P, post;
  int pad_id, bos_id, eos_id, unk_id;
  float eps;
  unsigned char* blob;
  size_t nbytes;
  int n_tensors;
  const int8_t* E;
  const float* s_E;
  const float* pe;
  float* c_emb;
  float* c_out;
  layer_t* enc;
  layer_t* dec;
  ln_t enc_ln, dec_ln;
  float s_enc, s_fin, inv_enc, inv_fin;
  /* factorized embedding (Section 2.1): E is [V, Ef], P [d, Ef] maps it to the
   * model width; Ef = 0 when the embedding has the model width */
  int Ef;
  const int8_t* Pw;
  linear_t proj_out; /* Pw transposed [Ef, d]: the final rows back to Ef codes */
  float s_P;
  float s_emb_out; /* scale of the output projection's int8 input: s_fin, or s_u when factorized */
};

static uint32_t rd_u32(const unsigned char* p) {
  uint32_t v;
  memcpy(&v, p, 4);
  return v;
}

/* The dimensions of a tensor of any type (0 if absent). */
static void tensor_dims(const orc_model* m, const char* name, uint32_t* d0, uint32_t* d1) {
  *d0 = *d1 = 0;
  for (int i = 0; i < m->n_tensors; ++i) {
    const unsigned char* e = m->blob + 64 + (size_t)i * 64;
    char nm[41];
    memcpy(nm, e, 40);
    nm[40] = 0;
    if (strcmp(nm, name) != 0) continue;
    memcpy(d0, e + 48, 4);
    memcpy(d1, e + 52, 4);
    return;
  }
}

/* Look up a tensor by name; check dtype (1 int8, 2 fp32, 3 packed 4-bit)
 * and shape. */
static const void* find_tensor(const orc_model* m, const char* name, uint32_t dtype, uint32_t d0,
                               uint32_t d1) {
  for (int i = 0; i < m->n_tensors; ++i) {
    const unsigned char* e = m->blob + 64 + (size_t)i * 64;
    char nm[41];
    memcpy(nm, e, 40);
    nm[40] = 0;
    if (strcmp(nm, name) != 0) continue;
    uint32_t dt = rd_u32(e + 40), a = rd_u32(e + 48), b = rd_u32(e + 52);
    uint64_t off;
    memcpy(&off, e + 56, 8);
    if (dt != dtype || a != d0 || b != d1) return NULL;
    if (dtype == 3 && b % 16 != 0) return NULL;
    uint64_t bytes = dtype == 3 ? (uint64_t)a * b / 2 : (uint64_t)a * b * (dtype == 1 ? 1u : 4u);
    if (off % 256 != 0 || off + bytes > m->nbytes) return NULL;
    return m->blob + off;
  }
  return NULL;
}

static int scalar(const orc_model* m, const char* name, float* v) {
  const float* p = (const float*)find_tensor(m, name, 2, 1, 1);
  if (!p || !(p[0] > 0.0f) || !isfinite(p[0])) return ORC_E_MODEL;
  *v = p[0];
  return ORC_OK;
}

/* A linear layer's tensors "<pfx>.w", ".sw", ".b", and either ".sin" or the
 * given input scale.  out_scales (n_blocks of them) select the int8 output
 * form; NULL selects the full-precision output form. */
static int load_linear(orc_model* m, linear_t* L, const char* pfx, int N, int K, const float* s_in_given,
                       const float* out_scales, int n_blocks) {
  char nm[64];
  L->N = N;
  L->K = K;
  snprintf(nm, sizeof nm, "%s.w", pfx);
  L->w = (const int8_t*)find_tensor(m, nm, 1, (uint32_t)N, (uint32_t)K);
  if (!L->w) {
    /* 4-bit: in each group of 16 codes of a row, byte i (i < 8) holds code i
     * in its low nibble and code i + 8 in its high nibble, each plus 8 */
    const unsigned char* p = (const unsigned char*)find_tensor(m, nm, 3, (uint32_t)N, (uint32_t)K);
    if (p) {
      L->w_own = (int8_t*)malloc((size_t)N * K);
      if (!L->w_own) return ORC_E_NOMEM;
      for (size_t r = 0; r < (size_t)N; ++r)
        for (int g = 0; g < K / 16; ++g)
          for (int i = 0; i < 8; ++i) {
            const unsigned char byte = p[r * (size_t)K / 2 + (size_t)g * 8 + i];
            L->w_own[r * K + 16 * g + i] = (int8_t)((int)(byte & 15) - 8);
            L->w_own[r * K + 16 * g + 8 + i] = (int8_t)((int)(byte >> 4) - 8);
          }
      L->w = L->w_own;
    }
  }
  snprintf(nm, sizeof nm, "%s.sw", pfx);
  L->s_w = (const float*)find_tensor(m, nm, 2, (uint32_t)N, 1);
  snprintf(nm, sizeof nm, "%s.b", pfx);
  L->b = (const float*)find_tensor(m, nm, 2, (uint32_t)N, 1);
  if (!L->w || !L->s_w || !L->b) return ORC_E_MODEL;
  for (int n = 0; n < N; ++n)
    if (!(L->s_w[n] > 0.0f) || !isfinite(L->s_w[n]) || !isfinite(L->b[n])) return ORC_E_MODEL;
  if (s_in_given) {
    L->s_in = *s_in_given;
  } else {
    snprintf(nm, sizeof nm, "%s.sin", pfx);
    if (scalar(m, nm, &L->s_in)) return ORC_E_MODEL;
  }
  L->inv_in = (float)(1.0 / (double)L->s_in);
  L->scale = (float*)malloc(sizeof(float) * (size_t)N);
  L->bias = (float*)malloc(sizeof(float) * (size_t)N);
  if (!L->scale || !L->bias) return ORC_E_NOMEM;
  if (out_scales) {
    int blk = N / n_blocks;
    for (int i = 0; i < n_blocks; ++i)
      orc_fold_requant(L->s_in, L->s_w + i * blk, L->b + i * blk, out_scales[i], blk, L->scale + i * blk,
                       L->bias + i * blk);
  } else {
    orc_fold_dequant(L->s_in, L->s_w, N, L->scale);
    for (int n = 0; n < N; ++n) L->bias[n] = L->b[n];
  }
  return ORC_OK;
}

static int load_ln(orc_model* m, ln_t* ln, const char* pfx) {
  char nm[64];
  snprintf(nm, sizeof nm, "%s.g", pfx);
  ln->g = (const float*)find_tensor(m, nm, 2, (uint32_t)m->d, 1);
  snprintf(nm, sizeof nm, "%s.b", pfx);
  ln->b = (const float*)find_tensor(m, nm, 2, (uint32_t)m->d, 1);
  return (ln->g && ln->b) ? ORC_OK : ORC_E_MODEL;
}

static int load_out_scales(orc_model* m, const char* name, int n, float* out) {
  const float* p = (const float*)find_tensor(m, name, 2, (uint32_t)n, 1);
  if (!p) return ORC_E_MODEL;
  for (int i = 0; i < n; ++i) {
    if (!(p[i] > 0.0f) || !isfinite(p[i])) return ORC_E_MODEL;
    out[i] = p[i];
  }
  return ORC_OK;
}

static int load_layer(orc_model* m, layer_t* L, const char* side, int l, int is_dec) {
  char pfx[64], nm[64];
  int d = m->d, F = m->F;
  float s3[3], s_ctx;
  /* Cross-layer parameter sharing (Section 2.2, Encoder/Decoder Compression):
   * an int8 tensor "<side>.<l>.share" = j (0 <= j < l) makes layer l run with
   * every parameter of layer j of the same stack. */
  snprintf(nm, sizeof nm, "%s.%d.share", side, l);
  {
    const int8_t* sh = (const int8_t*)find_tensor(m, nm, 1, 1, 1);
    if (sh) {
      const int j = sh[0];
      if (j < 0 || j >= l) return ORC_E_MODEL;
      *L = (is_dec ? m->dec : m->enc)[j];
      L->alias = 1;
      return ORC_OK;
    }
  }
  /* self-attention */
  snprintf(pfx, sizeof pfx, "%s.%d.sa.ln", side, l);
  if (load_ln(m, &L->sa.ln, pfx)) return ORC_E_MODEL;
  snprintf(nm, sizeof nm, "%s.%d.sa.qkv.sout", side, l);
  if (load_out_scales(m, nm, 3, s3)) return ORC_E_MODEL;
  snprintf(pfx, sizeof pfx, "%s.%d.sa.qkv", side, l);
  if (load_linear(m, &L->sa.qkv, pfx, 3 * d, d, NULL, s3, 3)) return ORC_E_MODEL;
  snprintf(pfx, sizeof pfx, "%s.%d.sa.o", side, l);
  if (load_linear(m, &L->sa.o, pfx, d, d, NULL, NULL, 1)) return ORC_E_MODEL;
  s_ctx = L->sa.o.s_in;
  L->sa.c_qk = (float)((double)s3[0] * (double)s3[1] / sqrt((double)m->dh));
  L->sa.c_pv = (float)((double)s3[2] / (double)s_ctx);
  snprintf(nm, sizeof nm, "%s.%d.sa.gamma", side, l);
  {
    const float* g = (const float*)find_tensor(m, nm, 2, 1, 1);
    if (!g || !isfinite(g[0])) return ORC_E_MODEL;
    L->sa.gamma = g[0];
  }
  if (is_dec) {
    float sq[1], skv[2];
    snprintf(pfx, sizeof pfx, "%s.%d.ca.ln", side, l);
    if (load_ln(m, &L->ca.ln, pfx)) return ORC_E_MODEL;
    snprintf(nm, sizeof nm, "%s.%d.ca.q.sout", side, l);
    if (load_out_scales(m, nm, 1, sq)) return ORC_E_MODEL;
    snprintf(pfx, sizeof pfx, "%s.%d.ca.q", side, l);
    if (load_linear(m, &L->ca.q, pfx, d, d, NULL, sq, 1)) return ORC_E_MODEL;
    snprintf(nm, sizeof nm, "%s.%d.ca.kv.sout", side, l);
    if (load_out_scales(m, nm, 2, skv)) return ORC_E_MODEL;
    snprintf(pfx, sizeof pfx, "%s.%d.ca.kv", side, l);
    if (load_linear(m, &L->ca.kv, pfx, 2 * d, d, &m->s_enc, skv, 2)) return ORC_E_MODEL;
    snprintf(pfx, sizeof pfx, "%s.%d.ca.o", side, l);
    if (load_linear(m, &L->ca.o, pfx, d, d, NULL, NULL, 1)) return ORC_E_MODEL;
    L->ca.c_qk = (float)((double)sq[0] * (double)skv[0] / sqrt((double)m->dh));
    L->ca.c_pv = (float)((double)skv[1] / (double)L->ca.o.s_in);
    snprintf(nm, sizeof nm, "%s.%d.ca.gamma", side, l);
    const float* g = (const float*)find_tensor(m, nm, 2, 1, 1);
    if (!g || !isfinite(g[0])) return ORC_E_MODEL;
    L->ca.gamma = g[0];
  }
  /* FFN: W1 output (ReLU) quantized with w1.sout, which is W2's input scale */
  {
    float sh[1];
    snprintf(pfx, sizeof pfx, "%s.%d.ff.ln", side, l);
    if (load_ln(m, &L->ff.ln, pfx)) return ORC_E_MODEL;
    snprintf(nm, sizeof nm, "%s.%d.ff.w1.sout", side, l);
    if (load_out_scales(m, nm, 1, sh)) return ORC_E_MODEL;
    snprintf(pfx, sizeof pfx, "%s.%d.ff.w1", side, l);
    if (load_linear(m, &L->ff.w1, pfx, F, d, NULL, sh, 1)) return ORC_E_MODEL;
    snprintf(pfx, sizeof pfx, "%s.%d.ff.w2", side, l);
    if (load_linear(m, &L->ff.w2, pfx, d, F, &sh[0], NULL, 1)) return ORC_E_MODEL;
    snprintf(nm, sizeof nm, "%s.%d.ff.gamma", side, l);
    const float* g = (const float*)find_tensor(m, nm, 2, 1, 1);
    if (!g || !isfinite(g[0])) return ORC_E_MODEL;
    L->ff.gamma = g[0];
  }
  return ORC_OK;
}

static void free_linear(linear_t* L) {
  free(L->scale);
  free(L->bias);
  free(L->w_own);
}

void orc_model_free(orc_model* m) {
  if (!m) return;
  for (int l = 0; m->enc && l < m->Le; ++l) {
    if (m->enc[l].alias) continue;
    free_linear(&m->enc[l].sa.qkv);
    free_linear(&m->enc[l].sa.o);
    free_linear(&m->enc[l].ff.w1);
    free_linear(&m->enc[l].ff.w2);
  }
  for (int l = 0; m->dec && l < m->Ld; ++l) {
    if (m->dec[l].alias) continue;
    free_linear(&m->dec[l].sa.qkv);
    free_linear(&m->dec[l].sa.o);
    free_linear(&m->dec[l].ca.q);
    free_linear(&m->dec[l].ca.kv);
    free_linear(&m->dec[l].ca.o);
    free_linear(&m->dec[l].ff.w1);
    free_linear(&m->dec[l].ff.w2);
  }
  free(m->proj_out.scale);
  free(m->proj_out.bias);
  free(m->proj_out.w_own);
  free(m->enc);
  free(m->dec);
  free(m->c_emb);
  free(m->c_out);
  free(m->blob);
  free(m);
}

int orc_model_load(const void* blob, size_t nbytes, orc_model** out) {
  if (!blob || !out || nbytes < 64) return ORC_E_ARG;
  const unsigned char* p = (const unsigned char*)blob;
  if (memcmp(p, "MNMT", 4) != 0 || rd_u32(p + 4) != 1) return ORC_E_MODEL;
  orc_model* m = (orc_model*)calloc(1, sizeof(orc_model));
  if (!m) return ORC_E_NOMEM;
  m->blob = (unsigned char*)malloc(nbytes);
  if (!m->blob) {
    free(m);
    return ORC_E_NOMEM;
  }
  memcpy(m->blob, blob, nbytes);
  m->nbytes = nbytes;
  m->d = (int)rd_u32(p + 8);
  m->h = (int)rd_u32(p + 12);
  m->F = (int)rd_u32(p + 16);
  m->Le = (int)rd_u32(p + 20);
  m->Ld = (int)rd_u32(p + 24);
  m->V = (int)rd_u32(p + 28);
  m->P = (int)rd_u32(p + 32);
  m->post = (int)rd_u32(p + 36);
  m->pad_id = (int)rd_u32(p + 40);
  m->bos_id = (int)rd_u32(p + 44);
  m->eos_id = (int)rd_u32(p + 48);
  m->unk_id = (int)rd_u32(p + 52);
  memcpy(&m->eps, p + 56, 4);
  m->n_tensors = (int)rd_u32(p + 60);
  int rc = ORC_E_MODEL;
  if (m->d <= 0 || m->h <= 0 || m->d % m->h != 0 || m->F <= 0 || m->Le < 1 || m->Ld < 1 || m->V < 5 ||
      m->P < 1 || m->post > 1 || !(m->eps > 0.0f) || m->n_tensors <= 0 ||
      (size_t)64 + (size_t)m->n_tensors * 64 > nbytes)
    goto fail;
  if (m->pad_id < 0 || m->pad_id >= m->V || m->bos_id < 0 || m->bos_id >= m->V || m->eos_id < 0 ||
      m->eos_id >= m->V || m->unk_id < 0 || m->unk_id >= m->V)
    goto fail;
  m->dh = m->d / m->h;
  if (scalar(m, "enc.sout", &m->s_enc) || scalar(m, "dec.sout", &m->s_fin)) goto fail;
  m->s_emb_out = m->s_fin;
  {
    /* factorized embedding: emb.proj.w [d, Ef] with a per-tensor scale (the
     * matrix serves in both orientations) and the output side's scale s_u */
    uint32_t p0, p1;
    tensor_dims(m, "emb.proj.w", &p0, &p1);
    if (p0 || p1) {
      float s_u;
      m->Pw = (const int8_t*)find_tensor(m, "emb.proj.w", 1, (uint32_t)m->d, p1);
      if (!m->Pw || p1 < 4 || p1 % 4 || p1 > (uint32_t)m->d) goto fail;
      if (scalar(m, "emb.proj.sw", &m->s_P) || scalar(m, "emb.proj.sout", &s_u)) goto fail;
      m->Ef = (int)p1;
      linear_t* L = &m->proj_out;
      L->N = m->Ef;
      L->K = m->d;
      L->w_own = (int8_t*)malloc((size_t)m->d * m->Ef);
      L->scale = (float*)malloc(sizeof(float) * (size_t)m->Ef);
      L->bias = (float*)malloc(sizeof(float) * (size_t)m->Ef);
      if (!L->w_own || !L->scale || !L->bias) {
        rc = ORC_E_NOMEM;
        goto fail;
      }
      for (int n = 0; n < m->d; ++n)
        for (int k = 0; k < m->Ef; ++k) L->w_own[(size_t)k * m->d + n] = m->Pw[(size_t)n * m->Ef + k];
      L->w = L->w_own;
      /* u = requant(a . P) with a = s_fin codes, P = s_P codes, u = s_u codes */
      for (int k = 0; k < m->Ef; ++k) {
        L->scale[k] = (float)((double)m->s_fin * (double)m->s_P / (double)s_u);
        L->bias[k] = 0.0f;
      }
      m->s_emb_out = s_u;
    }
  }
  m->E = (const int8_t*)find_tensor(m, "emb.w", 1, (uint32_t)m->V, (uint32_t)(m->Ef ? m->Ef : m->d));
  m->s_E = (const float*)find_tensor(m, "emb.s", 2, (uint32_t)m->V, 1);
  m->pe = (const float*)find_tensor(m, "pe", 2, (uint32_t)m->P, (uint32_t)m->d);
  if (!m->E || !m->s_E || !m->pe) goto fail;
  m->inv_enc = (float)(1.0 / (double)m->s_enc);
  m->inv_fin = (float)(1.0 / (double)m->s_fin);
  if (!m->post) {
    if (load_ln(m, &m->enc_ln, "enc.ln") || load_ln(m, &m->dec_ln, "dec.ln")) goto fail;
  }
  m->c_emb = (float*)malloc(sizeof(float) * (size_t)m->V);
  m->c_out = (float*)malloc(sizeof(float) * (size_t)m->V);
  m->enc = (layer_t*)calloc((size_t)m->Le, sizeof(layer_t));
  m->dec = (layer_t*)calloc((size_t)m->Ld, sizeof(layer_t));
  if (!m->c_emb || !m->c_out || !m->enc || !m->dec) {
    rc = ORC_E_NOMEM;
    goto fail;
  }
  /* Shared embedding (Appendix D): input rows scaled by sqrt(d) (reading),
   * output projection dequantized by the scale of its int8 input (the final
   * activation scale, or s_u after a factorized embedding's projection). */
  for (int v = 0; v < m->V; ++v) {
    if (!(m->s_E[v] > 0.0f) || !isfinite(m->s_E[v])) goto fail;
    m->c_emb[v] = (float)((double)m->s_E[v] * sqrt((double)m->d));
    m->c_out[v] = (float)((double)m->s_emb_out * (double)m->s_E[v]);
  }
  for (int l = 0; l < m->Le; ++l)
    if (load_layer(m, &m->enc[l], "enc", l, 0)) goto fail;
  for (int l = 0; l < m->Ld; ++l)
    if (load_layer(m, &m->dec[l], "dec", l, 1)) goto fail;
  *out = m;
  return ORC_OK;
fail:
  orc_model_free(m);
  return rc;
}

int orc_model_dims(const orc_model* m, int32_t* dims) {
  if (!m || !dims) return ORC_E_ARG;
  int32_t v[16] = {m->d, m->h, m->F, m->Le, m->Ld, m->V, m->P, m->post,
                   m->pad_id, m->bos_id, m->eos_id, m->unk_id, m->Ef, 0, 0, 0};
  memcpy(dims, v, sizeof v);
  return ORC_OK;
}

/* Derived constants by name, for bit-comparison with other implementations:
 * "c_emb", "c_out" ([V]); "<side>.<l>.<sub>.<lin>.scale|bias" ([N]);
 * "<side>.<l>.<sa|ca>.c" ([2] = c_qk, c_pv). */
int orc_model_constants(const orc_model* m, const char* name, float* out, int n) {
  if (!m || !name || !out) return ORC_E_ARG;
  if (strcmp(name, "c_emb") == 0 || strcmp(name, "c_out") == 0) {
    if (n != m->V) return ORC_E_ARG;
    memcpy(out, name[2] == 'e' ? m->c_emb : m->c_out, sizeof(float) * (size_t)n);
    return ORC_OK;
  }
  char side[8], sub[8], lin[8], what[8];
  int l;
  if (sscanf(name, "%3[a-z].%d.%2[a-z].%3[a-z0-9].%5[a-z]", side, &l, sub, lin, what) == 5) {
    layer_t* L = strcmp(side, "enc") == 0 ? (l < m->Le ? &m->enc[l] : NULL)
                                           : (strcmp(side, "dec") == 0 && l < m->Ld ? &m->dec[l] : NULL);
    if (!L || l < 0) return ORC_E_ARG;
    const linear_t* ln = NULL;
    if (!strcmp(sub, "sa") && !strcmp(lin, "qkv")) ln = &L->sa.qkv;
    else if (!strcmp(sub, "sa") && !strcmp(lin, "o")) ln = &L->sa.o;
    else if (!strcmp(sub, "ca") && !strcmp(lin, "q")) ln = &L->ca.q;
    else if (!strcmp(sub, "ca") && !strcmp(lin, "kv")) ln = &L->ca.kv;
    else if (!strcmp(sub, "ca") && !strcmp(lin, "o")) ln = &L->ca.o;
    else if (!strcmp(sub, "ff") && !strcmp(lin, "w1")) ln = &L->ff.w1;
    else if (!strcmp(sub, "ff") && !strcmp(lin, "w2")) ln = &L->ff.w2;
    if (!ln || !ln->scale || n != ln->N) return ORC_E_ARG;
    if (!strcmp(what, "scale")) memcpy(out, ln->scale, sizeof(float) * (size_t)n);
    else if (!strcmp(what, "bias")) memcpy(out, ln->bias, sizeof(float) * (size_t)n);
    else return ORC_E_ARG;
    return ORC_OK;
  }
  if (sscanf(name, "%3[a-z].%d.%2[a-z].c", side, &l, sub) == 3 && n == 2) {
    layer_t* L = strcmp(side, "enc") == 0 ? (l < m->Le ? &m->enc[l] : NULL)
                                           : (strcmp(side, "dec") == 0 && l < m->Ld ? &m->dec[l] : NULL);
    if (!L || l < 0) return ORC_E_ARG;
    const attn_t* a = !strcmp(sub, "sa") ? &L->sa : (!strcmp(sub, "ca") ? &L->ca : NULL);
    if (!a) return ORC_E_ARG;
    out[0] = a->c_qk;
    out[1] = a->c_pv;
    return ORC_OK;
  }
  return ORC_E_ARG;
}

/* ------------------------------------------------------------------------- */
/* Transformer layers over a block of rows (Appendix A; quantizer figure)    */
/* ------------------------------------------------------------------------- */

/* Quantized input of a sublayer: pre-LN normalizes first; post-LN quantizes
 * the (already normalized) residual stream. */
static void sublayer_input(const orc_model* m, const ln_t* ln, const float* x, int rows, float inv_s,
                           int8_t* a) {
  if (!m->post) {
    orc_layernorm_quant(x, rows, m->d, ln->g, ln->b, m->eps, inv_s, a, NULL);
  } else {
    for (size_t i = 0; i < (size_t)rows * m->d; ++i) a[i] = orc_quantize(x[i], inv_s);
  }
}

/* Residual with the learnable weight gamma (Section 3.2): x = gamma x + F(.),
 * done inside the F32_RESID epilogue; post-LN then normalizes x. */
static void residual_linear(const orc_model* m, const linear_t* L, const ln_t* ln, float gamma,
                            const int8_t* a, int rows, float* x) {
  orc_qlinear(a, L->w, rows, L->K, L->N, L->scale, L->bias, gamma, ORC_EPI_F32_RESID, x);
  if (m->post) orc_layernorm_quant(x, rows, m->d, ln->g, ln->b, m->eps, 1.0f, NULL, x);
}

static void linear_i8(const linear_t* L, const int8_t* a, int rows, int relu, int8_t* y) {
  orc_qlinear(a, L->w, rows, L->K, L->N, L->scale, L->bias, 1.0f, relu ? ORC_EPI_I8_RELU : ORC_EPI_I8, y);
}

/* Copies of a forward pass's intermediate values (orc_encode_trace,
 * orc_decoder_trace): the sublayers u = 0, 1, ... of all layers in order
 * (encoder: self-attention, FFN; decoder: self-attention, cross-attention,
 * FFN), each traced for `rows` rows starting at row `row0`.  Slots:
 *   x   [U + 1][rows][d]  residual stream entering sublayer u; slot U after the last
 *   a   [U][rows][d]      int8 input of the sublayer's first linear layer
 *   pj  [U][rows][P]      QKV codes (self-attention, 3d), Q codes (cross, d) or the
 *                         ReLU hidden codes (FFN, F); P = max(3d, F)
 *   ctx [U][rows][d]      attention context codes (FFN sublayers: not written)
 * Any pointer may be NULL.  Copying changes none of the arithmetic. */
typedef struct {
  float* x;
  int8_t* a;
  int8_t* pj;
  int8_t* ctx;
  int rows, row0, P;
} trace_t;

static void tr_x(const orc_model* m, const trace_t* tr, int u, const float* x, int n) {
  if (tr && tr->x) memcpy(tr->x + ((size_t)u * tr->rows + tr->row0) * m->d, x, sizeof(float) * (size_t)n * m->d);
}

static void tr_i8(const trace_t* tr, int8_t* base, int u, int width, const int8_t* v, int n) {
  if (!tr || !base) return;
  for (int r = 0; r < n; ++r) memcpy(base + ((size_t)u * tr->rows + tr->row0 + r) * width, v + (size_t)r * width, (size_t)width);
}

/* Token embedding (shared matrix, scaled by sqrt(d)) plus the sinusoidal
 * position table stored in the model file: x = fma(E[tok], c_emb[tok], PE[pos]). */
static void embed(const orc_model* m, int tok, int pos, float* x) {
  const float* pe = m->pe + (size_t)pos * m->d;
  if (m->Ef) {
    /* factorized (Section 2.1): the token's Ef codes times the projection
     * Pw [d, Ef], dequantized by s_P, then scaled and positioned as above */
    const int8_t* ef = m->E + (size_t)tok * m->Ef;
    for (int n = 0; n < m->d; ++n) {
      int32_t acc = 0;
      for (int k = 0; k < m->Ef; ++k) acc += (int32_t)ef[k] * (int32_t)m->Pw[(size_t)n * m->Ef + k];
      x[n] = fmaf((float)acc * m->s_P, m->c_emb[tok], pe[n]);
    }
    return;
  }
  const int8_t* e = m->E + (size_t)tok * m->d;
  for (int j = 0; j < m->d; ++j) x[j] = fmaf((float)e[j], m->c_emb[tok], pe[j]);
}

/* Tied output projection (Appendix D) of the final int8 rows a [rows, d];
 * a factorized embedding first maps them back to its width Ef (Section 2.1):
 * u = requant(a . Pw, s_fin s_P / s_u), z = (u . E[v]) * s_u * s_E[v]. */
static void output_logits(const orc_model* m, const int8_t* a, int rows, float* z, int8_t* u_out) {
  if (!m->Ef) {
    orc_qlinear(a, m->E, rows, m->d, m->V, m->c_out, NULL, 1.0f, ORC_EPI_LOGITS, z);
    return;
  }
  int8_t* u = (int8_t*)malloc((size_t)rows * m->Ef);
  linear_i8(&m->proj_out, a, rows, 0, u);
  orc_qlinear(u, m->E, rows, m->Ef, m->V, m->c_out, NULL, 1.0f, ORC_EPI_LOGITS, z);
  if (u_out) memcpy(u_out, u, (size_t)rows * m->Ef);
  free(u);
}

static void ffn_sublayer(const orc_model* m, const ffn_t* f, float* x, int rows, const trace_t* tr, int u) {
  int8_t* a = (int8_t*)malloc((size_t)rows * m->d);
  int8_t* hb = (int8_t*)malloc((size_t)rows * m->F);
  tr_x(m, tr, u, x, rows);
  sublayer_input(m, &f->ln, x, rows, f->w1.inv_in, a);
  linear_i8(&f->w1, a, rows, 1, hb);
  if (tr) {
    tr_i8(tr, tr->a, u, m->d, a, rows);
    for (int r = 0; r < rows && tr->pj; ++r)
      memcpy(tr->pj + ((size_t)u * tr->rows + tr->row0 + r) * tr->P, hb + (size_t)r * m->F, (size_t)m->F);
  }
  residual_linear(m, &f->w2, &f->ln, f->gamma, hb, rows, x);
  free(a);
  free(hb);
}

/* Encoder of one sentence of S tokens -> enc codes [S, d] (scale s_enc). */
static void encode_sentence(const orc_model* m, const int32_t* src, int S, int8_t* enc, const trace_t* tr) {
  int d = m->d, dh = m->dh;
  float* x = (float*)malloc(sizeof(float) * (size_t)S * d);
  int8_t* a = (int8_t*)malloc((size_t)S * d);
  int8_t* qkv = (int8_t*)malloc((size_t)S * 3 * d);
  int8_t* ctx = (int8_t*)malloc((size_t)S * d);
  for (int t = 0; t < S; ++t) embed(m, src[t], t, x + (size_t)t * d);
  for (int l = 0; l < m->Le; ++l) {
    const layer_t* L = &m->enc[l];
    tr_x(m, tr, 2 * l, x, S);
    sublayer_input(m, &L->sa.ln, x, S, L->sa.qkv.inv_in, a);
    linear_i8(&L->sa.qkv, a, S, 0, qkv);
    for (int t = 0; t < S; ++t)
      for (int hd = 0; hd < m->h; ++hd)
        orc_attend(qkv + (size_t)t * 3 * d + hd * dh, qkv + d + hd * dh, qkv + 2 * d + hd * dh, S, dh, 3 * d,
                   L->sa.c_qk, L->sa.c_pv, ctx + (size_t)t * d + hd * dh);
    if (tr) {
      tr_i8(tr, tr->a, 2 * l, d, a, S);
      tr_i8(tr, tr->ctx, 2 * l, d, ctx, S);
      for (int t = 0; t < S && tr->pj; ++t)
        memcpy(tr->pj + ((size_t)(2 * l) * tr->rows + t) * tr->P, qkv + (size_t)t * 3 * d, (size_t)3 * d);
    }
    residual_linear(m, &L->sa.o, &L->sa.ln, L->sa.gamma, ctx, S, x);
    ffn_sublayer(m, &L->ff, x, S, tr, 2 * l + 1);
  }
  tr_x(m, tr, 2 * m->Le, x, S);
  if (!m->post)
    orc_layernorm_quant(x, S, d, m->enc_ln.g, m->enc_ln.b, m->eps, m->inv_enc, enc, NULL);
  else
    for (size_t i = 0; i < (size_t)S * d; ++i) enc[i] = orc_quantize(x[i], m->inv_enc);
  free(x);
  free(a);
  free(qkv);
  free(ctx);
}

static int check_batch(const orc_model* m, const int32_t* src, const int32_t* len, int B, int S_max) {
  if (!m || !src || !len || B <= 0 || S_max <= 0 || S_max > m->P) return ORC_E_ARG;
  for (int b = 0; b < B; ++b) {
    if (len[b] < 1 || len[b] > S_max) return ORC_E_ARG;
    for (int t = 0; t < len[b]; ++t)
      if (src[(size_t)b * S_max + t] < 0 || src[(size_t)b * S_max + t] >= m->V) return ORC_E_ARG;
  }
  return ORC_OK;
}

int orc_encode(const orc_model* m, const int32_t* src, const int32_t* len, int B, int S_max, int8_t* enc) {
  int rc = check_batch(m, src, len, B, S_max);
  if (rc) return rc;
  memset(enc, 0, (size_t)B * S_max * m->d);
  for (int b = 0; b < B; ++b) encode_sentence(m, src + (size_t)b * S_max, len[b], enc + (size_t)b * S_max * m->d, NULL);
  return ORC_OK;
}

int orc_cross_kv(const orc_model* m, const int8_t* enc, const int32_t* len, int B, int S_max, int layer,
                 int8_t* kv) {
  if (!m || layer < 0 || layer >= m->Ld || B <= 0 || S_max <= 0) return ORC_E_ARG;
  memset(kv, 0, (size_t)B * S_max * 2 * m->d);
  for (int b = 0; b < B; ++b)
    linear_i8(&m->dec[layer].ca.kv, enc + (size_t)b * S_max * m->d, len[b], 0,
              kv + (size_t)b * S_max * 2 * m->d);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Decoder: one step of one hypothesis with its own key/value cache          */
/* ------------------------------------------------------------------------- */

typedef struct {
  int8_t** k; /* per layer [T, d] self-attention key codes */
  int8_t** v;
} kv_cache_t;

static void cache_alloc(const orc_model* m, kv_cache_t* c, int T) {
  c->k = (int8_t**)malloc(sizeof(int8_t*) * (size_t)m->Ld);
  c->v = (int8_t**)malloc(sizeof(int8_t*) * (size_t)m->Ld);
  for (int l = 0; l < m->Ld; ++l) {
    c->k[l] = (int8_t*)calloc((size_t)T * m->d, 1);
    c->v[l] = (int8_t*)calloc((size_t)T * m->d, 1);
  }
}

static void cache_copy(const orc_model* m, kv_cache_t* dst, const kv_cache_t* src, int T) {
  for (int l = 0; l < m->Ld; ++l) {
    memcpy(dst->k[l], src->k[l], (size_t)T * m->d);
    memcpy(dst->v[l], src->v[l], (size_t)T * m->d);
  }
}

static void cache_free(const orc_model* m, kv_cache_t* c) {
  for (int l = 0; l < m->Ld; ++l) {
    free(c->k[l]);
    free(c->v[l]);
  }
  free(c->k);
  free(c->v);
}

/* Decoder step at position t for input token tok: appends this step's K/V to
 * the cache, attends over positions 0..t (self) and over the S source
 * positions (cross), and writes the logits z[V]. */
static void decoder_step(const orc_model* m, int tok, int t, kv_cache_t* c, int8_t* const* cross_kv, int S,
                         float* z, const trace_t* tr, int8_t* fin, int8_t* fin_u) {
  int d = m->d, dh = m->dh;
  float* x = (float*)malloc(sizeof(float) * (size_t)d);
  int8_t* a = (int8_t*)malloc((size_t)d);
  int8_t* qkv = (int8_t*)malloc((size_t)3 * d);
  int8_t* q = (int8_t*)malloc((size_t)d);
  int8_t* ctx = (int8_t*)malloc((size_t)d);
  embed(m, tok, t, x);
  for (int l = 0; l < m->Ld; ++l) {
    const layer_t* L = &m->dec[l];
    const int u = 3 * l;
    /* self-attention over the cache (causal: positions 0..t) */
    tr_x(m, tr, u, x, 1);
    sublayer_input(m, &L->sa.ln, x, 1, L->sa.qkv.inv_in, a);
    linear_i8(&L->sa.qkv, a, 1, 0, qkv);
    memcpy(c->k[l] + (size_t)t * d, qkv + d, (size_t)d);
    memcpy(c->v[l] + (size_t)t * d, qkv + 2 * d, (size_t)d);
    for (int hd = 0; hd < m->h; ++hd)
      orc_attend(qkv + hd * dh, c->k[l] + hd * dh, c->v[l] + hd * dh, t + 1, dh, d, L->sa.c_qk, L->sa.c_pv,
                 ctx + hd * dh);
    if (tr) {
      tr_i8(tr, tr->a, u, d, a, 1);
      tr_i8(tr, tr->ctx, u, d, ctx, 1);
      if (tr->pj) memcpy(tr->pj + ((size_t)u * tr->rows + tr->row0) * tr->P, qkv, (size_t)3 * d);
    }
    residual_linear(m, &L->sa.o, &L->sa.ln, L->sa.gamma, ctx, 1, x);
    /* cross-attention over the encoder output */
    tr_x(m, tr, u + 1, x, 1);
    sublayer_input(m, &L->ca.ln, x, 1, L->ca.q.inv_in, a);
    linear_i8(&L->ca.q, a, 1, 0, q);
    for (int hd = 0; hd < m->h; ++hd)
      orc_attend(q + hd * dh, cross_kv[l] + hd * dh, cross_kv[l] + d + hd * dh, S, dh, 2 * d, L->ca.c_qk,
                 L->ca.c_pv, ctx + hd * dh);
    if (tr) {
      tr_i8(tr, tr->a, u + 1, d, a, 1);
      tr_i8(tr, tr->ctx, u + 1, d, ctx, 1);
      if (tr->pj) memcpy(tr->pj + ((size_t)(u + 1) * tr->rows + tr->row0) * tr->P, q, (size_t)d);
    }
    residual_linear(m, &L->ca.o, &L->ca.ln, L->ca.gamma, ctx, 1, x);
    ffn_sublayer(m, &L->ff, x, 1, tr, u + 2);
  }
  tr_x(m, tr, 3 * m->Ld, x, 1);
  if (!m->post)
    orc_layernorm_quant(x, 1, d, m->dec_ln.g, m->dec_ln.b, m->eps, m->inv_fin, a, NULL);
  else
    for (int j = 0; j < d; ++j) a[j] = orc_quantize(x[j], m->inv_fin);
  if (fin) memcpy(fin, a, (size_t)d);
  /* tied output projection over the shared embedding */
  output_logits(m, a, 1, z, fin_u);
  free(x);
  free(a);
  free(qkv);
  free(q);
  free(ctx);
}

static int8_t** build_cross(const orc_model* m, const int32_t* src, int S) {
  int8_t* enc = (int8_t*)malloc((size_t)S * m->d);
  encode_sentence(m, src, S, enc, NULL);
  int8_t** kv = (int8_t**)malloc(sizeof(int8_t*) * (size_t)m->Ld);
  for (int l = 0; l < m->Ld; ++l) {
    kv[l] = (int8_t*)malloc((size_t)S * 2 * m->d);
    linear_i8(&m->dec[l].ca.kv, enc, S, 0, kv[l]);
  }
  free(enc);
  return kv;
}

static void free_cross(const orc_model* m, int8_t** kv) {
  for (int l = 0; l < m->Ld; ++l) free(kv[l]);
  free(kv);
}

/* Greedy search (Appendix D): the next token is the arg max of the logits,
 * the smallest index among equal maxima. */
int orc_translate_greedy(const orc_model* m, const int32_t* src, const int32_t* len, int B, int S_max,
                         int steps, int stop_at_eos, int32_t* out, int32_t* out_len, float* logits) {
  int rc = check_batch(m, src, len, B, S_max);
  if (rc) return rc;
  if (steps < 1 || steps > m->P || !out || !out_len) return ORC_E_ARG;
  float* z = (float*)malloc(sizeof(float) * (size_t)m->V);
  for (int b = 0; b < B; ++b) {
    int8_t** cross = build_cross(m, src + (size_t)b * S_max, len[b]);
    kv_cache_t c;
    cache_alloc(m, &c, steps);
    int tok = m->bos_id, n_out = steps, done = 0;
    for (int t = 0; t < steps; ++t) {
      if (done) {
        out[(size_t)b * steps + t] = m->pad_id;
        continue;
      }
      decoder_step(m, tok, t, &c, cross, len[b], z, NULL, NULL, NULL);
      if (logits) memcpy(logits + ((size_t)b * steps + t) * m->V, z, sizeof(float) * (size_t)m->V);
      int best = 0;
      for (int v = 1; v < m->V; ++v)
        if (z[v] > z[best]) best = v;
      out[(size_t)b * steps + t] = best;
      tok = best;
      if (stop_at_eos && best == m->eos_id) {
        done = 1;
        n_out = t + 1;
      }
    }
    out_len[b] = n_out;
    cache_free(m, &c);
    free_cross(m, cross);
  }
  free(z);
  return ORC_OK;
}

/* Teacher-forced decoding of one sentence: inputs BOS, tok[0], ..., tok[n-2]
 * at positions 0..n-1; z[n, V] receives the logits of every step. */
int orc_decoder_logits(const orc_model* m, const int32_t* src, int S, const int32_t* tok, int n, float* z) {
  if (!m || !src || !tok || !z || S < 1 || S > m->P || n < 1 || n > m->P) return ORC_E_ARG;
  for (int t = 0; t < S; ++t)
    if (src[t] < 0 || src[t] >= m->V) return ORC_E_ARG;
  for (int t = 0; t < n; ++t)
    if (tok[t] < 0 || tok[t] >= m->V) return ORC_E_ARG;
  int8_t** cross = build_cross(m, src, S);
  kv_cache_t c;
  cache_alloc(m, &c, n);
  for (int t = 0; t < n; ++t)
    decoder_step(m, t == 0 ? m->bos_id : tok[t - 1], t, &c, cross, S, z + (size_t)t * m->V, NULL, NULL, NULL);
  cache_free(m, &c);
  free_cross(m, cross);
  return ORC_OK;
}

/* The encoder of one sentence with its intermediate values copied out (see
 * trace_t; U = 2 n_enc sublayers, rows = S) and its output codes enc [S, d]. */
int orc_encode_trace(const orc_model* m, const int32_t* src, int S, float* x, int8_t* a, int8_t* pj, int8_t* ctx,
                     int8_t* enc) {
  if (!m || !src || !enc || S < 1 || S > m->P) return ORC_E_ARG;
  for (int t = 0; t < S; ++t)
    if (src[t] < 0 || src[t] >= m->V) return ORC_E_ARG;
  trace_t tr = {x, a, pj, ctx, S, 0, 3 * m->d > m->F ? 3 * m->d : m->F};
  encode_sentence(m, src, S, enc, &tr);
  return ORC_OK;
}

/* Teacher-forced decoding (as orc_decoder_logits) with each step's
 * intermediate values copied out: trace_t with U = 3 n_dec sublayers and one
 * row per step; fin [n, d] receives each step's int8 final rows, fin_u [n, Ef]
 * (factorized embeddings) their projection back to the embedding width, z
 * [n, V] the logits. */
int orc_decoder_trace(const orc_model* m, const int32_t* src, int S, const int32_t* tok, int n, float* x, int8_t* a,
                      int8_t* pj, int8_t* ctx, int8_t* fin, int8_t* fin_u, float* z) {
  if (!m || !src || !tok || !z || S < 1 || S > m->P || n < 1 || n > m->P) return ORC_E_ARG;
  for (int t = 0; t < S; ++t)
    if (src[t] < 0 || src[t] >= m->V) return ORC_E_ARG;
  for (int t = 0; t < n; ++t)
    if (tok[t] < 0 || tok[t] >= m->V) return ORC_E_ARG;
  int8_t** cross = build_cross(m, src, S);
  kv_cache_t c;
  cache_alloc(m, &c, n);
  for (int t = 0; t < n; ++t) {
    trace_t tr = {x, a, pj, ctx, n, t, 3 * m->d > m->F ? 3 * m->d : m->F};
    decoder_step(m, t == 0 ? m->bos_id : tok[t - 1], t, &c, cross, S, z + (size_t)t * m->V, &tr,
                 fin ? fin + (size_t)t * m->d : NULL, fin_u && m->Ef ? fin_u + (size_t)t * m->Ef : NULL);
  }
  cache_free(m, &c);
  free_cross(m, cross);
  return ORC_OK;
}

/* The same teacher-forced logits computed without a cache: all n target
 * positions go through each layer as one block, position t attending over
 * block rows 0..t (causal mask), like the encoder does over the source. */
int orc_decoder_logits_full(const orc_model* m, const int32_t* src, int S, const int32_t* tok, int n, float* z) {
  if (!m || !src || !tok || !z || S < 1 || S > m->P || n < 1 || n > m->P) return ORC_E_ARG;
  for (int t = 0; t < S; ++t)
    if (src[t] < 0 || src[t] >= m->V) return ORC_E_ARG;
  for (int t = 0; t < n; ++t)
    if (tok[t] < 0 || tok[t] >= m->V) return ORC_E_ARG;
  int d = m->d, dh = m->dh;
  int8_t** cross = build_cross(m, src, S);
  float* x = (float*)malloc(sizeof(float) * (size_t)n * d);
  int8_t* a = (int8_t*)malloc((size_t)n * d);
  int8_t* qkv = (int8_t*)malloc((size_t)n * 3 * d);
  int8_t* q = (int8_t*)malloc((size_t)n * d);
  int8_t* ctx = (int8_t*)malloc((size_t)n * d);
  for (int t = 0; t < n; ++t) embed(m, t == 0 ? m->bos_id : tok[t - 1], t, x + (size_t)t * d);
  for (int l = 0; l < m->Ld; ++l) {
    const layer_t* L = &m->dec[l];
    sublayer_input(m, &L->sa.ln, x, n, L->sa.qkv.inv_in, a);
    linear_i8(&L->sa.qkv, a, n, 0, qkv);
    for (int t = 0; t < n; ++t)
      for (int hd = 0; hd < m->h; ++hd)
        orc_attend(qkv + (size_t)t * 3 * d + hd * dh, qkv + d + hd * dh, qkv + 2 * d + hd * dh, t + 1, dh, 3 * d,
                   L->sa.c_qk, L->sa.c_pv, ctx + (size_t)t * d + hd * dh);
    residual_linear(m, &L->sa.o, &L->sa.ln, L->sa.gamma, ctx, n, x);
    sublayer_input(m, &L->ca.ln, x, n, L->ca.q.inv_in, a);
    linear_i8(&L->ca.q, a, n, 0, q);
    for (int t = 0; t < n; ++t)
      for (int hd = 0; hd < m->h; ++hd)
        orc_attend(q + (size_t)t * d + hd * dh, cross[l] + hd * dh, cross[l] + d + hd * dh, S, dh, 2 * d,
                   L->ca.c_qk, L->ca.c_pv, ctx + (size_t)t * d + hd * dh);
    residual_linear(m, &L->ca.o, &L->ca.ln, L->ca.gamma, ctx, n, x);
    ffn_sublayer(m, &L->ff, x, n, NULL, 0);
  }
  if (!m->post)
    orc_layernorm_quant(x, n, d, m->dec_ln.g, m->dec_ln.b, m->eps, m->inv_fin, a, NULL);
  else
    for (size_t i = 0; i < (size_t)n * d; ++i) a[i] = orc_quantize(x[i], m->inv_fin);
  output_logits(m, a, n, z, NULL);
  free(x);
  free(a);
  free(qkv);
  free(q);
  free(ctx);
  free_cross(m, cross);
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Beam search (R8)                                                       */
/* ------------------------------------------------------------------------- */
/* Per sentence, W live hypotheses.  Step 0 expands only hypothesis 0.  Each
 * step scores every expansion as score + (z_v - lse) and keeps the 2W best by
 * (score desc, flat index j*V + v asc), or all of them when there are fewer
 * (then fewer than W slots may stay live).  Walking them in that order: an EOS
 * candidate among the first W is finished with normalized score
 * score / lp(t + 1); other candidates refill the W live slots in order.  The
 * sentence stops once W hypotheses are finished.  After the last step the
 * live hypotheses are finished with score / lp(max_steps).  The result is the
 * finished hypothesis with the highest normalized score, the earliest
 * finished among equals. */

typedef struct {
  float score;
  int slot;
  int v;
} cand_t;

static int cand_better(const cand_t* a, const cand_t* b, int V) {
  if (a->score != b->score) return a->score > b->score;
  return (long)a->slot * V + a->v < (long)b->slot * V + b->v;
}

static void translate_one_beam(const orc_model* m, const int32_t* src, int S, int W, int T, float alpha,
                               int32_t* out, int32_t* out_len, float* out_score) {
  int V = m->V;
  int8_t** cross = build_cross(m, src, S);
  kv_cache_t* cache = (kv_cache_t*)malloc(sizeof(kv_cache_t) * (size_t)W);
  kv_cache_t* next_cache = (kv_cache_t*)malloc(sizeof(kv_cache_t) * (size_t)W);
  int32_t* toks = (int32_t*)calloc((size_t)W * T, sizeof(int32_t));
  int32_t* next_toks = (int32_t*)calloc((size_t)W * T, sizeof(int32_t));
  float* score = (float*)calloc((size_t)W, sizeof(float));
  float* next_score = (float*)calloc((size_t)W, sizeof(float));
  int* alive = (int*)calloc((size_t)W, sizeof(int));
  float* z = (float*)malloc(sizeof(float) * (size_t)V);
  cand_t* best = (cand_t*)malloc(sizeof(cand_t) * (size_t)2 * W);
  /* finished list */
  int fin_cap = 2 * W + 1, n_fin = 0;
  float* fin_score = (float*)malloc(sizeof(float) * (size_t)fin_cap);
  int32_t* fin_len = (int32_t*)malloc(sizeof(int32_t) * (size_t)fin_cap);
  int32_t* fin_toks = (int32_t*)calloc((size_t)fin_cap * T, sizeof(int32_t));
  for (int j = 0; j < W; ++j) {
    cache_alloc(m, &cache[j], T);
    cache_alloc(m, &next_cache[j], T);
  }
  alive[0] = 1;
  int done = 0;
  for (int t = 0; t < T && !done; ++t) {
    int n_best = 0;
    for (int j = 0; j < W; ++j) {
      if (!alive[j]) continue;
      int tok = t == 0 ? m->bos_id : toks[(size_t)j * T + t - 1];
      decoder_step(m, tok, t, &cache[j], cross, S, z, NULL, NULL, NULL);
      float lse;
      orc_log_softmax_stats(z, V, NULL, &lse);
      for (int v = 0; v < V; ++v) {
        cand_t c = {score[j] + (z[v] - lse), j, v};
        /* insert into the sorted list of the 2W best */
        if (n_best == 2 * W && !cand_better(&c, &best[n_best - 1], V)) continue;
        int pos = n_best < 2 * W ? n_best++ : n_best - 1;
        while (pos > 0 && cand_better(&c, &best[pos - 1], V)) {
          best[pos] = best[pos - 1];
          --pos;
        }
        best[pos] = c;
      }
    }
    int n_live = 0;
    for (int r = 0; r < n_best && n_live < W; ++r) {
      const cand_t* c = &best[r];
      if (c->v == m->eos_id) {
        if (r < W && n_fin < W) {
          fin_score[n_fin] = c->score / orc_length_penalty(t + 1, alpha);
          fin_len[n_fin] = t + 1;
          memcpy(fin_toks + (size_t)n_fin * T, toks + (size_t)c->slot * T, sizeof(int32_t) * (size_t)t);
          fin_toks[(size_t)n_fin * T + t] = c->v;
          ++n_fin;
        }
        continue;
      }
      memcpy(next_toks + (size_t)n_live * T, toks + (size_t)c->slot * T, sizeof(int32_t) * (size_t)t);
      next_toks[(size_t)n_live * T + t] = c->v;
      next_score[n_live] = c->score;
      cache_copy(m, &next_cache[n_live], &cache[c->slot], T);
      ++n_live;
    }
    if (n_fin >= W) {
      done = 1;
      break;
    }
    /* swap in the refilled slots */
    kv_cache_t* tc = cache;
    cache = next_cache;
    next_cache = tc;
    int32_t* tt = toks;
    toks = next_toks;
    next_toks = tt;
    float* ts = score;
    score = next_score;
    next_score = ts;
    for (int j = 0; j < W; ++j) alive[j] = j < n_live;
  }
  if (!done) {
    for (int j = 0; j < W; ++j) {
      if (!alive[j]) continue;
      fin_score[n_fin] = score[j] / orc_length_penalty(T, alpha);
      fin_len[n_fin] = T;
      memcpy(fin_toks + (size_t)n_fin * T, toks + (size_t)j * T, sizeof(int32_t) * (size_t)T);
      ++n_fin;
    }
  }
  int bi = 0;
  for (int i = 1; i < n_fin; ++i)
    if (fin_score[i] > fin_score[bi]) bi = i;
  for (int t = 0; t < T; ++t) out[t] = t < fin_len[bi] ? fin_toks[(size_t)bi * T + t] : m->pad_id;
  *out_len = fin_len[bi];
  *out_score = fin_score[bi];
  for (int j = 0; j < W; ++j) {
    cache_free(m, &cache[j]);
    cache_free(m, &next_cache[j]);
  }
  free(cache);
  free(next_cache);
  free(toks);
  free(next_toks);
  free(score);
  free(next_score);
  free(alive);
  free(z);
  free(best);
  free(fin_score);
  free(fin_len);
  free(fin_toks);
  free_cross(m, cross);
}

int orc_translate_beam(const orc_model* m, const int32_t* src, const int32_t* len, int B, int S_max, int beam,
                       int max_steps, float alpha, int32_t* out, int32_t* out_len, float* score) {
  int rc = check_batch(m, src, len, B, S_max);
  if (rc) return rc;
  if (beam < 1 || beam > 4096 || max_steps < 1 || max_steps > m->P || !out || !out_len || !score)
    return ORC_E_ARG;
  for (int b = 0; b < B; ++b)
    translate_one_beam(m, src + (size_t)b * S_max, len[b], beam, max_steps, alpha, out + (size_t)b * max_steps,
                       out_len + b, score + b);
  return ORC_OK;
}
