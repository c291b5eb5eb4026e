/*
 * mnmt_oracle.h -- plain CPU oracle for INT8 encoder-decoder inference as
 * described in MobileNMT (arXiv 2306.04235).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that the GPU library can
 * be checked against an obviously correct, slow, scalar implementation.  It
 * shares no code, header, table or constant generator with the GPU library.
 * Only tests, the smoke check and the benchmark's CPU-baseline leg use it.
 *
 * Arithmetic: int8 x int8 -> int32 for every linear layer; IEEE binary32 with
 * round-to-nearest-even for everything else (the paper keeps biases, residuals,
 * attention scores and softmax output in full precision, Section 3.2 and the
 * quantizer figure).  fmaf only where written; the build disables contraction.
 *
 * Every function returns 0 on success or a negative ORC_E_* code.
 */
#ifndef MNMT_ORACLE_H
#define MNMT_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_OK 0
#define ORC_E_ARG (-1)
#define ORC_E_MODEL (-2)
#define ORC_E_NOMEM (-3)

/* Epilogue selectors for orc_qlinear (see the .c file for the formulas). */
#define ORC_EPI_I32 0
#define ORC_EPI_I8 1
#define ORC_EPI_I8_RELU 2
#define ORC_EPI_F32 3
#define ORC_EPI_F32_RESID 4
#define ORC_EPI_LOGITS 5

typedef struct orc_model orc_model;

/* --- canonical fp32 primitives (exposed so tests can pin them) --- */
float orc_exp(float x);                       /* e^x for x <= 0 */
float orc_log(float x);                       /* ln x for normal x > 0 */
float orc_canon_sum(const float* x, int n);   /* 64 interleaved partial sums, halving combine */
float orc_canon_sum_squares(const float* x, int n); /* the same order, partials p = fma(x, x, p) */
float orc_canon_vocab_sum(const float* x, int n);   /* vocabulary sums: 512 partials, 4 terms a turn, tree of 8 */
int8_t orc_quantize(float y, float inv_s);    /* clamp(rne(y * inv_s), -127, 127) */
float orc_length_penalty(int L, float alpha); /* ((5 + L) / 6)^alpha */
int orc_map(int fn, const float* x, int n, float* y); /* fn 0: orc_exp, 1: orc_log */

/* --- stage functions --- */
int orc_qgemm_i32(const int8_t* X, const int8_t* W, int M, int K, int N, int32_t* Y);
int orc_qlinear(const int8_t* X, const int8_t* W, int M, int K, int N, const float* scale,
                const float* bias, float gamma, int epilogue, void* Y);
int orc_fold_requant(float s_in, const float* s_w, const float* b, float s_out, int N, float* scale,
                     float* bias);
int orc_fold_dequant(float s_in, const float* s_w, int N, float* scale);
int orc_layernorm_quant(const float* x, int rows, int d, const float* g, const float* b, float eps,
                        float inv_s, int8_t* q, float* y);
int orc_attend(const int8_t* q, const int8_t* K, const int8_t* V, int n, int dh, int ldk,
               float c_qk, float c_pv, int8_t* out);
int orc_log_softmax_stats(const float* z, int n, float* max_out, float* lse_out);

/* --- model level --- */
int orc_model_load(const void* blob, size_t nbytes, orc_model** out);
void orc_model_free(orc_model* m);
int orc_model_dims(const orc_model* m, int32_t* dims /* [16] */);
int orc_model_constants(const orc_model* m, const char* name, float* out, int n);

/* Encoder output codes [B, S_max, d] (rows >= len[b] are zero). */
int orc_encode(const orc_model* m, const int32_t* src, const int32_t* len, int B, int S_max,
               int8_t* enc);
/* Cross-attention K|V codes of decoder layer `layer` for encoder codes [B,S_max,d] -> [B,S_max,2d]. */
int orc_cross_kv(const orc_model* m, const int8_t* enc, const int32_t* len, int B, int S_max,
                 int layer, int8_t* kv);
/* Greedy search: out [B, steps] (PAD after EOS when stop_at_eos), out_len [B],
 * logits optional [B, steps, V]. */
int orc_translate_greedy(const orc_model* m, const int32_t* src, const int32_t* len, int B,
                         int S_max, int steps, int stop_at_eos, int32_t* out, int32_t* out_len,
                         float* logits);
/* Teacher-forced decoder logits z[n, V] for inputs BOS, tok[0..n-2] of one sentence. */
int orc_decoder_logits(const orc_model* m, const int32_t* src, int S, const int32_t* tok, int n, float* z);
/* The same logits from a cache-free block computation with a causal mask. */
int orc_decoder_logits_full(const orc_model* m, const int32_t* src, int S, const int32_t* tok, int n,
                            float* z);
/* Intermediate values for stage-by-stage tests.  Sublayers u in order
 * (encoder: self-attention, FFN; decoder: self-attention, cross-attention,
 * FFN), U of them; P = max(3d, F).  Any of x, a, pj, ctx may be NULL.
 *   x [U+1][rows][d] fp32 residual stream entering sublayer u (slot U: after the last)
 *   a [U][rows][d] int8 input of the sublayer's first linear layer
 *   pj [U][rows][P] int8 QKV (3d), cross Q (d) or FFN hidden (F) codes
 *   ctx [U][rows][d] int8 attention context codes
 * Encoder of one sentence: rows = S, enc [S, d] output codes. */
int orc_encode_trace(const orc_model* m, const int32_t* src, int S, float* x, int8_t* a, int8_t* pj, int8_t* ctx,
                     int8_t* enc);
/* Teacher-forced decoding with rows = n steps; fin [n, d] the int8 final rows
 * at each step (or NULL), fin_u [n, Ef] their projection back to the width Ef
 * of a factorized embedding (or NULL); z [n, V] logits. */
int orc_decoder_trace(const orc_model* m, const int32_t* src, int S, const int32_t* tok, int n, float* x, int8_t* a,
                      int8_t* pj, int8_t* ctx, int8_t* fin, int8_t* fin_u, float* z);
/* Beam search: out [B, max_steps] (PAD-filled), out_len [B], score [B]. */
int orc_translate_beam(const orc_model* m, const int32_t* src, const int32_t* len, int B, int S_max,
                       int beam, int max_steps, float alpha, int32_t* out, int32_t* out_len,
                       float* score);

#ifdef __cplusplus
}
#endif
#endif
