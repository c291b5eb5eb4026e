/*
 * mnmt.h -- C ABI of libmnmt, an INT8 encoder-decoder Transformer inference
 * engine for AMD Instinct MI355X (gfx950), after MobileNMT (arXiv 2306.04235).
 *
 * What the engine computes (paper passages):
 *   - Transformer encoder-decoder with self-attention, cross-attention and a
 *     ReLU FFN, residual connections (Appendix A, self-weight / self-sum / FFN
 *     equations), LayerNorm at each sublayer input (Appendix D) or, for
 *     post-LN model files, after each residual add.
 *   - One shared vocabulary embedding for encoder input, decoder input and the
 *     output projection (Appendix D; "Embed x1" in the settings tables).
 *   - Quantizers of Section 3.2 (quantizer figure): every linear layer takes
 *     int8 inputs and int8 weights and accumulates in int32; Q, K and V are
 *     int8 (the key/value caches hold these codes); biases, the residual
 *     stream, attention scores, softmax output and logits stay fp32; a
 *     learnable weight gamma scales each sublayer's residual.
 *   - 8-bit integer GEMM (Section 4.1) and fused element-wise work between
 *     GEMMs plus shared scratch buffers (Section 4.2).
 *   - Greedy search (Appendix D) and beam search.
 * Every fp32 step is fixed to a canonical IEEE binary32 evaluation order so
 * that results are reproducible bit for bit (documented in the design notes).
 *
 * Conventions for every entry point:
 *   - Return MNMT_OK (0) or a negative MNMT_E_* status; no C++ exception
 *     crosses this boundary.  mnmt_last_error() gives a thread-local message.
 *   - The library never allocates device memory.  The caller allocates the
 *     model arena and the session workspace (sizes from mnmt_model_bytes /
 *     mnmt_session_bytes) and owns them; they must stay valid while the model
 *     or session exists.  The library owns only small host structures.
 *   - "d_" pointers are device pointers (HIP global memory); "h_" pointers are
 *     host pointers.  `stream` is a hipStream_t passed as void* (NULL is the
 *     null stream); device work is enqueued on it asynchronously unless stated.
 *   - Device pointers passed to the engine must be 16-byte aligned.
 *   - A session is not thread-safe.  Several sessions may share one model.
 *   - Token ids are int32: PAD, BOS, EOS, UNK come from the model file
 *     (0, 1, 2, 3 in the files this project writes).
 *
 * Model file (little endian), version 1:
 *   header, 64 bytes: char magic[4] = "MNMT"; u32 version = 1; u32 d_model,
 *   n_heads, d_ffn, n_enc, n_dec, vocab, max_pos, ln_post (0 pre-LN,
 *   1 post-LN); i32 pad_id, bos_id, eos_id, unk_id; f32 ln_eps; u32 n_tensors.
 *   n_tensors entries of 64 bytes: char name[40] (NUL padded); u32 dtype
 *   (1 int8, 2 fp32, 3 packed 4-bit: linear weights only, dim1 a multiple of
 *   16, dim0 * dim1 / 2 bytes); u32 rank (1 or 2); u32 dim0; u32 dim1 (1 for
 *   rank 1);
 *   u64 offset (from file start, multiple of 256).  Tensors, d = d_model,
 *   F = d_ffn, V = vocab, P = max_pos; <e> = "enc.<l>", <t> = "dec.<l>":
 *     emb.w i8 [V,d], emb.s f32 [V] (per-row scale), pe f32 [P,d],
 *     enc.sout, dec.sout f32 [1] (encoder-output / final activation scales),
 *     enc.ln.{g,b}, dec.ln.{g,b} f32 [d] (final LayerNorms, pre-LN files),
 *     <e|t>.sa.ln.{g,b}, .sa.qkv.{w [3d,d], sw [3d], b [3d], sin [1], sout [3]},
 *     .sa.o.{w [d,d], sw, b, sin (= context scale)}, .sa.gamma [1],
 *     <t>.ca.ln.{g,b}, .ca.q.{w,sw,b,sin,sout [1]}, .ca.kv.{w [2d,d],sw,b,
 *     sout [2]} (input scale = enc.sout), .ca.o.{w,sw,b,sin}, .ca.gamma,
 *     <e|t>.ff.ln.{g,b}, .ff.w1.{w [F,d],sw,b,sin,sout [1]},
 *     .ff.w2.{w [d,F],sw,b} (input scale = ff.w1.sout), .ff.gamma.
 *   Optional, cross-layer parameter sharing (Section 2.2): an int8 tensor
 *   <e|t>.share [1] = j < l replaces all of layer l's tensors: layer l runs
 *   on layer j's parameters (stored once).
 *   Optional, embedding factorization (Section 2.1, "Scaling E"): emb.w is
 *   [V, E] (E a multiple of 64, E <= d) with emb.proj.w i8 [d, E], emb.proj.sw
 *   f32 [1] (one scale: the matrix is used in both orientations) and
 *   emb.proj.sout f32 [1] (scale s_u of the output projection's int8 input):
 *   input rows x = (float)(E[tok] . P[n]) * sw * c_emb[tok] + PE; output
 *   u = requant(a P, s_fin * sw / s_u), logits z[v] = (u . E[v]) * s_u * s_E[v].
 *   Such models run on the general (unfused) decode paths.
 *   Weights are symmetric per-output-channel int8: w_real = sw[n] * w[n,k].
 *   4-bit weights (the paper's W-E-A 4-8-8 setting) hold codes in [-7, 7]:
 *   in each group of 16 codes of a row, byte i (i < 8) holds code i in its
 *   low nibble and code i + 8 in its high nibble, each stored plus 8.  The
 *   batch-1 decoder step and the small-batch encoder read them packed and
 *   widen them to int8 in registers.  The batched kernels read an int8 copy
 *   that the loader also keeps, or, with MNMT_LOAD_PACKED_4BIT_ONLY, the
 *   packed rows too (widened on their way to the matrix cores).
 */
#ifndef MNMT_H
#define MNMT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MNMT_OK 0
#define MNMT_E_INVALID_ARG (-1)  /* bad pointer, size, alignment or value */
#define MNMT_E_BAD_MODEL (-2)    /* model file malformed or inconsistent */
#define MNMT_E_CAPACITY (-3)     /* request exceeds the session's capacity */
#define MNMT_E_HIP (-4)          /* a HIP runtime call failed (text in last_error) */
#define MNMT_E_UNSUPPORTED (-5)  /* valid but not supported by this build */
#define MNMT_E_TIMEOUT (-6)      /* a kernel's bounded wait for another kernel gave up (see mnmt_session_status) */

/* Linear-layer epilogues (quantizer figure, Section 3.2), y = acc*scale+bias:
 *   MNMT_EPI_I32:       Y int32 = acc
 *   MNMT_EPI_I8:        Y int8  = clamp(rint(fma(acc, scale[n], bias[n])), -127, 127)
 *   MNMT_EPI_I8_RELU:   Y int8  = clamp(rint(max(fma(acc, scale[n], bias[n]), 0)), ..)
 *   MNMT_EPI_F32:       Y fp32  = fma(acc, scale[n], bias[n])
 *   MNMT_EPI_F32_RESID: Y fp32  = fma(gamma, Y, fma(acc, scale[n], bias[n]))  (in place)
 *   MNMT_EPI_LOGITS:    Y fp32  = acc * scale[n]                      (bias unused)
 *   MNMT_EPI_ARGMAX:    Y uint64 [M] (caller zero-fills) receives, per row, the
 *                       maximum over n of key(z) << 32 | (0xFFFFFFFF - n) with
 *                       z = acc * scale[n] and key() order-preserving on
 *                       floats: the arg max with the smallest index among
 *                       equal maxima, fused into the logits pass (M <= 8).
 *   MNMT_EPI_ARGMAX_PARTIAL: Y uint64 [M, P], P = mnmt_argmax_partials(N): the
 *                       same keys, one maximum per block of the logits kernel
 *                       (plain stores, no zero-fill needed); the row's arg-max
 *                       key is the largest of its P entries (M <= 2, K <= 512,
 *                       as the decoder's batch-1 step writes it).
 *   MNMT_EPI_ARGMAX_PARTIAL_PACKED: MNMT_EPI_ARGMAX_PARTIAL with d_W the
 *                       fragment-order copy that mnmt_pack_weights writes
 *                       (the layout the batch-1 decoder reads its tied
 *                       output embedding in); same keys, same P.
 * acc = sum_k X[m,k] W[n,k] in int32, converted to fp32 with round-to-nearest-even. */
#define MNMT_EPI_I32 0
#define MNMT_EPI_I8 1
#define MNMT_EPI_I8_RELU 2
#define MNMT_EPI_F32 3
#define MNMT_EPI_F32_RESID 4
#define MNMT_EPI_LOGITS 5
#define MNMT_EPI_ARGMAX 6
#define MNMT_EPI_ARGMAX_PARTIAL 7
#define MNMT_EPI_ARGMAX_PARTIAL_PACKED 8

typedef struct mnmt_model mnmt_model;
typedef struct mnmt_session mnmt_session;

typedef struct {
  int32_t d_model, n_heads, d_ffn, n_enc, n_dec, vocab, max_pos, ln_post;
  int32_t pad_id, bos_id, eos_id, unk_id;
  float ln_eps;
  int32_t emb_dim; /* factorized embedding width (0: the embedding has width d_model) */
} mnmt_model_info;

/* Capacity of a session: batch, source and target lengths, beam width. */
typedef struct {
  int32_t max_batch;
  int32_t max_src_len;
  int32_t max_tgt_len;
  int32_t beam; /* 1 = greedy only */
} mnmt_session_cfg;

typedef struct {
  int32_t beam;              /* 1 = greedy search; else beam width (<= session beam) */
  int32_t max_steps;         /* decode steps (<= max_tgt_len) */
  float len_penalty_alpha;   /* beam: final score = score / ((5 + L) / 6)^alpha */
  int32_t stop_at_eos;       /* greedy: rows stop (PAD-fill) after EOS; beam always stops */
  int32_t use_graph;         /* replay a captured hipGraph of the whole search */
} mnmt_search_cfg;

/* ---- model --------------------------------------------------------------- */

/* Load flags (mnmt_model_bytes_ex, mnmt_model_load_ex).
 * MNMT_LOAD_PACKED_4BIT_ONLY: keep 4-bit weights only in their packed form
 * (half the bytes of int8 codes), without the int8 copy; every kernel then
 * reads the packed rows.  Every linear weight of the file must be 4-bit
 * (else MNMT_E_UNSUPPORTED). */
#define MNMT_LOAD_PACKED_4BIT_ONLY 1u

/* Validate a model file held in host memory and report the device arena size
 * it needs.  Host only.  blob: the whole file; device_bytes: out. */
int mnmt_model_bytes(const void* h_blob, size_t blob_bytes, size_t* device_bytes);

/* Load a model into a caller-allocated device arena (>= mnmt_model_bytes,
 * 256-byte aligned): validates, derives the folded fp32 constants in double
 * precision (each rounded once), lays the tensors out for the kernels and
 * copies them with one transfer on `stream`, then synchronizes `stream`.
 * *out receives a host handle; free it with mnmt_model_free (the arena stays
 * the caller's).  The model is bound to the current HIP device. */
int mnmt_model_load(const void* h_blob, size_t blob_bytes, void* d_arena, size_t arena_bytes,
                    void* stream, mnmt_model** out);

/* The same with load flags (MNMT_LOAD_*); flags 0 is mnmt_model_bytes /
 * mnmt_model_load. */
int mnmt_model_bytes_ex(const void* h_blob, size_t blob_bytes, unsigned flags, size_t* device_bytes);
int mnmt_model_load_ex(const void* h_blob, size_t blob_bytes, unsigned flags, void* d_arena, size_t arena_bytes,
                       void* stream, mnmt_model** out);

int mnmt_model_get_info(const mnmt_model* model, mnmt_model_info* out);
void mnmt_model_free(mnmt_model* model);

/* ---- session ------------------------------------------------------------- */

/* Workspace bytes for a session of capacity `cfg` (host only).  The plan
 * shares one region between encoder scratch and decoder logits (Section 4.2). */
int mnmt_session_bytes(const mnmt_model* model, const mnmt_session_cfg* cfg, size_t* bytes);

/* Create a session over a caller-allocated device workspace (>= the size
 * above, 256-byte aligned). */
int mnmt_session_create(const mnmt_model* model, const mnmt_session_cfg* cfg, void* d_ws,
                        size_t ws_bytes, mnmt_session** out);
void mnmt_session_free(mnmt_session* session);

/* Encode a batch: d_src [B, S_max] int32 row-major, right-padded; d_len [B]
 * int32 with 1 <= len <= S_max.  Computes the encoder output and every decoder
 * layer's cross-attention keys and values, and resets the decode state (step
 * 0, every row's next input BOS).  Asynchronous on `stream`.
 * Errors: MNMT_E_CAPACITY if B or S_max exceed the session. */
int mnmt_encode(mnmt_session* session, const int32_t* d_src, const int32_t* d_len, int B, int S_max,
                void* stream);

/* One greedy decoder step for the B rows of the last encode: input tokens
 * d_prev [B] (NULL: the session's device-resident tokens, BOS at step 0 or
 * the previous step's outputs), output d_next [B] = arg max of the logits
 * (smallest id among equal maxima), optional d_logits [B, V] fp32.  The step
 * index lives in device memory.  Errors: MNMT_E_CAPACITY past max_tgt_len;
 * MNMT_E_UNSUPPORTED on a session created with beam > 1 (beam search keeps
 * its hypotheses, parents and finished list across steps and runs only as a
 * whole search through mnmt_translate). */
int mnmt_decode_step(mnmt_session* session, const int32_t* d_prev, int32_t* d_next, float* d_logits,
                     void* stream);

/* Encode and search.  d_out [B, max_steps] int32 (PAD after the end),
 * d_out_len [B] int32, d_score [B] fp32 (beam: normalized score of the
 * returned hypothesis; greedy: unused, may be NULL).  Asynchronous: only
 * device work is enqueued (no host wait, no copy; capturable), and results
 * are valid after `stream` synchronizes.  Greedy with stop_at_eos = 0 runs
 * exactly max_steps steps.
 * Batch-1 greedy searches (and encoders of at most 64 rows) run as a chain of
 * kernels alternating between `stream` and a second session stream, each
 * kernel waiting in a bounded spin on its predecessor's flags or partial
 * sums (a decoder step is one launch per layer, its attention and FFN blocks
 * handing off the same way inside it, then the output projection): the chain
 * needs the two streams' kernels to run concurrently, which a tool that
 * serializes dispatches prevents (set MNMT_SERIAL_STEPS=1 in the environment
 * before creating the session to run them in one stream).  A wait that gives
 * up sets a session error word: every later translate writes -1 into
 * d_out_len until mnmt_session_status reports and clears it. */
int mnmt_translate(mnmt_session* session, const int32_t* d_src, const int32_t* d_len, int B,
                   int S_max, const mnmt_search_cfg* search, int32_t* d_out, int32_t* d_out_len,
                   float* d_score, void* stream);

/* Synchronizes `stream`, then reports (and clears) the session's error word:
 * MNMT_E_TIMEOUT if a chained kernel's wait gave up since the last call
 * (those translations' outputs are invalid), else MNMT_OK. */
int mnmt_session_status(mnmt_session* session, void* stream);

/* Device pointer and size of a session buffer, for inspection by tests:
 * "enc_out" int8 [B*S_max, d] (encoder output codes, padded rows undefined),
 * "cross_kv.<l>" int8 [B*S_max, 2d], "dec_x" fp32 [R, d], "logits" fp32 [R, V],
 * "step" int32 [1], "chain_err" int32 [1], "out_key" uint64 [max_tgt_len][R]
 * (greedy: each step's winning arg-max key, key(z) << 32 | (0xFFFFFFFF - id)
 * as MNMT_EPI_ARGMAX packs it), "kcache.<l>", "vcache.<l>" int8 [R][T][d]. */
int mnmt_session_tensor(const mnmt_session* session, const char* name, void** d_ptr, size_t* bytes);

/* ---- single quantized linear layer --------------------------------------- */

/* Y = epilogue(X W^T): d_X int8 [M, K] row-major (row stride K), d_W int8
 * [N, K] row-major (for MNMT_EPI_ARGMAX_PARTIAL_PACKED: mnmt_pack_weights'
 * copy of it), d_scale/d_bias fp32 [N] (bias may be NULL for I32, LOGITS and
 * the arg-max epilogues), d_Y [M, N] of the epilogue's type.  K must be a positive multiple
 * of 64 and at most 8192; M >= 0, N >= 1.  M <= 8 runs the wavefront
 * reduction kernel (the arg-max epilogue at M <= 2, K <= 512: the decoder's
 * logits kernel on the matrix cores), larger M the i8 matrix-core kernels. */
int mnmt_qlinear(const int8_t* d_X, const int8_t* d_W, const float* d_scale, const float* d_bias,
                 int M, int K, int N, int epilogue, float gamma, void* d_Y, void* stream);

/* mnmt_qlinear over 4-bit weights (the paper's W-E-A 4-8-8 setting, its
 * quantization study): d_W4 holds the packed rows [N, K / 2] of the model
 * file's 4-bit format (in each group of 16 codes of a row, byte i holds code
 * i in its low nibble and code i + 8 in its high nibble, each plus 8; 8-byte
 * aligned).  The kernels widen the codes to int8 as they load them, so Y is
 * what mnmt_qlinear gives for the int8 codes.  Epilogues MNMT_EPI_I32 ..
 * MNMT_EPI_LOGITS (not the arg-max ones: MNMT_E_UNSUPPORTED); otherwise as
 * mnmt_qlinear. */
int mnmt_qlinear_w4(const int8_t* d_X, const uint8_t* d_W4, const float* d_scale, const float* d_bias,
                    int M, int K, int N, int epilogue, float gamma, void* d_Y, void* stream);

/* Number of partial keys per row that MNMT_EPI_ARGMAX_PARTIAL writes for N
 * outputs (one per 128 outputs), or -1 for N < 1. */
int mnmt_argmax_partials(int N);

/* Bytes of the fragment-order copy of an int8 weight [N, K]:
 * ceil(N / 16) * 16 * K, or 0 unless N >= 1 and K is a positive multiple of 64. */
size_t mnmt_packed_bytes(int N, int K);

/* Reorder d_W int8 [N, K] row-major (16-byte aligned, K a multiple of 64) into
 * d_P (mnmt_packed_bytes(N, K) bytes, 16-byte aligned, caller-owned, not
 * overlapping d_W), asynchronously on the stream: for tile t of 16 rows and
 * slice j of 64 columns one contiguous kilobyte at offset (t * K/64 + j) * 1024
 * whose 16-byte chunk l holds W[16t + l % 16, 64j + 16(l / 16) .. +15] (zeros
 * for rows >= N) -- the operand each lane of an i8 16x16x64 matrix-core
 * instruction takes, so the logits kernel reads each kilobyte with one
 * coalesced load per wave.  This is a memory layout, not a change of the
 * arithmetic: MNMT_EPI_ARGMAX_PARTIAL_PACKED on d_P gives the keys that
 * MNMT_EPI_ARGMAX_PARTIAL gives on d_W. */
int mnmt_pack_weights(const int8_t* d_W, int N, int K, int8_t* d_P, void* stream);

/* mnmt_qlinear with timing events (hipEvent_t, created with timing enabled,
 * or NULL).  On the fused arg-max path (MNMT_EPI_ARGMAX,
 * MNMT_EPI_ARGMAX_PARTIAL or MNMT_EPI_ARGMAX_PARTIAL_PACKED, M <= 2, K <= 512:
 * the decoder's logits kernel on int8 rows) the two events take the kernel's
 * own start and end times (hipExtLaunchKernel), so their elapsed time is the
 * kernel's duration without launch gaps; on other paths they are recorded on
 * the stream before and after the launch. */
int mnmt_qlinear_timed(const int8_t* d_X, const int8_t* d_W, const float* d_scale, const float* d_bias,
                       int M, int K, int N, int epilogue, float gamma, void* d_Y, void* stream,
                       void* ev_start, void* ev_stop);

/* For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid allocation): the fused logits +
 * arg-max of mnmt_qlinear with MNMT_EPI_ARGMAX_PARTIAL_PACKED, reduced to each
 * row's final result without a caller buffer for the partial keys.  d_X int8
 * [M, K], d_Wp the fragment-order copy of W [N, K] (mnmt_pack_weights), d_scale
 * fp32 [N] (z = acc * scale[n]); outputs d_key [M] (the row's largest packed
 * key, key(z) << 32 | (0xFFFFFFFF - n), as MNMT_EPI_ARGMAX writes it) and/or
 * d_tok [M] int32 (its index: the arg max, smallest index among equal
 * maxima); either may be NULL, not both.  Limits: 1 <= M <= 2, K a multiple of
 * 64 up to 512, 1 <= N <= 262144 (else MNMT_E_INVALID_ARG).  The partial keys
 * live in a 32 KiB device array inside the library, one per GPU, held until
 * the process ends; the call allocates nothing.  Every call on a GPU uses that
 * GPU's array: calls that overlap on one GPU (other streams, other threads)
 * race and must be serialized by the caller. */
int mnmt_logits_argmax_noalloc(const int8_t* d_X, const int8_t* d_Wp, const float* d_scale, int M, int K, int N,
                               unsigned long long* d_key, int32_t* d_tok, void* stream);

/* Folded requantization constants (host): scale[n] = s_in*s_w[n]/s_out,
 * bias[n] = b[n]/s_out, each computed in double and rounded once to fp32. */
int mnmt_fold_requant(float s_in, const float* h_s_w, const float* h_b, float s_out, int N,
                      float* h_scale, float* h_bias);

/* ---- canonical arithmetic self-check -------------------------------------- */

/* Run the engine's device fp32 primitives on d_x[n] -> d_y[n]: fn 0 exp
 * (x <= 0), 1 natural log (x > 0), 2 canonical-order sum of all n values
 * into d_y[0].  For tests of the canonical arithmetic. */
int mnmt_debug_canon(int fn, const float* d_x, int n, float* d_y, void* stream);

/* Read bandwidth probe (not part of inference): 2048 blocks of 256 threads
 * read d_x [bytes] (16-byte aligned, bytes a multiple of 16) `reps` >= 1
 * times with 16-byte loads, each block the same share every time, and each
 * block stores one word into d_sink [2048].  Over a buffer that fits the
 * last-level cache but not the L2 caches, read many times, it measures the
 * last-level cache's bandwidth; over a buffer far larger than it, HBM's. */
int mnmt_debug_read(const void* d_x, size_t bytes, int reps, unsigned* d_sink, void* stream);

/* ---- errors ---------------------------------------------------------------- */
const char* mnmt_status_str(int status);
const char* mnmt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
